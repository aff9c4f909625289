"""Pins of the oracle's sampled policy: the learned score over two randomly
drawn candidates per pool (the mitigation Section V-E and Section VI name for
scarce pools).  CPU only.

What fixes it, beyond the oracle's own code:
  * a pool of at most two instances offers both, so the policy is then the
    full learned argmin exactly (checked against the learned policy);
  * the candidate rule draws an ordered pair of distinct instances, every
    pair equally likely (chi-square against the uniform law);
  * choosing the cheaper of two uniformly drawn distinct instances picks the
    instance of cost rank k (0 = cheapest of n) with probability
    (n - 1 - k) / C(n, 2), a combinatorial closed form (chi-square);
  * the event-heap simulation agrees with it on random tiny traces (in
    test_oracle_sim.test_event_heap_bruteforce_agrees).
"""
import math

import numpy as np
import pytest

from oracle import oracle as O
from paper_2609_16206_amd import workload as W

pytestmark = pytest.mark.filterwarnings("ignore")


def _chi2_ok(counts, probs, alpha_z=4.5):
    """Pearson chi-square against expected probabilities, judged through the
    Wilson-Hilferty normal approximation (|z| < alpha_z: about 3e-6 two-sided
    at 4.5), so no table is needed."""
    counts = np.asarray(counts, np.float64)
    n = counts.sum()
    exp = n * np.asarray(probs, np.float64)
    chi2 = float(((counts - exp) ** 2 / exp).sum())
    k = len(counts) - 1
    z = ((chi2 / k) ** (1 / 3) - (1 - 2 / (9 * k))) / math.sqrt(2 / (9 * k))
    return abs(z) < alpha_z, chi2, z


def test_candidates_range_and_extremes():
    rng = np.random.default_rng(5)
    for n in range(1, 12):
        for u, v in rng.integers(0, 1 << 32, size=(300, 2), dtype=np.uint64):
            c1, c2 = O.candidates(int(u), int(v), n)
            assert 0 <= c1 < n and 0 <= c2 < n
            assert (c1 != c2) if n >= 2 else (c1 == c2 == 0)
        # the extreme words reach the ends of the range
        assert O.candidates(0, 0, n)[0] == 0
        assert O.candidates(0xFFFFFFFF, 0, n)[0] == n - 1
        if n >= 2:
            assert O.candidates(0, 0, n)[1] == 1            # first of the others
            assert O.candidates(0, 0xFFFFFFFF, n)[1] == n - 1
            assert O.candidates(0xFFFFFFFF, 0xFFFFFFFF, n)[1] == n - 2


@pytest.mark.parametrize("n", [2, 3, 5, 8])
def test_candidate_pairs_uniform(n):
    rng = np.random.default_rng(100 + n)
    words = rng.integers(0, 1 << 32, size=(40_000, 2), dtype=np.uint64)
    counts = np.zeros((n, n), np.int64)
    for u, v in words:
        c1, c2 = O.candidates(int(u), int(v), n)
        counts[c1, c2] += 1
    assert np.all(np.diag(counts) == 0)
    off = counts[~np.eye(n, dtype=bool)]
    ok, chi2, z = _chi2_ok(off, np.full(off.size, 1.0 / off.size))
    assert ok, (n, chi2, z)


@pytest.mark.parametrize("n", [3, 4, 7, 16])
def test_rank_law_of_two_choices(n):
    """Costs strictly increasing with the index (queue only: w_b = w_s = 0,
    w_q = 1): the choice's rank law is (n - 1 - k) / C(n, 2)."""
    rng = np.random.default_rng(7 + n)
    m = 30_000
    router = dict(w_b=0.0, w_s=0.0, w_q=1.0, rho=0.0, tau_pre_s=1e-5, tau_dec_s=1e-3, pre_base_s=0.0,
                  sigma=[1.0] * 8)
    backlog = np.zeros(n, np.float32)
    queue = np.arange(n, dtype=np.int32)
    kv = np.zeros(n, np.int32)
    p = np.full(m, 100, np.int32)
    oh = np.full(m, 50, np.int32)
    c = np.zeros(m, np.uint8)
    words = rng.integers(0, 1 << 32, size=(m, 2), dtype=np.uint64).astype(np.uint32)
    idx, sc, sec = O.score(router, "decode", backlog, queue, kv, 200_000, n, 0, p, oh, c, sample_bits=words)
    assert np.all(sc == idx.astype(np.float32))          # the cost of the pick is its queue
    assert np.all(sec > sc)                               # the other candidate costs more
    counts = np.bincount(idx, minlength=n)
    assert counts[n - 1] == 0                             # the dearest is never chosen
    probs = np.array([(n - 1 - k) / math.comb(n, 2) for k in range(n - 1)])
    ok, chi2, z = _chi2_ok(counts[:n - 1], probs)
    assert ok, (n, counts, chi2, z)


def test_one_instance_pool():
    router = dict(w_b=1.0, w_s=1.0, w_q=1e-3, rho=1.0, tau_pre_s=1e-5, tau_dec_s=1e-3, pre_base_s=0.0,
                  sigma=[1.0] * 8)
    one = np.ones(1, np.float32)
    words = np.array([[0xFFFFFFFF, 123], [0, 0]], np.uint32)
    idx, sc, sec = O.score(router, "prefill", one, np.zeros(1, np.int32), np.zeros(1, np.int32), 1000, 1, 0,
                           np.array([5, 6], np.int32), np.array([1, 1], np.int32), np.zeros(2, np.uint8),
                           sample_bits=words)
    assert list(idx) == [0, 0] and np.all(np.isinf(sec))


@pytest.mark.parametrize("P,D", [(1, 1), (1, 2), (2, 1), (2, 2)])
@pytest.mark.parametrize("mode", ["true", "proxy"])
def test_pools_of_two_are_the_full_argmin(P, D, mode):
    """Two candidates out of at most two instances are the whole pool."""
    wl = W.Workload("t", 9, 3, 3000, [W.make_point(P, D, n_classes=3, backlog_mode=mode)], [W.mixed_bursty()])
    tr = W.make_trace(wl)
    W.add_sample_words(tr, 9)
    ptl = W.make_point(P, D, n_classes=3, backlog_mode=mode)
    pts = W.make_point(P, D, n_classes=3, backlog_mode=mode, policy="learned_sampled")
    for i in range(3):
        sl = slice(int(tr["offsets"][i]), int(tr["offsets"][i + 1]))
        args = [tr[k][sl] for k in ("arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class")]
        a, sa = O.sim_replica(ptl, *args)
        b, sb = O.sim_replica(pts, *args, sample_bits=tr["sample_bits"][sl])
        for k in a:
            assert np.array_equal(a[k], b[k]), (P, D, mode, i, k)
        assert sa["violations"] == sb["violations"] == 0


def test_sampled_placements_are_candidates_and_conserve():
    """On a wide pool: every placement is one of the request's two candidates
    and the cheaper of them on the state the oracle rebuilds; the simulation
    keeps its invariants."""
    pt = W.make_point(3, 9, n_classes=3, policy="learned_sampled")
    wl = W.Workload("t", 4, 2, 4000, [pt], [W.mixed_bursty().scaled(1.5)])
    tr = W.make_trace(wl)
    assert "sample_bits" in tr
    for i in range(2):
        sl = slice(int(tr["offsets"][i]), int(tr["offsets"][i + 1]))
        args = [tr[k][sl] for k in ("arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class")]
        w = tr["sample_bits"][sl]
        out, st = O.sim_replica(pt, *args, sample_bits=w)
        assert st["violations"] == 0 and st["invalid"] == 0
        for r in range(len(w)):
            assert out["i_pre"][r] in O.candidates(w[r, 0], w[r, 1], 3)
            assert out["i_dec"][r] in O.candidates(w[r, 2], w[r, 3], 9)
        # a sampled router does not reduce to the full argmin on wide pools
        full, _ = O.sim_replica(W.make_point(3, 9, n_classes=3), *args)
        assert not np.array_equal(full["i_dec"], out["i_dec"])


def test_sampled_needs_words():
    pt = W.make_point(2, 3, policy="learned_sampled")
    z = np.zeros(2, np.int64)
    o = np.ones(2, np.int32)
    with pytest.raises(ValueError):
        O.sim_replica(pt, z, o, o, o, np.zeros(2, np.uint8))
