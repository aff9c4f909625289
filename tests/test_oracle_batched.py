"""Pins of the oracle's continuous-batching service model (Section VI: the
paper's correction to the serial model, continuous batching at the prefill and the decode stage alike,
a batch of b slowing each member by 1 + beta (b - 1)).  CPU only.

What fixes it, beyond the oracle's own code:
  * requests that never overlap see the serial model exactly (a batch of one
    runs at full speed), under every policy;
  * beta = 0 is an infinite-server system: every request's stage times are
    its stand-alone service times, whatever the load;
  * closed forms: b equal requests joining one decode instance together
    finish after W (1 + beta (b - 1)); two staggered joins; a burst under pure
    processor sharing (beta = 1) leaves in order of size, the k-th smallest
    at the sum of the smaller works plus (b - k + 1) times its own;
  * queueing theory: one prefill instance under beta = 1 is M/G/1
    processor sharing, whose mean sojourn is E[S] / (1 - rho) and whose
    conditional mean sojourn is linear in the job size with slope
    1 / (1 - rho);
  * an independent brute force (remaining work per request instead of a
    virtual clock per instance), exact in rationals on tiny traces and in
    floats on small ones, agrees to within 1 ns with the same placements;
  * conservation: every count returns to zero and no invariant breaks.
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle as O
from oracle.ps_brute import simulate_batched
from paper_2609_16206_amd import workload as W

KEYS = ("arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class")
OUTS = ("i_pre", "i_dec", "ttft_ns", "decode_span_ns")
POLICIES = [("learned", "true"), ("learned", "proxy"), ("round_robin", "true"), ("least_loaded", "true"),
            ("learned_sampled", "true"), ("length_threshold", "true")]


def _trace(P, D, n, seed, scale=1.0, reps=1, traffic=None):
    pt = W.make_point(P, D, n_classes=3)
    wl = W.Workload("t", seed, reps, n, [pt], [(traffic or W.mixed_bursty()).scaled(scale)])
    tr = W.make_trace(wl)
    W.add_sample_words(tr, seed)
    return tr


def _args(tr, i=0):
    sl = slice(int(tr["offsets"][i]), int(tr["offsets"][i + 1]))
    return [tr[k][sl] for k in KEYS], tr["sample_bits"][sl]


def _work(pt, p, o):
    w_pre = pt["pre_base_ns"] + p.astype(np.int64) * pt["pre_tok_ns"]
    w_dec = (o.astype(np.int64) - 1) * pt["dec_tok_ns"]
    return w_pre, w_dec, p.astype(np.int64) * pt["xfer_tok_ns"]


@pytest.mark.parametrize("policy,mode", POLICIES)
def test_no_overlap_equals_serial(policy, mode):
    tr = _trace(3, 4, 400, seed=5)
    (a, p, o, oh, c), words = _args(tr)
    ser = W.make_point(3, 4, n_classes=3, policy=policy, backlog_mode=mode)
    w_pre, w_dec, xf = _work(ser, p, o)
    # space arrivals beyond the longest request's whole stay
    gap = int((w_pre + w_dec + xf).max()) + 1
    a = np.arange(len(a), dtype=np.int64) * gap
    bat = dict(ser, service="batched", beta_pre=0.3, beta_dec=0.05)
    ref, _ = O.sim_replica(ser, a, p, o, oh, c, sample_bits=words)
    out, st = O.sim_replica(bat, a, p, o, oh, c, sample_bits=words)
    assert st["violations"] == 0
    for k in OUTS:
        assert np.array_equal(out[k], ref[k]), k
    assert np.array_equal(out["ttft_ns"], w_pre)
    assert np.array_equal(out["decode_span_ns"], xf + w_dec)


@pytest.mark.parametrize("policy,mode", POLICIES)
def test_beta_zero_is_infinite_server(policy, mode):
    tr = _trace(2, 6, 3000, seed=7, scale=3.0)  # far beyond serial capacity
    (a, p, o, oh, c), words = _args(tr)
    pt = W.make_point(2, 6, n_classes=3, policy=policy, backlog_mode=mode, service="batched", beta_pre=0.0,
                      beta_dec=0.0)
    out, st = O.sim_replica(pt, a, p, o, oh, c, sample_bits=words)
    w_pre, w_dec, xf = _work(pt, p, o)
    assert st["violations"] == 0 and st["invalid"] == 0
    assert np.array_equal(out["ttft_ns"], w_pre)
    assert np.array_equal(out["decode_span_ns"], xf + w_dec)
    assert st["max_queue_dec"] > 1  # requests did overlap


def _closed_point(P, D, beta_pre, beta_dec, **kw):
    pt = W.make_point(P, D, n_classes=1, policy="round_robin", service="batched", beta_pre=beta_pre,
                      beta_dec=beta_dec, **kw)
    pt.update(pre_base_ns=1_000_000, pre_tok_ns=1000, dec_tok_ns=1_000_000, xfer_tok_ns=100)
    return pt


def _rint(x):
    return int(round(Fraction(x)))


@pytest.mark.parametrize("b", [1, 2, 3, 5, 8, 13])
@pytest.mark.parametrize("beta", [0.029 / 7, 0.125, 1.0])
def test_equal_decode_joins_closed_form(b, beta):
    # b equal requests at t = 0, each on its own prefill instance, one decode
    # instance: they join together and leave together after W (1 + beta (b-1)).
    pt = _closed_point(b, 1, beta_pre=0.5, beta_dec=beta)
    p = np.full(b, 300, np.int32)
    o = np.full(b, 41, np.int32)
    out, st = O.sim_replica(pt, np.zeros(b, np.int64), p, o, o, np.zeros(b, np.uint8))
    assert st["violations"] == 0
    w_pre, w_dec, xf = 1_000_000 + 300 * 1000, 40 * 1_000_000, 300 * 100
    assert np.all(out["ttft_ns"] == w_pre)
    exact = xf + Fraction(w_dec) * (1 + Fraction(beta) * (b - 1))
    assert np.all(np.abs(out["decode_span_ns"] - _rint(exact)) <= 1)


@pytest.mark.parametrize("beta", [0.029 / 7, 0.25, 1.0])
@pytest.mark.parametrize("delta", [1, 7_000_000, 39_999_999])
def test_staggered_decode_pair_closed_form(beta, delta):
    # A joins at J, B at J + delta (delta < W): A runs alone for delta, then
    # both share at 1 + beta; A leaves after W - delta more work, B then has
    # delta of work left and runs alone.
    pt = _closed_point(2, 1, beta_pre=0.0, beta_dec=beta)
    p = np.array([300, 300], np.int32)
    o = np.array([41, 41], np.int32)
    a = np.array([0, delta], np.int64)
    out, st = O.sim_replica(pt, a, p, o, o, np.zeros(2, np.uint8))
    assert st["violations"] == 0
    W_ = Fraction(40 * 1_000_000)
    xf = 300 * 100
    s = 1 + Fraction(beta)
    end_a = delta + (W_ - delta) * s
    end_b = end_a + delta
    assert abs(int(out["decode_span_ns"][0]) - _rint(xf + end_a)) <= 1
    assert abs(int(out["decode_span_ns"][1]) - _rint(xf + end_b - delta)) <= 1


def test_processor_sharing_burst_order_and_times():
    # beta = 1 is pure processor sharing: the instance's total rate is 1.
    rng = np.random.default_rng(3)
    b = 12
    p = rng.integers(1, 5000, b).astype(np.int32)
    pt = _closed_point(1, b, beta_pre=1.0, beta_dec=0.0)
    pt.update(pre_base_ns=0)
    o = np.ones(b, np.int32)
    out, st = O.sim_replica(pt, np.zeros(b, np.int64), p, o, o, np.zeros(b, np.uint8))
    assert st["violations"] == 0
    w = p.astype(np.int64) * 1000
    ws = np.sort(w)
    for r in range(b):
        k = int(np.searchsorted(ws, w[r]))  # 0-based rank among the smaller
        want = int(ws[:k].sum()) + (b - k) * int(w[r])
        assert abs(int(out["ttft_ns"][r]) - want) <= 1
    assert int(out["ttft_ns"].max()) == int(w.sum())  # work conserving


def test_mg1_processor_sharing_mean_sojourn():
    # One prefill instance with beta = 1, Poisson arrivals at load rho,
    # uniform job sizes: E[T] = E[S] / (1 - rho), E[T | S] = S / (1 - rho).
    rng = np.random.default_rng(12)
    n, rho = 120_000, 0.6
    p = rng.integers(1, 2001, n).astype(np.int32)
    es = 1000.5 * 1000.0  # ns
    gaps = rng.exponential(es / rho, n)
    a = np.cumsum(gaps).astype(np.int64)
    pt = _closed_point(1, 1, beta_pre=1.0, beta_dec=0.0)
    pt.update(pre_base_ns=0, pre_tok_ns=1000, xfer_tok_ns=0)
    o = np.ones(n, np.int32)
    out, st = O.sim_replica(pt, a, p, o, o, np.zeros(n, np.uint8))
    assert st["violations"] == 0
    T = out["ttft_ns"][n // 10:].astype(np.float64)  # drop the warm-up
    S = p[n // 10:].astype(np.float64) * 1000.0
    assert abs(T.mean() / (es / (1 - rho)) - 1.0) < 0.05
    slope = np.polyfit(S, T, 1)[0]
    assert abs(slope * (1 - rho) - 1.0) < 0.06


def _follow_check(pt, a, p, o, oh, c, words, ref, exact=None):
    """The oracle follows the brute force's placements: no divergence beyond
    a near-tie, times within 1 ns, and (given the brute force's exact
    unrounded times) equal wherever the exact time is not within 1e-4 ns of
    a rounding boundary."""
    out, st = O.sim_replica(pt, a, p, o, oh, c, follow_pre=ref["i_pre"], follow_dec=ref["i_dec"], tie_rel=1e-5,
                            sample_bits=words)
    assert st["violations"] == 0
    assert st["mismatch_pre"] == 0 and st["mismatch_dec"] == 0
    for k in ("ttft_ns", "decode_span_ns"):
        assert int(np.abs(out[k] - ref[k]).max()) <= 1, k
        if exact is not None:
            frac = np.array([float(x - int(x)) for x in exact[k]])  # exact values are >= 0
            clear = np.abs(frac - 0.5) > 1e-4
            assert np.array_equal(out[k][clear], ref[k][clear]), k
    return out, st


@pytest.mark.parametrize("policy,mode", POLICIES)
@pytest.mark.parametrize("seed", [1, 2])
def test_brute_force_exact_rationals(policy, mode, seed):
    tr = _trace(2, 3, 28, seed=20 + seed, scale=2.5)
    (a, p, o, oh, c), words = _args(tr)
    pt = W.make_point(2, 3, n_classes=3, policy=policy, backlog_mode=mode, service="batched", beta_pre=0.125,
                      beta_dec=0.25)
    ref = simulate_batched(pt, a, p, o, oh, c, words=words, exact=True)
    out, st = _follow_check(pt, a, p, o, oh, c, words, ref, exact=ref["exact"])
    assert st["max_queue_pre"] > 1 or st["max_queue_dec"] > 1


@pytest.mark.parametrize("policy,mode", POLICIES)
def test_brute_force_floats(policy, mode):
    tr = _trace(2, 6, 400, seed=31, scale=2.0)
    (a, p, o, oh, c), words = _args(tr)
    pt = W.make_point(2, 6, n_classes=3, policy=policy, backlog_mode=mode, service="batched")
    ref = simulate_batched(pt, a, p, o, oh, c, words=words)
    _follow_check(pt, a, p, o, oh, c, words, ref)
    own, _ = O.sim_replica(pt, a, p, o, oh, c, sample_bits=words)
    # without following, the placements agree except at near-ties
    assert np.mean(own["i_dec"] == ref["i_dec"]) > 0.95


@pytest.mark.parametrize("policy,mode", POLICIES)
def test_conservation_under_overload(policy, mode):
    tr = _trace(2, 6, 5000, seed=41, scale=4.0, reps=2)
    pt = W.make_point(2, 6, n_classes=3, policy=policy, backlog_mode=mode, service="batched", beta_pre=0.5)
    for i in range(2):
        (a, p, o, oh, c), words = _args(tr, i)
        out, st = O.sim_replica(pt, a, p, o, oh, c, sample_bits=words)
        assert st["violations"] == 0 and st["invalid"] == 0
        assert st["retired_pre"] + st["end_inflight_pre"] == len(a)
        assert st["retired_dec"] + st["end_inflight_dec"] == len(a)
        w_pre, w_dec, xf = _work(pt, p, o)
        assert np.all(out["ttft_ns"] >= w_pre)  # sharing never speeds a request up
        assert np.all(out["decode_span_ns"] >= xf + w_dec)


@pytest.mark.parametrize("beta", [0.0, 0.125, 1.0])
def test_completion_at_an_arrival_leaves_first(beta):
    # A alone on prefill 0 ends at exactly W; B arrives at W.  The completion
    # comes first, so both prefill instances are idle for B and the least
    # loaded choice is instance 0 (lowest index), not instance 1.
    pt = _closed_point(2, 1, beta_pre=beta, beta_dec=beta)
    pt["policy"] = "least_loaded"
    w_pre = 1_000_000 + 300 * 1000
    p = np.array([300, 300, 300], np.int32)
    o = np.array([5, 5, 5], np.int32)
    a = np.array([0, w_pre, w_pre + 1], np.int64)
    out, st = O.sim_replica(pt, a, p, o, o, np.zeros(3, np.uint8))
    assert st["violations"] == 0
    assert list(out["i_pre"]) == [0, 0, 1]
    assert st["retired_pre"] == 1


def test_rejects_like_serial():
    tr = _trace(2, 2, 50, seed=3)
    (a, p, o, oh, c), _ = _args(tr)
    p = p.copy()
    p[7] = 0
    a = a.copy()
    a[20] = a[19] - 1
    pt = W.make_point(2, 2, n_classes=3, service="batched")
    out, st = O.sim_replica(pt, a, p, o, oh, c)
    assert st["invalid"] == 2 and st["violations"] == 0
    for k in OUTS:
        assert out[k][7] == -1 and out[k][20] == -1


def test_bad_beta_rejected():
    tr = _trace(2, 2, 10, seed=3)
    (a, p, o, oh, c), _ = _args(tr)
    for bad in (-0.1, float("nan"), float("inf")):
        pt = W.make_point(2, 2, n_classes=3, service="batched", beta_dec=bad)
        with pytest.raises(ValueError):
            O.sim_replica(pt, a, p, o, oh, c)


def test_random_tiny_traces_match_exact_brute_force():
    """Many random tiny traces on a coarse time grid (simultaneous arrivals,
    equal works, so equal finish times and landings at equal times are
    frequent), every policy, dyadic betas (so exact rationals stay small):
    the oracle following the brute force's placements has no divergence
    beyond a near-tie and its times are the exact ones rounded (within 1 ns
    where the exact value is within 1e-4 ns of a half)."""
    rng = np.random.default_rng(77)
    pols = POLICIES
    for trial in range(150):
        P, D = int(rng.integers(1, 4)), int(rng.integers(1, 4))
        n = int(rng.integers(1, 13))
        policy, mode = pols[trial % len(pols)]
        pt = W.make_point(P, D, n_classes=2, policy=policy, backlog_mode=mode, service="batched",
                          beta_pre=float(rng.choice([0.0, 0.125, 0.5, 1.0])),
                          beta_dec=float(rng.choice([0.0, 0.25, 1.0])), len_threshold=3)
        pt.update(pre_base_ns=int(rng.choice([0, 4])), pre_tok_ns=int(rng.choice([1, 2])),
                  dec_tok_ns=int(rng.choice([1, 3])), xfer_tok_ns=int(rng.choice([0, 1])))
        a = np.sort(rng.integers(0, 8, n)).astype(np.int64) * 4
        p = rng.integers(1, 5, n).astype(np.int32)
        o = rng.integers(1, 5, n).astype(np.int32)
        oh = rng.integers(1, 6, n).astype(np.int32)
        c = rng.integers(0, 2, n).astype(np.uint8)
        words = rng.integers(0, 2 ** 32, (n, 4), dtype=np.uint64).astype(np.uint32)
        ref = simulate_batched(pt, a, p, o, oh, c, words=words, exact=True)
        _follow_check(pt, a, p, o, oh, c, words, ref, exact=ref["exact"])
