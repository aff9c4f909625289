"""Pins of the oracle's scorer (Section III-A cost equation, per-pool argmin).

Hand-worked examples (tests/golden/score_hand_examples.json) fix every term
of the equation; the property tests below fix its structure: permutation
equivariance, dominance, monotonicity in each feature, and the feature
removals of the ablation study (Section V-G) reducing to what they must.
"""
import json
import os

import numpy as np
import pytest

from oracle import oracle as O

GOLD = os.path.join(os.path.dirname(__file__), "golden", "score_hand_examples.json")
BASE = {"w_b": 1.0, "w_s": 1.0, "w_q": 1e-3, "rho": 1.0, "tau_pre_s": 1e-5, "tau_dec_s": 1.8e-3,
        "pre_base_s": 5e-3, "sigma": [2.0, 1.3333334, 1.1111112, 1.037037, 1, 1, 1, 1]}


def _score_one(router, pool, inst, req, kv_cap):
    n = len(inst["queue"])
    return O.score(router, pool, np.array(inst["backlog_s"], np.float32), np.array(inst["queue"], np.int32),
                   np.array(inst["kv_occ"], np.int32), kv_cap, n, 0, np.array(req["prompt_len"], np.int32),
                   np.array(req["pred_out_len"], np.int32), np.array(req["slo_class"], np.uint8))


@pytest.mark.parametrize("case", json.load(open(GOLD))["cases"], ids=lambda c: c["name"][:40])
def test_hand_examples(case):
    n = len(case["costs"])
    costs = []
    for j in range(n):  # one instance at a time gives each instance's own cost
        inst = {k: [v[j]] for k, v in case["instances"].items()}
        req = {k: [v] for k, v in case["request"].items()}
        _, sc, _ = _score_one(case["router"], case["pool"], inst, req, case["kv_cap"])
        costs.append(float(sc[0]))
    assert costs == case["costs"]
    req = {k: [v] for k, v in case["request"].items()}
    idx, sc, _ = _score_one(case["router"], case["pool"], case["instances"], req, case["kv_cap"])
    assert idx[0] == case["argmin"]
    assert float(sc[0]) == min(case["costs"])


def _rand_snapshot(rng, n_req, n_inst, per_request=False):
    rows = n_req if per_request else 1
    return dict(backlog_s=rng.uniform(0, 10, (rows, n_inst)).astype(np.float32).ravel(),
                queue=rng.integers(0, 257, (rows, n_inst)).astype(np.int32).ravel(),
                kv_occ=rng.integers(0, 200_000, (rows, n_inst)).astype(np.int32).ravel())


def _rand_req(rng, n):
    return (rng.integers(16, 8192, n).astype(np.int32), rng.integers(1, 4096, n).astype(np.int32),
            rng.integers(0, 4, n).astype(np.uint8))


@pytest.mark.parametrize("pool", ["prefill", "decode"])
def test_permutation_equivariance(pool):
    rng = np.random.default_rng(7)
    snap = _rand_snapshot(rng, 1, 33)
    p, oh, c = _rand_req(rng, 500)
    idx, sc, sec = O.score(BASE, pool, snap["backlog_s"], snap["queue"], snap["kv_occ"], 200_000, 33, 0, p, oh, c)
    perm = rng.permutation(33)
    idx2, sc2, _ = O.score(BASE, pool, snap["backlog_s"][perm], snap["queue"][perm], snap["kv_occ"][perm], 200_000,
                           33, 0, p, oh, c)
    assert np.array_equal(sc, sc2)
    distinct = sec > sc
    assert np.array_equal(perm[idx2[distinct]], idx[distinct])


def test_all_equal_state_picks_index_zero():
    n = 17
    idx, _, sec = O.score(BASE, "decode", np.full(n, 1.5, np.float32), np.full(n, 4, np.int32),
                          np.full(n, 1000, np.int32), 200_000, n, 0, np.array([100], np.int32),
                          np.array([50], np.int32), np.array([1], np.uint8))
    assert idx[0] == 0


def _costs_each(router, pool, b, q, kv, p, oh, c, kv_cap=200_000):
    """Cost of request (p, oh, c) on each instance separately: one 1-instance
    row per repeated request (inst_stride 1)."""
    n = len(b)
    return O.score(router, pool, b, q, kv, kv_cap, 1, 1, np.repeat(p, n), np.repeat(oh, n), np.repeat(c, n))[1]


def test_dominance():
    """An instance no worse on every state field never costs more."""
    rng = np.random.default_rng(3)
    for _ in range(200):
        b = rng.uniform(0, 5, 2).astype(np.float32)
        q = rng.integers(0, 50, 2).astype(np.int32)
        kv = rng.integers(0, 100_000, 2).astype(np.int32)
        b[1] = max(b[1], b[0]); q[1] = max(q[1], q[0]); kv[1] = max(kv[1], kv[0])
        p, oh, c = _rand_req(rng, 1)
        for pool in ("prefill", "decode"):
            c0, c1 = _costs_each(BASE, pool, b, q, kv, p, oh, c)
            assert c0 <= c1


@pytest.mark.parametrize("field", ["backlog_s", "queue", "kv_occ"])
@pytest.mark.parametrize("pool", ["prefill", "decode"])
def test_monotone_in_each_state_field(field, pool):
    rng = np.random.default_rng(11)
    n = 64
    snap = _rand_snapshot(rng, 1, n)
    vary = {k: np.full(n, snap[k][0], snap[k].dtype) for k in snap}
    vary[field] = np.sort(snap[field])
    p, oh, c = _rand_req(rng, 20)
    for i in range(20):
        costs = _costs_each(BASE, pool, vary["backlog_s"], vary["queue"], vary["kv_occ"], p[i], oh[i], c[i])
        assert np.all(np.diff(costs) >= 0)
        assert costs[-1] > costs[0]
        idx = O.score(BASE, pool, vary["backlog_s"], vary["queue"], vary["kv_occ"], 200_000, n, 0,
                      p[i:i + 1], oh[i:i + 1], c[i:i + 1])[0]
        assert idx[0] == 0


def test_ablation_reductions():
    """Section V-G feature removals: rho=0 drops occupancy, sigma=1 drops the
    class, w_s=0 drops the predicted length."""
    rng = np.random.default_rng(5)
    snap = _rand_snapshot(rng, 1, 24)
    p, oh, c = _rand_req(rng, 300)

    r0 = dict(BASE, rho=0.0)
    a = O.score(r0, "decode", snap["backlog_s"], snap["queue"], snap["kv_occ"], 200_000, 24, 0, p, oh, c)
    b = O.score(r0, "decode", snap["backlog_s"], snap["queue"], rng.permutation(snap["kv_occ"]), 200_000, 24, 0,
                p, oh, c)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])

    r1 = dict(BASE, sigma=[1.0] * 8)
    a = O.score(r1, "decode", snap["backlog_s"], snap["queue"], snap["kv_occ"], 200_000, 24, 0, p, oh, c)
    b = O.score(r1, "decode", snap["backlog_s"], snap["queue"], snap["kv_occ"], 200_000, 24, 0, p, oh,
                (c + 1) % 4)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])

    r2 = dict(BASE, w_s=0.0)
    a = O.score(r2, "decode", snap["backlog_s"], snap["queue"], snap["kv_occ"], 200_000, 24, 0, p, oh, c)
    # occupancy still sees the predicted length through press+, which is
    # multiplied by the zeroed size term: the cost must not move at all
    b = O.score(r2, "decode", snap["backlog_s"], snap["queue"], snap["kv_occ"], 200_000, 24, 0, p, oh * 3 + 1, c)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_queue_term_only_is_join_shortest_queue():
    rng = np.random.default_rng(9)
    snap = _rand_snapshot(rng, 1, 40)
    p, oh, c = _rand_req(rng, 200)
    r = dict(BASE, w_b=0.0, w_s=0.0, w_q=1.0)
    idx, sc, _ = O.score(r, "decode", snap["backlog_s"], snap["queue"], snap["kv_occ"], 200_000, 40, 0, p, oh, c)
    assert np.all(idx == np.argmin(snap["queue"]))
    assert np.all(sc == snap["queue"].min())


def test_sigma_scales_load_terms_not_queue():
    """sigma(s) multiplies the backlog and size terms and leaves w_q*queue alone."""
    one = dict(BASE, w_q=0.0)
    q_only = dict(BASE, w_b=0.0, w_s=0.0, w_q=0.5)
    b = np.array([0.5], np.float32); q = np.array([4], np.int32); kv = np.array([1024], np.int32)
    p = np.array([64], np.int32); oh = np.array([32], np.int32)
    c0 = O.score(one, "decode", b, q, kv, 200_000, 1, 0, p, oh, np.array([0], np.uint8))[1][0]
    c3 = O.score(one, "decode", b, q, kv, 200_000, 1, 0, p, oh, np.array([3], np.uint8))[1][0]
    # sigma_0 = 2 and sigma_3 = 1.037037: the ratio carries through exactly up to rounding
    assert c0 / c3 == pytest.approx(2.0 / 1.037037, rel=1e-6)
    q0 = O.score(q_only, "decode", b, q, kv, 200_000, 1, 0, p, oh, np.array([0], np.uint8))[1][0]
    q3 = O.score(q_only, "decode", b, q, kv, 200_000, 1, 0, p, oh, np.array([3], np.uint8))[1][0]
    assert q0 == q3 == 2.0


def test_per_request_snapshot_rows():
    rng = np.random.default_rng(4)
    n_req, n = 50, 12
    snap = _rand_snapshot(rng, n_req, n, per_request=True)
    p, oh, c = _rand_req(rng, n_req)
    idx, sc, _ = O.score(BASE, "decode", snap["backlog_s"], snap["queue"], snap["kv_occ"], 200_000, n, n, p, oh, c)
    for i in range(n_req):
        s = slice(i * n, (i + 1) * n)
        j, v, _ = O.score(BASE, "decode", snap["backlog_s"][s], snap["queue"][s], snap["kv_occ"][s], 200_000, n, 0,
                          p[i:i + 1], oh[i:i + 1], c[i:i + 1])
        assert j[0] == idx[i] and v[0] == sc[i]


def test_invalid_requests_flagged():
    snap = dict(backlog_s=np.zeros(3, np.float32), queue=np.zeros(3, np.int32), kv_occ=np.zeros(3, np.int32))
    p = np.array([0, 5, 5, 5, 2 ** 30], np.int32)
    oh = np.array([5, 0, 5, 5, 2 ** 30], np.int32)
    c = np.array([0, 0, 8, 7, 0], np.uint8)
    idx, sc, _ = O.score(BASE, "decode", snap["backlog_s"], snap["queue"], snap["kv_occ"], 1000, 3, 0, p, oh, c)
    assert list(idx) == [-1, -1, -1, 0, -1]
    assert np.isnan(sc[[0, 1, 2, 4]]).all() and np.isfinite(sc[3])
    # prefill does not read the predicted length
    idx, _, _ = O.score(BASE, "prefill", snap["backlog_s"], snap["queue"], snap["kv_occ"], 1000, 3, 0, p, oh, c)
    assert list(idx) == [-1, 0, -1, 0, 0]
