"""Pins of the oracle's replica simulation.

Closed forms and special cases that the paper's router and simulator fix:
  * round-robin is r mod N (Section IV-C baselines);
  * simultaneous identical requests spread cyclically under the learned
    router and least-loaded alike;
  * the learned score with only the queue term is least-loaded exactly, and
    a ledger priced with zero constants collapses to queue counting (Section
    III-B / V-B: mispriced constants reduce the router to queue counting);
  * one prefill and one decode instance form a tandem of single-server FIFO
    queues whose departure times have the max-plus closed form;
  * a single Poisson-fed prefill instance has the Pollaczek-Khinchine mean
    wait;
  * brute force: an independent event-heap simulation agrees exactly;
  * conservation, FIFO order and drain-to-zero, and an independent
    recomputation of every learned decision from the recorded trajectory.
"""
import math

import numpy as np
import pytest

from oracle import des_heap as H
from oracle import oracle as O
from paper_2609_16206_amd import workload as W


def _trace(n, rng, rate=4.0, p_rng=(16, 4096), o_rng=(1, 2048), n_classes=2):
    arr = np.cumsum(rng.exponential(1.0 / rate, n) * 1e9).astype(np.int64)
    p = rng.integers(*p_rng, n).astype(np.int32)
    o = rng.integers(*o_rng, n).astype(np.int32)
    oh = np.maximum(1, (o * np.exp(0.3 * rng.standard_normal(n)))).astype(np.int32)
    c = rng.integers(0, n_classes, n).astype(np.uint8)
    return arr, p, o, oh, c


def _run(pt, tr, **kw):
    return O.sim_replica(pt, *tr, **kw)


@pytest.mark.parametrize("P,D", [(1, 1), (2, 6), (3, 3), (5, 17)])
def test_round_robin_exact(P, D):
    rng = np.random.default_rng(P * 100 + D)
    tr = _trace(3000, rng)
    out, st = _run(W.make_point(P, D, policy="round_robin"), tr)
    r = np.arange(3000)
    assert np.array_equal(out["i_pre"], r % P)
    assert np.array_equal(out["i_dec"], r % D)
    assert st["violations"] == 0


@pytest.mark.parametrize("policy", ["learned", "least_loaded"])
@pytest.mark.parametrize("mode", ["true", "proxy"])
def test_simultaneous_identical_requests_spread_cyclically(policy, mode):
    n, P, D = 97, 3, 7
    tr = (np.zeros(n, np.int64), np.full(n, 300, np.int32), np.full(n, 40, np.int32), np.full(n, 40, np.int32),
          np.zeros(n, np.uint8))
    out, st = _run(W.make_point(P, D, policy=policy, backlog_mode=mode), tr)
    r = np.arange(n)
    assert np.array_equal(out["i_pre"], r % P)
    assert np.array_equal(out["i_dec"], r % D)


@pytest.mark.parametrize("mode", ["true", "proxy"])
def test_queue_only_learned_equals_least_loaded(mode):
    wl = W.paper_cluster(n_replicas=3, requests=4000)
    tr = W.make_trace(wl, workers=1)
    for i in range(3):
        sl = slice(int(tr["offsets"][i]), int(tr["offsets"][i + 1]))
        args = [tr[k][sl] for k in ("arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class")]
        a, _ = O.sim_replica(W.make_point(2, 6, n_classes=3, policy="learned", backlog_mode=mode, w_b=0.0, w_s=0.0,
                                          w_q=1.0), *args)
        b, _ = O.sim_replica(W.make_point(2, 6, n_classes=3, policy="least_loaded", backlog_mode=mode), *args)
        for k in a:
            assert np.array_equal(a[k], b[k]), k


def test_zero_priced_ledger_collapses_to_queue_counting():
    wl = W.paper_cluster(n_replicas=2, requests=4000)
    tr = W.make_trace(wl, workers=1)
    args = [tr[k][:4000] for k in ("arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class")]
    pt = W.make_point(2, 6, n_classes=3, backlog_mode="proxy", tau_pre_scale=0.0, tau_dec_scale=0.0)
    pt["pre_base_s"] = 0.0
    a, _ = O.sim_replica(pt, *args)
    b, _ = O.sim_replica(W.make_point(2, 6, n_classes=3, policy="least_loaded"), *args)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def test_mispricing_moves_router_towards_queue_counting():
    """Directional (Section III-B, V-B): as the ledger's priced constants shrink
    relative to the queue term, the router's decode choices agree more with
    least-loaded.  Agreement is counted along the router's own trajectory
    (least-loaded run in follow mode: every differing choice is a mismatch)."""
    wl = W.paper_cluster(n_replicas=4, requests=3000)
    tr = W.make_trace(wl, workers=1)
    agree = []
    for scale in (1.0, 1.0 / 1024, 1.0 / 4096, 0.0):
        same = 0
        for i in range(4):
            sl = slice(i * 3000, (i + 1) * 3000)
            args = [tr[k][sl] for k in ("arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class")]
            pt = W.make_point(2, 6, n_classes=3, backlog_mode="proxy", tau_pre_scale=scale, tau_dec_scale=scale)
            pt["pre_base_s"] = W.f32(pt["pre_base_s"] * scale)
            a, _ = O.sim_replica(pt, *args)
            _, st = O.sim_replica(W.make_point(2, 6, n_classes=3, policy="least_loaded"), *args,
                                  follow_pre=a["i_pre"], follow_dec=a["i_dec"])
            same += 3000 - st["mismatch_dec"]
        agree.append(same)
    assert agree[0] < agree[1] < agree[2] < agree[3] == 12000


def _maxplus_departures(arrive, service):
    """Single FIFO server: d_r = C_r + max_{j<=r}(a_j - C_{j-1}), C = prefix
    sums of service times (the max-plus solution of d_r = max(a_r, d_{r-1}) + s_r
    with d_{-1} = -inf)."""
    c = np.cumsum(service)
    c_prev = np.concatenate(([0], c[:-1]))
    return c + np.maximum.accumulate(arrive - c_prev)


@pytest.mark.parametrize("policy", ["learned", "round_robin", "least_loaded"])
def test_tandem_single_servers_max_plus(policy):
    rng = np.random.default_rng(21)
    tr = _trace(5000, rng, rate=30.0)  # heavily loaded: long busy periods
    pt = W.make_point(1, 1, policy=policy)
    out, st = _run(pt, tr)
    arr, p, o = tr[0], tr[1].astype(np.int64), tr[2].astype(np.int64)
    s_pre = pt["pre_base_ns"] + p * pt["pre_tok_ns"]
    pf_end = _maxplus_departures(arr, s_pre)
    kv_at = pf_end + p * pt["xfer_tok_ns"]
    dec_end = _maxplus_departures(kv_at, (o - 1) * pt["dec_tok_ns"])
    assert np.array_equal(out["ttft_ns"], pf_end - arr)
    assert np.array_equal(out["decode_span_ns"], dec_end - pf_end)
    assert st["max_queue_dec"] > 50  # the case exercises deep queues


def test_pollaczek_khinchine_mean_wait():
    """M/G/1 prefill: mean wait = lambda E[S^2] / (2 (1 - rho))."""
    rng = np.random.default_rng(99)
    n = 400_000
    lam = 60.0  # req/s
    p = rng.integers(16, 1200, n).astype(np.int32)
    arr = np.cumsum(rng.exponential(1.0 / lam, n) * 1e9).astype(np.int64)
    o = np.ones(n, np.int32)
    pt = W.make_point(1, 1, policy="round_robin")
    out, _ = O.sim_replica(pt, arr, p, o, o, np.zeros(n, np.uint8))
    s = (pt["pre_base_ns"] + p.astype(np.float64) * pt["pre_tok_ns"]) * 1e-9
    wait = out["ttft_ns"] * 1e-9 - s
    # service distribution is known exactly: p uniform on [16, 1199]
    pv = np.arange(16, 1200, dtype=np.float64)
    sv = (pt["pre_base_ns"] + pv * pt["pre_tok_ns"]) * 1e-9
    es, es2 = sv.mean(), (sv ** 2).mean()
    rho = lam * es
    expect = lam * es2 / (2 * (1 - rho))
    # batch means for a confidence interval on the correlated waits
    nb = 40
    bm = wait[: n // nb * nb].reshape(nb, -1).mean(axis=1)
    half = 2.7 * bm.std(ddof=1) / math.sqrt(nb)  # ~99 % two-sided
    assert abs(wait.mean() - expect) < half + 1e-4, (wait.mean(), expect, half)


def test_event_heap_bruteforce_agrees():
    """Independent event-driven simulation on random tiny traces with
    frequent timestamp ties (arrivals and service times on a coarse grid)."""
    rng = np.random.default_rng(2024)
    for case in range(2000):
        P, D = (int(x) for x in rng.integers(1, 4, size=2))
        n = int(rng.integers(1, 17))
        pol = ("learned", "round_robin", "least_loaded", "learned_sampled", "length_threshold")[case % 5]
        mode = ("true", "proxy")[(case // 5) % 2]
        pt = W.make_point(P, D, n_classes=3, policy=pol, backlog_mode=mode,
                          physics=dict(pre_base_ns=int(rng.integers(0, 3)) * 10,
                                       pre_tok_ns=int(rng.integers(0, 3)) * 10,
                                       dec_tok_ns=int(rng.integers(0, 4)) * 10, kv_bytes_per_token=2048),
                          kv_cap=int(rng.integers(1, 50)), w_q=float(rng.choice([0.0, 1e-3, 1.0])),
                          rho=float(rng.choice([0.0, 1.0, 3.0])), w_b=float(rng.choice([0.0, 1.0, 1e7])),
                          len_threshold=int(rng.integers(1, 6)))
        pt["xfer_tok_ns"] = int(rng.integers(0, 3)) * 10
        arr = np.sort(rng.integers(0, 8, n) * 10).astype(np.int64)
        p = rng.integers(1, 5, n).astype(np.int32)
        o = rng.integers(1, 5, n).astype(np.int32)
        oh = rng.integers(1, 5, n).astype(np.int32)
        c = rng.integers(0, 3, n).astype(np.uint8)
        words = rng.integers(0, 1 << 32, size=(n, 4), dtype=np.uint64).astype(np.uint32)
        ref = H.simulate(pt, arr, p, o, oh, c, words)
        got, st = O.sim_replica(pt, arr, p, o, oh, c, sample_bits=words)
        for k in ref:
            assert np.array_equal(ref[k], got[k]), (case, k, ref[k], got[k])
        assert st["violations"] == 0


def _recompute_state(pt, tr, out, r):
    """State every instance had when request r arrived, rebuilt from the
    recorded trajectory by brute force (in flight = admitted before r with a
    release time after arrival[r])."""
    arr, p, o, oh, c = tr
    now = arr[r]
    pf_end = arr[:r] + out["ttft_ns"][:r]
    dec_end = pf_end + out["decode_span_ns"][:r]
    res = {}
    for pool, n, idx, rel, fp, pend in (
            ("prefill", pt["n_prefill"], out["i_pre"][:r], pf_end, p[:r].astype(np.int64), p[:r].astype(np.int64)),
            ("decode", pt["n_decode"], out["i_dec"][:r], dec_end, p[:r].astype(np.int64) + o[:r],
             oh[:r].astype(np.int64))):
        live = rel > now
        q = np.array([np.sum(live & (idx == j)) for j in range(n)], np.int64)
        kv = np.array([np.sum(fp[live & (idx == j)]) for j in range(n)], np.int64)
        pd = np.array([np.sum(pend[live & (idx == j)]) for j in range(n)], np.int64)
        busy = np.array([rel[idx == j].max() if np.any(idx == j) else 0 for j in range(n)], np.int64)
        res[pool] = (q, kv, pd, busy)
    return res


@pytest.mark.parametrize("mode", ["true", "proxy"])
def test_decisions_recomputed_from_trajectory(mode):
    """Every learned decision is the argmin of costs recomputed in numpy
    float32 from a state rebuilt by brute force."""
    rng = np.random.default_rng(5 if mode == "true" else 6)
    tr = _trace(600, rng, rate=12.0, n_classes=3)
    pt = W.make_point(3, 5, n_classes=3, backlog_mode=mode, kv_cap=20_000)
    out, _ = _run(pt, tr)
    F = np.float32
    arr, p, o, oh, c = tr
    for r in range(600):
        st = _recompute_state(pt, tr, out, r)
        sg = F(pt["sigma"][c[r]])
        for pool, chosen in (("prefill", out["i_pre"][r]), ("decode", out["i_dec"][r])):
            q, kv, pd, busy = st[pool]
            if pool == "prefill":
                work = F(pt["w_s"]) * F(p[r]) * F(pt["tau_pre_s"])
                k = int(p[r])
                inv = F(1) / F(pt["kv_cap_pre"])
            else:
                work = F(pt["w_s"]) * F(oh[r]) * F(pt["tau_dec_s"])
                k = int(p[r]) + int(oh[r])
                inv = F(1) / F(pt["kv_cap_dec"])
            costs = []
            for j in range(len(q)):
                if mode == "true":
                    bl = F(max(int(busy[j]) - int(arr[r]), 0)) * F(1e-9)
                elif pool == "prefill":
                    bl = F(pt["tau_pre_s"]) * F(pd[j]) + F(pt["pre_base_s"]) * F(q[j])
                else:
                    bl = F(pt["tau_dec_s"]) * F(pd[j])
                press = F(int(kv[j]) + k) * inv
                cost = F(pt["w_b"]) * bl * sg + work * (F(1) + F(pt["rho"]) * press) * sg + F(pt["w_q"]) * F(q[j])
                costs.append(cost)
            assert chosen == int(np.argmin(np.array(costs, np.float32))), (r, pool, costs)


def test_conservation_and_fifo():
    wl = W.paper_cluster(n_replicas=2, requests=10_000)
    tr = W.make_trace(wl, workers=1)
    pt = wl.points[0]
    args = [tr[k][:10_000] for k in ("arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class")]
    out, st = O.sim_replica(pt, *args)
    arr, p, o = args[0], args[1].astype(np.int64), args[2].astype(np.int64)
    assert st["violations"] == 0 and st["invalid"] == 0
    # each request leaves each pool once: pops before the last arrival plus
    # what is still in flight equals the number admitted
    assert st["retired_pre"] + st["end_inflight_pre"] == 10_000
    assert st["retired_dec"] + st["end_inflight_dec"] == 10_000
    pf_end = arr + out["ttft_ns"]
    dec_end = pf_end + out["decode_span_ns"]
    s_pre = pt["pre_base_ns"] + p * pt["pre_tok_ns"]
    s_dec = (o - 1) * pt["dec_tok_ns"]
    assert np.all(out["ttft_ns"] >= s_pre)
    assert np.all(out["decode_span_ns"] >= p * pt["xfer_tok_ns"] + s_dec)
    for pool, idx, end, s in (("pre", out["i_pre"], pf_end, s_pre), ("dec", out["i_dec"], dec_end, s_dec)):
        for j in range(pt["n_prefill"] if pool == "pre" else pt["n_decode"]):
            m = idx == j
            e = end[m]
            assert np.all(np.diff(e) >= 0)  # FIFO: releases in admission order
            # serial service: consecutive services never overlap
            assert np.all(e[1:] - s[m][1:] >= e[:-1])


def test_invalid_requests_are_skipped_without_side_effects():
    """A rejected request (length < 1, class out of range, arrival before the
    previous accepted one) is not routed, leaves no state behind and is
    reported with -1 outputs."""
    rng = np.random.default_rng(8)
    arr, p, o, oh, c = _trace(400, rng, n_classes=2)
    pt = W.make_point(2, 3, n_classes=2)
    good, _ = O.sim_replica(pt, arr, p, o, oh, c)
    bad_after = {3: "p0", 50: "o0", 51: "oh0", 120: "big", 200: "class", 399: "early"}
    A, Pp, Oo, OH, CC = [], [], [], [], []
    for r in range(400):
        A.append(arr[r]); Pp.append(p[r]); Oo.append(o[r]); OH.append(oh[r]); CC.append(c[r])
        kind = bad_after.get(r)
        if kind is None:
            continue
        a, pp, oo, ohh, cc = arr[r], 5, 5, 5, 0
        if kind == "p0": pp = 0
        if kind == "o0": oo = 0
        if kind == "oh0": ohh = 0
        if kind == "class": cc = 2
        if kind == "early": a = arr[r] - 1
        if kind == "big": pp, oo = 2 ** 30, 2 ** 30  # token total 2^31 does not fit int32
        A.append(a); Pp.append(pp); Oo.append(oo); OH.append(ohh); CC.append(cc)
    out, st = O.sim_replica(pt, np.array(A, np.int64), np.array(Pp, np.int32), np.array(Oo, np.int32),
                            np.array(OH, np.int32), np.array(CC, np.uint8))
    assert st["invalid"] == 6
    bad = out["ttft_ns"] < 0
    assert bad.sum() == 6
    for k in out:
        assert np.all(out[k][bad] == -1)
        assert np.array_equal(out[k][~bad], good[k])


def test_follow_mode_accounting():
    wl = W.paper_cluster(n_replicas=1, requests=3000)
    tr = W.make_trace(wl, workers=1)
    pt = wl.points[0]
    args = [tr[k] for k in ("arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class")]
    own, st0 = O.sim_replica(pt, *args)
    # following its own choices: no divergence at all
    same, st = O.sim_replica(pt, *args, follow_pre=own["i_pre"], follow_dec=own["i_dec"])
    assert st["mismatch_pre"] == st["mismatch_dec"] == st["near_tie_pre"] == st["near_tie_dec"] == 0
    for k in own:
        assert np.array_equal(own[k], same[k])
    # plant a wrong decode placement at a decision that is not a tie
    fd = own["i_dec"].copy()
    r = 1234
    fd[r] = (fd[r] + 1) % pt["n_decode"]
    _, st = O.sim_replica(pt, *args, follow_pre=own["i_pre"], follow_dec=fd)
    assert st["mismatch_dec"] + st["near_tie_dec"] >= 1
    assert st["first_mismatch"] == r or st["near_tie_dec"] >= 1
    # an exact tie is accepted either way: identical simultaneous requests on
    # an empty pool tie on every prefill instance
    n = 2
    z = (np.zeros(n, np.int64), np.full(n, 10, np.int32), np.full(n, 2, np.int32), np.full(n, 2, np.int32),
         np.zeros(n, np.uint8))
    pt2 = W.make_point(2, 2)
    _, st = O.sim_replica(pt2, *z, follow_pre=np.array([1, 0], np.int32), follow_dec=np.array([0, 1], np.int32))
    assert st["near_tie_pre"] == 1 and st["mismatch_pre"] == 0
    # round-robin has no tolerance
    pt3 = W.make_point(2, 2, policy="round_robin")
    _, st = O.sim_replica(pt3, *z, follow_pre=np.array([1, 0], np.int32), follow_dec=np.array([0, 1], np.int32))
    assert st["mismatch_pre"] == 2


def test_goodput_hand_example():
    pt = W.make_point(1, 1, n_classes=2)
    tt0, tp0 = pt["slo_ttft_ns"][0], pt["slo_tpot_ns"][0]
    o = np.array([1, 5, 5, 5, 5, 3], np.int32)
    c = np.array([0, 0, 0, 1, 1, 0], np.uint8)
    ttft = np.array([tt0, tt0, tt0 + 1, 3 * tt0, 3 * tt0 + 1, -1], np.int64)
    span = np.array([10 ** 12, 4 * tp0, 4 * tp0, 4 * 3 * tp0, 0, 0], np.int64)
    g, met = O.goodput(pt, o, c, ttft, span)
    # r0 one-token answer: TPOT not applicable -> met; r1 met at both limits;
    # r2 TTFT 1 ns late; r3 class-1 loose limits exactly met; r4 TTFT late;
    # r5 rejected request
    assert met == 3 and g == 0.5
    span[1] += 1
    assert O.goodput(pt, o, c, ttft, span)[1] == 2
    assert O.goodput(pt, o[:0], c[:0], ttft[:0], span[:0]) == (0.0, 0)
