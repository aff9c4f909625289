"""The continuous-batching service model on the GPU vs the oracle: every
policy and backlog mode on the tiny 3P+3D workload, the paper-shaped 2P+6D
cluster (4,096 x 10,000) in full, ragged replicas of several pool shapes and
betas in one batch with serial points, simultaneous arrivals and rejected
requests, the ring-capacity flag, and determinism."""
import numpy as np
import pytest

from paper_2609_16206_amd import rt_router as R
from paper_2609_16206_amd import workload as W
from tests.gpu_common import log, run_sim
from tests.parity import check_properties, follow_replicas, goodput_recount

pytestmark = pytest.mark.gpu

POLICIES = [("learned", "true"), ("learned", "proxy"), ("round_robin", "true"), ("least_loaded", "true"),
            ("learned_sampled", "true"), ("learned_sampled", "proxy"), ("length_threshold", "true")]


def _batched(pt, beta_pre=None, beta_dec=None, **kw):
    return dict(pt, service="batched", beta_pre=W.BATCH_BETA if beta_pre is None else beta_pre,
                beta_dec=W.BATCH_BETA if beta_dec is None else beta_dec, **kw)


@pytest.mark.parametrize("policy,mode", POLICIES)
def test_tiny_full(policy, mode):
    wl = W.tiny_sim()
    pts = [_batched(wl.points[0], policy=policy, backlog_mode=mode, len_threshold=150)]
    tr = W.make_trace(wl)
    tr["arrival_ns"] = tr["arrival_ns"] // 4  # four times the load: batches form
    W.add_sample_words(tr, 5)
    gpu, g, met, flags = run_sim(pts, tr)
    assert flags == 0
    check_properties(pts, tr, gpu)
    rep = follow_replicas(pts, tr, gpu, [0], gpu_goodput=g, gpu_met=met)
    log(f"batched tiny {policy}/{mode}: {rep}, goodput {g[0]:.4f}")
    if policy == "round_robin":
        r = np.arange(2000)
        assert np.array_equal(gpu["i_pre"], r % 3) and np.array_equal(gpu["i_dec"], r % 3)


def test_cluster_full_size():
    wl = W.paper_cluster()
    pts = [_batched(wl.points[0])]
    tr = W.make_trace(wl)
    log(f"batched cluster trace: {tr['arrival_ns'].size} requests")
    gpu, g, met, flags = run_sim(pts, tr)
    assert flags == 0
    check_properties(pts, tr, gpu)
    assert np.array_equal(goodput_recount(pts, tr, gpu), met)
    rep = follow_replicas(pts, tr, gpu, range(wl.n_replicas), gpu_goodput=g, gpu_met=met)
    log(f"batched cluster 4096x10000: {rep}; mean goodput {g.mean():.4f}")


def _ragged(pts, lengths, seed, rate_scale=1.0):
    parts, pp = [], []
    tr0 = W.mixed_bursty()
    for i, n in enumerate(lengths):
        pid = i % len(pts)
        traf = tr0.scaled(rate_scale * W.capacity_rps(pts[pid], tr0) / tr0.mean_rate())
        parts.append(W.replica_arrays(seed, i, traf, n))
        pp.append(pid)
    keys = ("arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class")
    tr = {k: np.concatenate([q[k] for q in parts]) for k in keys}
    tr["offsets"] = np.concatenate(([0], np.cumsum(lengths))).astype(np.int64)
    tr["param_point"] = np.array(pp, np.int32)
    W.add_sample_words(tr, seed)
    return tr


def test_mixed_shapes_betas_and_serial_points():
    """Batched points of several pool shapes and betas (0: infinite server;
    1: pure processor sharing) next to serial points in one call, so both
    kernel kinds run side by side; ragged and empty replicas."""
    # segment widths 4, 8, 16, 32 and 64 (P + D = 64 exactly), two instances
    # per lane up to 128 instances, and beyond that the one-replica-per-lane
    # kernel
    shapes = [(1, 1), (2, 6), (3, 9), (5, 16), (8, 8), (33, 64), (2, 2), (4, 12), (32, 32), (20, 44), (40, 100)]
    betas = [(0.0, 0.0), (W.BATCH_BETA, W.BATCH_BETA), (1.0, 0.25), (0.5, 1.0)]
    pts = []
    for k, (P, D) in enumerate(shapes):
        pol, mode = POLICIES[k % len(POLICIES)]
        bp, bd = betas[k % len(betas)]
        base = W.make_point(P, D, n_classes=3, policy=pol, backlog_mode=mode, kv_cap=50_000, len_threshold=200)
        # beta = 1 at twice the serial capacity is an overloaded processor-
        # sharing queue: its batches grow with the trace, hence the room
        pts.append(_batched(base, bp, bd, batch_cap=4096))
        pts.append(base)  # serial
    lengths = [1500, 3, 700, 0, 64, 65, 1, 999, 2000, 257, 0, 40, 129, 2, 1200, 300] * 2
    tr = _ragged(pts, lengths, seed=17, rate_scale=2.0)
    gpu, g, met, flags = run_sim(pts, tr)
    assert flags == 0
    check_properties(pts, tr, gpu)
    assert np.array_equal(goodput_recount(pts, tr, gpu), met)
    rep = follow_replicas(pts, tr, gpu, range(len(lengths)), gpu_goodput=g, gpu_met=met)
    log(f"batched mixed: {rep}")
    assert np.all(g[np.array(lengths) == 0] == 0.0)


def test_simultaneous_arrivals_and_rejections():
    pts = [_batched(W.make_point(3, 5, n_classes=2)),
           _batched(W.make_point(2, 2, n_classes=2, policy="least_loaded"), 1.0, 1.0)]
    rng = np.random.default_rng(3)
    n = 3000
    tr = _ragged(pts, [n] * 4, seed=21)
    tr["arrival_ns"] = (tr["arrival_ns"] // 500_000_000) * 500_000_000
    for i in range(4):
        s = slice(i * n, (i + 1) * n)
        tr["arrival_ns"][s] = np.sort(tr["arrival_ns"][s])
    bad = rng.choice(4 * n, 60, replace=False)
    kinds = np.arange(60) % 6
    tr["prompt_len"][bad[kinds == 0]] = 0
    tr["out_len"][bad[kinds == 1]] = 0
    tr["pred_out_len"][bad[kinds == 2]] = -3
    tr["slo_class"][bad[kinds == 3]] = 2
    tr["arrival_ns"][bad[kinds == 4]] = -1
    b5 = bad[kinds == 5]
    tr["prompt_len"][b5] = 2 ** 30
    tr["out_len"][b5] = 2 ** 30
    gpu, g, met, flags = run_sim(pts, tr)
    assert flags == 1
    assert (gpu["ttft_ns"] < 0).sum() >= 50
    rep = follow_replicas(pts, tr, gpu, range(4), gpu_goodput=g, gpu_met=met)
    log(f"batched ties+rejections: {rep}")


def test_ring_capacity_flag():
    """A batch_cap too small for the load sets flag bit 3; the replicas that
    fit are still exact."""
    wl = W.tiny_sim()
    small = _batched(wl.points[0], batch_cap=2)
    roomy = _batched(wl.points[0], batch_cap=4096)
    tr = W.make_trace(wl)
    tr["arrival_ns"] = tr["arrival_ns"] // 8
    gpu, _, _, flags = run_sim([small], tr)
    assert flags & 8
    gpu, g, met, flags = run_sim([roomy], tr)
    assert flags == 0
    follow_replicas([roomy], tr, gpu, [0], gpu_goodput=g, gpu_met=met)


def test_bad_points_rejected():
    base = W.make_point(2, 6)
    for bad in (dict(beta_dec=-1.0), dict(beta_pre=float("nan")), dict(batch_cap=3), dict(batch_cap=1 << 17),
                dict(batch_cap=1)):
        with pytest.raises(R.RtError):
            R.Simulator([_batched(base, **{k: v for k, v in bad.items() if k.startswith("beta")})
                         if "batch_cap" not in bad else _batched(base, batch_cap=bad["batch_cap"])])
    bad = dict(base, service=7)
    with pytest.raises(R.RtError):
        R.Simulator([bad])


def test_determinism_and_range_resume():
    wl = W.paper_cluster(n_replicas=300, requests=3000)
    pts = [_batched(wl.points[0])]
    tr = W.make_trace(wl)
    a, ga, _, _ = run_sim(pts, tr)
    b, gb, _, _ = run_sim(pts, tr)
    for k in a:
        assert np.array_equal(a[k], b[k]), k
    assert np.array_equal(ga, gb)
    sub = W.make_trace(wl, replicas=range(117, 211))
    c, gc, _, _ = run_sim(pts, sub)
    s = slice(117 * 3000, 211 * 3000)
    for k in a:
        assert np.array_equal(a[k][s], c[k]), k
    assert np.array_equal(ga[117:211], gc)


def test_wide_bench_workload_sampled():
    """The 65,536 x 2,000 batched bench workload in the launch configuration
    bench.py times: properties on every request, goodput recount on every
    replica, and follow-mode parity on a spread sample of replicas."""
    wl = W.paper_cluster(n_replicas=65536, requests=2000, service="batched")
    tr = W.make_trace(wl)
    gpu, g, met, flags = run_sim(wl.points, tr)
    assert flags == 0
    check_properties(wl.points, tr, gpu)
    assert np.array_equal(goodput_recount(wl.points, tr, gpu), met)
    sample = list(range(0, 65536, 1021)) + [65535]
    rep = follow_replicas(wl.points, tr, gpu, sample, gpu_goodput=g, gpu_met=met)
    log(f"batched 65536x2000: {rep}; mean goodput {g.mean():.4f}")


def test_wide_pool_bench_workload_sampled():
    """The batched bench workload whose pool (8 prefill + 64 decode) is too
    wide for one instance per lane, in the launch bench.py times (two
    instances per lane of a 64-lane segment): properties on every request, goodput recount on every replica,
    follow-mode parity on a spread sample of replicas."""
    wl = W.batched_wide_pool()
    tr = W.make_trace(wl)
    gpu, g, met, flags = run_sim(wl.points, tr)
    assert flags == 0
    check_properties(wl.points, tr, gpu)
    assert np.array_equal(goodput_recount(wl.points, tr, gpu), met)
    sample = list(range(0, wl.n_replicas, 1023)) + [wl.n_replicas - 1]
    rep = follow_replicas(wl.points, tr, gpu, sample, gpu_goodput=g, gpu_met=met)
    log(f"batched wide pool {wl.n_replicas}x{wl.requests}: {rep}; mean goodput {g.mean():.4f}")


def test_two_instances_per_lane_pools():
    """Pools of 65 to 128 instances, two per lane of a 64-lane segment: odd
    and even pool sizes on both sides (P = 65 with D = 1 as well as P = 2 with
    D = 126), every policy, several betas, ragged and empty replicas, each
    followed against the oracle."""
    shapes = [(33, 64), (5, 99), (64, 64), (65, 1), (2, 126), (9, 60), (17, 111)]
    betas = [(W.BATCH_BETA, W.BATCH_BETA), (0.0, 0.0), (1.0, 0.25), (0.5, 1.0)]
    pts = []
    for k, (P, D) in enumerate(shapes):
        pol, mode = POLICIES[k % len(POLICIES)]
        bp, bd = betas[k % len(betas)]
        base = W.make_point(P, D, n_classes=3, policy=pol, backlog_mode=mode, kv_cap=50_000, len_threshold=200)
        pts.append(_batched(base, bp, bd, batch_cap=4096))
    lengths = [900, 3, 1, 257, 0, 64, 1200, 129, 40, 700, 2, 300, 65, 0]
    tr = _ragged(pts, lengths, seed=23, rate_scale=2.0)
    gpu, g, met, flags = run_sim(pts, tr)
    assert flags == 0
    check_properties(pts, tr, gpu)
    assert np.array_equal(goodput_recount(pts, tr, gpu), met)
    rep = follow_replicas(pts, tr, gpu, range(len(lengths)), gpu_goodput=g, gpu_met=met)
    log(f"batched two per lane: {rep}")


def test_two_instances_per_lane_ring_capacity():
    """The ring-capacity flag and the stop of an overflowing replica with two
    instances per lane (a 9 + 91 pool): a batch_cap of 2 under eight times
    the load sets flag bit 3; with room, every replica is exact."""
    base = W.make_point(9, 91, n_classes=3)
    small = _batched(base, batch_cap=2)
    roomy = _batched(base, batch_cap=4096)
    lengths = [400, 1, 250, 0, 333]
    tr = _ragged([small], lengths, seed=29, rate_scale=8.0)
    gpu, _, _, flags = run_sim([small], tr)
    assert flags & 8
    tr = _ragged([roomy], lengths, seed=29, rate_scale=8.0)
    gpu, g, met, flags = run_sim([roomy], tr)
    assert flags == 0
    check_properties([roomy], tr, gpu)
    rep = follow_replicas([roomy], tr, gpu, range(len(lengths)), gpu_goodput=g, gpu_met=met)
    log(f"batched two per lane, ring capacity: {rep}")


def _coarse_grid(seed, pool_range, n_rep, max_len):
    """Replicas on a coarse time grid with tiny integer physics and transfers
    of zero: simultaneous arrivals, equal finish times within a batch,
    completions and KV landings at the same instant, zero decode work
    (o = 1)."""
    rng = np.random.default_rng(seed)
    pts = []
    for k in range(12):
        pol, mode = POLICIES[k % len(POLICIES)]
        pt = _batched(W.make_point(int(rng.integers(*pool_range)), int(rng.integers(*pool_range)), n_classes=2,
                                   policy=pol, backlog_mode=mode, len_threshold=3),
                      float(rng.choice([0.0, 0.125, 0.5, 1.0])), float(rng.choice([0.0, 0.25, 1.0])))
        pt.update(pre_base_ns=int(rng.choice([0, 4])), pre_tok_ns=int(rng.choice([1, 2])),
                  dec_tok_ns=int(rng.choice([1, 3])), xfer_tok_ns=int(rng.choice([0, 1])))
        pts.append(pt)
    lengths = rng.integers(1, max_len + 1, n_rep)
    parts = {k: [] for k in ("arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class")}
    for n in lengths:
        parts["arrival_ns"].append(np.sort(rng.integers(0, 12, n)).astype(np.int64) * 4)
        parts["prompt_len"].append(rng.integers(1, 5, n).astype(np.int32))
        parts["out_len"].append(rng.integers(1, 5, n).astype(np.int32))
        parts["pred_out_len"].append(rng.integers(1, 6, n).astype(np.int32))
        parts["slo_class"].append(rng.integers(0, 2, n).astype(np.uint8))
    tr = {k: np.concatenate(v) for k, v in parts.items()}
    tr["offsets"] = np.concatenate(([0], np.cumsum(lengths))).astype(np.int64)
    tr["param_point"] = (np.arange(n_rep) % len(pts)).astype(np.int32)
    W.add_sample_words(tr, seed)
    return pts, tr


def test_coarse_grid_ties_many_small_replicas():
    """Hundreds of small replicas (pools of 1 to 3 per side) on the coarse
    grid; every replica is checked against the oracle."""
    pts, tr = _coarse_grid(91, (1, 4), 480, 40)
    gpu, g, met, flags = run_sim(pts, tr)
    assert flags == 0
    rep = follow_replicas(pts, tr, gpu, range(480), gpu_goodput=g, gpu_met=met)
    log(f"batched coarse grid: {rep}")


def test_coarse_grid_ties_wide_pools():
    """The coarse grid on pools of 33 to 64 per side (66 to 128 instances, two
    per lane): ties between the two instances of one lane and between lanes;
    every replica is checked."""
    pts, tr = _coarse_grid(92, (33, 65), 96, 200)
    gpu, g, met, flags = run_sim(pts, tr)
    assert flags == 0
    rep = follow_replicas(pts, tr, gpu, range(96), gpu_goodput=g, gpu_met=met)
    log(f"batched coarse grid, wide pools: {rep}")
