"""Replica simulation on the GPU vs the oracle (Algorithm 1 on the
serial-service simulator): the tiny 3P+3D workload in full under every policy
and backlog mode, the paper-shaped 2P+6D cluster (4,096 x 10,000) in full, and
edge cases: ragged and empty replicas, rejected requests, simultaneous
arrivals, mixed pool shapes in one batch (every kernel class), determinism and
replica-range resume."""
import numpy as np
import pytest

from paper_2609_16206_amd import rt_router as R
from paper_2609_16206_amd import workload as W
from tests.gpu_common import log, run_sim
from tests.parity import check_properties, follow_replicas, goodput_recount

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("policy,mode", [("learned", "true"), ("learned", "proxy"), ("round_robin", "true"),
                                         ("least_loaded", "true")])
def test_tiny_full(policy, mode):
    wl = W.tiny_sim()
    pts = [dict(wl.points[0], policy=policy, backlog_mode=mode)]
    tr = W.make_trace(wl)
    gpu, g, met, flags = run_sim(pts, tr)
    assert flags == 0
    rep = follow_replicas(pts, tr, gpu, [0], gpu_goodput=g, gpu_met=met)
    log(f"tiny {policy}/{mode}: {rep}, goodput {g[0]:.4f}")
    if policy == "round_robin":
        r = np.arange(2000)
        assert np.array_equal(gpu["i_pre"], r % 3) and np.array_equal(gpu["i_dec"], r % 3)


def test_cluster_full_size():
    wl = W.paper_cluster()
    tr = W.make_trace(wl)
    log(f"cluster trace: {tr['arrival_ns'].size} requests")
    gpu, g, met, flags = run_sim(wl.points, tr)
    assert flags == 0
    check_properties(wl.points, tr, gpu)
    assert np.array_equal(goodput_recount(wl.points, tr, gpu), met)
    rep = follow_replicas(wl.points, tr, gpu, range(wl.n_replicas), gpu_goodput=g, gpu_met=met)
    log(f"cluster 4096x10000: {rep}; mean goodput {g.mean():.4f}")


def _mixed_points():
    """Pool shapes that exercise every kernel class, with all policies/modes."""
    shapes = [(1, 1), (2, 2), (3, 4), (2, 6), (4, 9), (5, 16), (2, 32), (33, 64), (70, 100), (128, 1024),
              (1000, 300), (2, 64), (60, 70), (1, 63), (64, 64)]
    pts = []
    for k, (P, D) in enumerate(shapes):
        pol = ("learned", "learned", "round_robin", "least_loaded")[k % 4]
        mode = ("true", "proxy")[(k // 2) % 2]
        pts.append(W.make_point(P, D, n_classes=3, policy=pol, backlog_mode=mode, kv_cap=50_000))
    return pts


def _ragged_trace(pts, lengths, seed=7, rate_scale=1.0):
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
    return tr


def test_mixed_shapes_ragged_lengths():
    pts = _mixed_points()
    lengths = [0, 1, 2, 63, 64, 65, 500, 3000, 1, 0, 777, 4096, 129, 2, 3, 5000, 40, 41, 0, 1200] * 3
    tr = _ragged_trace(pts, lengths)
    gpu, g, met, flags = run_sim(pts, tr)
    assert flags == 0
    check_properties(pts, tr, gpu)
    assert np.array_equal(goodput_recount(pts, tr, gpu), met)
    rep = follow_replicas(pts, tr, gpu, range(len(lengths)), gpu_goodput=g, gpu_met=met)
    log(f"mixed shapes: {rep}")
    assert np.all(g[np.array(lengths) == 0] == 0.0)


def test_pools_at_the_limit():
    """Pools of RT_MAX_POOL instances, and lopsided ones, in every scoring
    mode: each takes a multi-wave class."""
    shapes = [(1024, 1024), (1024, 1), (1, 1024), (1024, 700), (513, 1024), (900, 901)]
    pts = []
    for k, (P, D) in enumerate(shapes):
        pol = ("learned", "learned", "round_robin")[k % 3]
        mode = ("true", "proxy")[k % 2]
        pts.append(W.make_point(P, D, n_classes=3, policy=pol, backlog_mode=mode, kv_cap=50_000))
    lengths = [3000, 1, 2000, 0, 2500, 1500, 65, 4000, 700, 3]
    tr = _ragged_trace(pts, lengths, seed=17, rate_scale=1.5)
    gpu, g, met, flags = run_sim(pts, tr)
    assert flags == 0
    check_properties(pts, tr, gpu)
    rep = follow_replicas(pts, tr, gpu, range(len(lengths)), gpu_goodput=g, gpu_met=met)
    log(f"pools at the limit: {rep}")


def test_sampled_policy_mixed_with_learned():
    """The two-candidate policy in both scoring modes, on one-wave and
    multi-wave pool shapes, in one batch with full-argmin points (so each
    point's kernel class is picked by its mode); follow-mode parity."""
    shapes = [(1, 2), (2, 6), (3, 9), (5, 16), (2, 33), (33, 64), (70, 100), (128, 300)]
    pts = []
    for k, (P, D) in enumerate(shapes):
        mode = ("true", "proxy")[k % 2]
        pts.append(W.make_point(P, D, n_classes=3, policy="learned_sampled", backlog_mode=mode, kv_cap=50_000))
        pts.append(W.make_point(P, D, n_classes=3, policy="learned", backlog_mode=mode, kv_cap=50_000))
    lengths = [1500, 3, 700, 2000, 64, 65, 1, 999] * 4
    tr = _ragged_trace(pts, lengths, seed=23, rate_scale=1.3)
    W.add_sample_words(tr, 23)
    gpu, g, met, flags = run_sim(pts, tr)
    assert flags == 0
    check_properties(pts, tr, gpu)
    rep = follow_replicas(pts, tr, gpu, range(len(lengths)), gpu_goodput=g, gpu_met=met)
    log(f"sampled policy: {rep}")
    # every sampled placement is one of its request's two candidates
    from oracle import oracle as O
    off = tr["offsets"]
    for i in range(0, len(lengths), 2):
        P, D = pts[i % len(pts)]["n_prefill"], pts[i % len(pts)]["n_decode"]
        for r in range(int(off[i]), min(int(off[i + 1]), int(off[i]) + 50)):
            w = tr["sample_bits"][r]
            assert gpu["i_pre"][r] in O.candidates(w[0], w[1], P)
            assert gpu["i_dec"][r] in O.candidates(w[2], w[3], D)


def test_length_threshold_policy():
    """The length-threshold baseline on one-wave and multi-wave shapes, with
    thresholds that split the mixed traffic; follow-mode parity (exact:
    the policy has no floating point) and the part each request used."""
    shapes = [(1, 1), (2, 2), (2, 6), (3, 9), (5, 16), (33, 64), (70, 100), (128, 300)]
    pts = [W.make_point(P, D, n_classes=3, policy="length_threshold", len_threshold=(64, 256, 1000)[k % 3])
           for k, (P, D) in enumerate(shapes)]
    lengths = [1500, 3, 700, 2000, 64, 65, 1, 999] * 2
    tr = _ragged_trace(pts, lengths, seed=31, rate_scale=1.2)
    gpu, g, met, flags = run_sim(pts, tr)
    assert flags == 0
    check_properties(pts, tr, gpu)
    rep = follow_replicas(pts, tr, gpu, range(len(lengths)), gpu_goodput=g, gpu_met=met)
    log(f"length threshold: {rep}")
    assert rep["near_ties"] == 0
    off = tr["offsets"]
    for i in range(len(lengths)):
        pt = pts[i % len(pts)]
        D, thr = pt["n_decode"], pt["len_threshold"]
        sl = slice(int(off[i]), int(off[i + 1]))
        if D > 1:
            lng = tr["pred_out_len"][sl] >= thr
            assert np.all((gpu["i_dec"][sl] >= (D + 1) // 2) == lng)


def test_sampled_policy_requires_words():
    pts = [W.make_point(2, 6, policy="learned_sampled")]
    tr = _ragged_trace(pts, [10], seed=1)
    with pytest.raises(R.RtError):
        run_sim(pts, tr)


def test_overload_deep_queues():
    """Arrivals at 3x capacity: long FIFOs, many pops per step."""
    pts = [W.make_point(2, 3, n_classes=3), W.make_point(2, 6, n_classes=3, backlog_mode="proxy"),
           W.make_point(3, 40, n_classes=3, policy="least_loaded")]
    tr = _ragged_trace(pts, [4000] * 12, seed=11, rate_scale=3.0)
    gpu, g, met, flags = run_sim(pts, tr)
    rep = follow_replicas(pts, tr, gpu, range(12), gpu_goodput=g, gpu_met=met)
    log(f"overload: {rep}")


def test_simultaneous_arrivals_and_rejections():
    pts = [W.make_point(3, 5, n_classes=2), W.make_point(2, 2, n_classes=2, policy="round_robin")]
    rng = np.random.default_rng(3)
    n = 3000
    lengths = [n, n, n, n]
    tr = _ragged_trace(pts, lengths, seed=21)
    # coarse arrival grid: many equal timestamps
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
    log(f"ties+rejections: {rep}")
    assert rep["invalid"] == int((gpu["ttft_ns"] < 0).sum())


def test_many_replicas_packed_classes():
    """Enough replicas that the planner packs several instances per lane (the
    throughput classes), for every scoring mode and a spread of pool shapes."""
    shapes = [(1, 2), (2, 3), (2, 6), (3, 9), (2, 16), (4, 30), (2, 64), (5, 50)]
    modes = [("learned", "true"), ("learned", "proxy"), ("round_robin", "true"), ("least_loaded", "true")]
    pts = [W.make_point(P, D, n_classes=3, policy=pol, backlog_mode=bm, kv_cap=20_000)
           for (P, D) in shapes for (pol, bm) in modes]
    n_rep, n_req = 24576, 48
    lengths = [n_req - (i % 7) for i in range(n_rep)]
    tr = _ragged_trace(pts, lengths, seed=31, rate_scale=1.1)
    log(f"packed classes: {len(pts)} points, {n_rep} replicas, {tr['arrival_ns'].size} requests")
    gpu, g, met, flags = run_sim(pts, tr)
    assert flags == 0
    check_properties(pts, tr, gpu)
    assert np.array_equal(goodput_recount(pts, tr, gpu), met)
    rep = follow_replicas(pts, tr, gpu, range(n_rep), gpu_goodput=g, gpu_met=met)
    log(f"packed classes: {rep}")


def test_determinism_and_range_resume():
    wl = W.paper_cluster(n_replicas=300, requests=3000)
    tr = W.make_trace(wl)
    a, ga, _, _ = run_sim(wl.points, tr)
    b, gb, _, _ = run_sim(wl.points, tr)
    for k in a:
        assert np.array_equal(a[k], b[k]), k
    assert np.array_equal(ga, gb)
    # replicas [117, 211) alone, as their own batch
    sub = W.make_trace(wl, replicas=range(117, 211))
    c, gc, _, _ = run_sim(wl.points, sub)
    s = slice(117 * 3000, 211 * 3000)
    for k in a:
        assert np.array_equal(a[k][s], c[k]), k
    assert np.array_equal(ga[117:211], gc)


def test_coarse_grid_ties_many_small_replicas():
    """Hundreds of small replicas on a coarse time grid with tiny integer
    physics and transfers of zero (simultaneous arrivals, releases exactly at
    an arrival, equal costs), every policy and backlog mode: every replica
    is checked against the oracle."""
    rng = np.random.default_rng(92)
    pols = [("learned", "true"), ("learned", "proxy"), ("round_robin", "true"), ("least_loaded", "true"),
            ("learned_sampled", "true"), ("learned_sampled", "proxy"), ("length_threshold", "true")]
    pts = []
    for k in range(14):
        pol, mode = pols[k % len(pols)]
        pt = W.make_point(int(rng.integers(1, 4)), int(rng.integers(1, 4)), n_classes=2, policy=pol,
                          backlog_mode=mode, len_threshold=3)
        pt.update(pre_base_ns=int(rng.choice([0, 4])), pre_tok_ns=int(rng.choice([1, 2])),
                  dec_tok_ns=int(rng.choice([1, 3])), xfer_tok_ns=int(rng.choice([0, 1])))
        pts.append(pt)
    n_rep = 480
    lengths = rng.integers(1, 41, n_rep)
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
    W.add_sample_words(tr, 92)
    gpu, g, met, flags = run_sim(pts, tr)
    assert flags == 0
    rep = follow_replicas(pts, tr, gpu, range(n_rep), gpu_goodput=g, gpu_met=met)
    log(f"serial coarse grid: {rep}")


@pytest.mark.parametrize("P,D,n_rep", [(1, 1, 32768), (1, 2, 16384), (1, 1, 8192), (2, 6, 4096), (8, 8, 2048),
                                       (16, 16, 1024)])
def test_outcome_blocks_every_residue(P, D, n_rep):
    """The one-wave kernels write outcomes in blocks of S steps (lane k of a
    segment keeps step block start + k).  Replica lengths cycle through
    1..130, so a replica's last block ends at every residue modulo the
    segment width; the replica counts are chosen so that the planner's
    widening stops at S = 2, 4, 8, 16, 32 and 64 in turn (one wave per SIMD)."""
    pts = [W.make_point(P, D, n_classes=3, kv_cap=50_000)]
    lengths = [1 + (i % 130) for i in range(n_rep)]
    tr = _ragged_trace(pts, lengths, seed=23, rate_scale=1.2)
    gpu, g, met, flags = run_sim(pts, tr)
    assert flags == 0
    check_properties(pts, tr, gpu)
    assert np.array_equal(goodput_recount(pts, tr, gpu), met)
    rep = follow_replicas(pts, tr, gpu, range(n_rep), gpu_goodput=g, gpu_met=met)
    log(f"outcome blocks {P}P+{D}D x {n_rep}: {rep}")
