"""The seeded input generator: determinism, shapes and the paper's constants."""
import json
import os

import numpy as np
import pytest

from paper_2609_16206_amd import workload as W

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")))


def test_replica_regeneration_is_independent_of_batch():
    wl = W.paper_cluster(n_replicas=12, requests=500)
    full = W.make_trace(wl, workers=1)
    part = W.make_trace(wl, replicas=[7, 3], workers=1)
    for k in ("arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class"):
        assert np.array_equal(part[k][:500], full[k][7 * 500:8 * 500])
        assert np.array_equal(part[k][500:], full[k][3 * 500:4 * 500])


def test_parallel_generation_matches_serial():
    wl = W.paper_cluster(n_replicas=256, requests=8000)
    a = W.make_trace(wl, workers=1)
    b = W.make_trace(wl, workers=4)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def test_trace_shapes_and_ranges():
    wl = W.tiny_sim()
    tr = W.make_trace(wl)
    assert tr["arrival_ns"].dtype == np.int64 and tr["prompt_len"].dtype == np.int32
    assert tr["slo_class"].dtype == np.uint8 and tr["offsets"].tolist() == [0, 2000]
    assert np.all(np.diff(tr["arrival_ns"]) >= 0) and tr["arrival_ns"][0] > 0
    assert tr["prompt_len"].min() >= 16 and tr["prompt_len"].max() <= 8192
    assert tr["out_len"].min() >= 1 and tr["out_len"].max() <= 4096
    assert tr["pred_out_len"].min() >= 1
    # mean rate 4 req/s
    rate = 2000 / (tr["arrival_ns"][-1] * 1e-9)
    assert 3.6 < rate < 4.4
    # predicted / true is lognormal(0, 0.3)
    lr = np.log(tr["pred_out_len"][tr["out_len"] > 50] / tr["out_len"][tr["out_len"] > 50])
    assert abs(lr.mean()) < 0.03 and 0.27 < lr.std() < 0.33


def test_mmpp_mean_rate_and_burstiness():
    wl = W.paper_cluster(n_replicas=16, requests=10_000)
    tr = W.make_trace(wl, workers=1)
    rates = []
    for i in range(16):
        a = tr["arrival_ns"][i * 10_000:(i + 1) * 10_000] * 1e-9
        rates.append(10_000 / a[-1])
        gaps = np.diff(a)
        # index of dispersion of counts in 5 s windows is > 1 for an MMPP
        counts = np.bincount((a // 5.0).astype(int))
        assert counts.var() / counts.mean() > 2.0
    assert 6.5 < np.mean(rates) < 8.5  # equal dwell: mean of 3 and 12 req/s


def test_sweep_points_layout():
    pts, trafs = W.sweep_points()
    assert len(pts) == 1225
    widths = sorted({p["n_decode"] for p in pts})
    assert widths == list(W.SWEEP_WIDTHS)
    assert all(p["n_prefill"] == 2 and p["backlog_mode"] == "proxy" for p in pts)
    # load factor: mean rate / capacity equals the point's load
    for i in (0, 177, 600, 1224):
        w, ld = W.SWEEP_WIDTHS[i // 175], W.SWEEP_LOADS[(i // 25) % 7]
        cap = W.capacity_rps(pts[i], trafs[i])
        assert trafs[i].mean_rate() / cap == pytest.approx(ld, rel=1e-12)
        sp, sd = W.SWEEP_SCALES[(i % 25) // 5], W.SWEEP_SCALES[i % 5]
        assert pts[i]["tau_dec_s"] == W.f32(1.8e-3 * sd)
        assert pts[i]["tau_pre_s"] == W.f32(1e-5 * sp)


def test_paper_constants_and_slo_reading():
    a40, sim = GOLD["decode_s_per_token"]["a40"], GOLD["decode_s_per_token"]["simulator"]
    assert round(a40 / sim, 1) == GOLD["decode_ratio_printed"]  # "7.4x"
    assert W.A40_PHYSICS["dec_tok_ns"] == round(a40 * 1e9)
    assert W.SIM_PHYSICS["dec_tok_ns"] == round(sim * 1e9)
    assert W.A40_PHYSICS["pre_base_ns"] == round(GOLD["prefill_base_s"]["a40"] * 1e9)
    assert W.SIM_PHYSICS["pre_base_ns"] == round(GOLD["prefill_base_s"]["simulator"] * 1e9)
    assert W.A40_PHYSICS["kv_bytes_per_token"] == GOLD["kv_bytes_per_token"]["a40"]
    assert W.SIM_PHYSICS["kv_bytes_per_token"] == GOLD["kv_bytes_per_token"]["simulator"]
    # the SLO reading reproduces the printed tight targets on A40 constants
    ttft, tpot = W.slo_targets(W.A40_PHYSICS["dec_tok_ns"], 2)
    assert tpot[0] * 1e-9 == pytest.approx(GOLD["slo_tight"]["tpot_s"], rel=2e-3)
    assert ttft[0] * 1e-9 == pytest.approx(GOLD["slo_tight"]["ttft_s"], rel=2e-3)
    assert ttft[1] == GOLD["slo_loose_factor"] * ttft[0] and tpot[1] == GOLD["slo_loose_factor"] * tpot[0]


def test_large_pool_rate_and_pareto_mean():
    wl = W.large_pool_wl(n_replicas=1, requests=200_000)
    tr = W.make_trace(wl)
    o = tr["out_len"].astype(np.float64)
    pa = wl.traffic[0].output[0]
    assert o.max() <= 32768 and o.min() >= 100
    assert o.mean() == pytest.approx(pa.clipped_mean(), rel=0.05)
    rate = 200_000 / (tr["arrival_ns"][-1] * 1e-9)
    assert rate == pytest.approx(wl.meta["rate"], rel=0.02)
    assert wl.meta["rate"] == pytest.approx(0.95 * W.capacity_rps(wl.points[0], wl.traffic[0]))


def test_scorer_inputs():
    d = W.scorer_inputs(n_req=1000, n_inst=64)
    assert d["queue"].shape == (64,) and d["queue"].max() <= 256
    assert d["kv_occ"].max() < 200_000 and d["backlog_s"].max() < 10
    d2 = W.scorer_inputs(n_req=100, n_inst=8, per_request=True)
    assert d2["queue"].shape == (800,) and d2["inst_stride"] == 8
