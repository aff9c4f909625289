"""Experiment drivers on the GPU: batched policy grids on every workload
family of Table I (chat, document, reasoning, mixed bursty) agree with the
oracle replica by replica, and the saturation search (Section IV-B) probes
the same goodputs and finds the same scale as the same search run on the
oracle."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2609_16206_amd import experiments as E
from paper_2609_16206_amd import workload as W
from tests.gpu_common import log
from tests.parity import follow_replicas, oracle_run_cells

pytestmark = pytest.mark.gpu


def test_policy_grid_matches_oracle():
    traf = W.mixed_bursty().scaled(1.3)
    cells = E.policy_cells(2, 4, traf) + E.ablation_cells(2, 4, traf)[1:] + E.noise_cells(2, 4, traf, (0.0, 1.5))
    rows, tr, out, g = E.run_cells(cells, replicas=3, requests=1500, seed=4, return_trace=True)
    log("grid: " + ", ".join(f"{r['label']} {r['mean']:.3f}" for r in rows))
    ref = O.sim_trace([c.point for c in cells], tr, threads=16)
    for i, (o, st, gg, met) in ref.items():
        sl = slice(int(tr["offsets"][i]), int(tr["offsets"][i + 1]))
        assert np.array_equal(o["i_pre"], out["i_pre"][sl]) and np.array_equal(o["i_dec"], out["i_dec"][sl]), i
        assert np.array_equal(o["ttft_ns"], out["ttft_ns"][sl]) and np.array_equal(o["decode_span_ns"],
                                                                                   out["decode_span_ns"][sl]), i
        assert gg == g[i], i


FAMILIES = [("chat", W.chat(1.0)), ("document", W.document(1.0)), ("reasoning", W.reasoning(1.0)),
            ("mixed", W.mixed_bursty())]


@pytest.mark.parametrize("family,traffic", FAMILIES, ids=[f for f, _ in FAMILIES])
def test_table1_family_policy_grid_matches_oracle(family, traffic):
    """Every policy (learned, round robin, least loaded, length threshold,
    sampled learned) on one Table I family at 0.9 of the pool's serial
    capacity: each replica bitwise against the oracle in follow mode."""
    P, D = 2, 4
    cap = W.capacity_rps(W.make_point(P, D, n_classes=3), traffic)
    traf = traffic.scaled(0.9 * cap / traffic.mean_rate())
    cells = E.policy_cells(P, D, traf)
    rows, tr, out, g = E.run_cells(cells, replicas=3, requests=1500, seed=11, return_trace=True)
    log(f"{family}: " + ", ".join(f"{r['label']} {r['mean']:.3f}" for r in rows))
    rep = follow_replicas([c.point for c in cells], tr, out, range(len(cells) * 3), gpu_goodput=g)
    log(f"{family} policy grid vs oracle: {rep}")
    assert rep["replicas"] == len(cells) * 3


def test_saturation_search_matches_oracle():
    """The saturation search (round robin mid-collapse, Section IV-B) run
    on the GPU and on the oracle: every probe's mean goodput is identical
    and so are the bracket and the scale."""
    pt = W.make_point(2, 4, n_classes=3)
    traf = W.mixed_bursty()
    kw = dict(target=0.5, replicas=12, requests=2500, seed=3)
    gpu = E.saturation_scale(pt, traf, **kw)
    orc = E.saturation_scale(pt, traf, run=oracle_run_cells, **kw)
    log(f"saturation GPU {gpu['scale']} bracket {gpu.get('bracket')}; oracle {orc['scale']} bracket "
        f"{orc.get('bracket')}; {len(gpu['probes'])} probes")
    assert gpu["probes"] == orc["probes"]
    assert gpu["scale"] == orc["scale"] and gpu.get("bracket") == orc.get("bracket")
    assert gpu["scale"] is not None


def test_saturation_search_brackets_round_robin_collapse():
    pt = W.make_point(2, 4, n_classes=3)
    traf = W.mixed_bursty()
    res = E.saturation_scale(pt, traf, target=0.5, replicas=16, requests=3000, seed=1)
    log(f"saturation: scale {res['scale']}, probes {[(round(s, 3), round(g, 3)) for s, g in res['probes']]}")
    assert res["scale"] is not None
    s0, s1 = res["bracket"]
    assert s0 < res["scale"] <= s1
    # goodput falls with load across the probed grid (allowing replica noise)
    g = np.array([x for _, x in res["probes"]])
    assert g[0] > 0.5 > g[-1]
    assert np.all(np.diff(g) < 0.05)
    # at the found scale round robin is near the target
    rows = E.run_cells([E.Cell("rr", dict(pt, policy="round_robin"), traf.scaled(res["scale"]))],
                       replicas=16, requests=3000, seed=1)
    assert abs(rows[0]["mean"] - 0.5) < 0.1, rows


def test_service_study_matches_oracle_and_batching_raises_capacity():
    """Serial vs continuous-batching cells in one batch: every replica
    agrees with the oracle (bitwise), batching serves traffic that has
    collapsed the serial model at least as well, and round robin's collapse
    under batching comes at a higher arrival rate."""
    traf = W.mixed_bursty()
    cells = E.service_cells(2, 4, traf.scaled(1.0), policies=("learned", "round_robin"))
    rows, tr, out, g = E.run_cells(cells, replicas=3, requests=1500, seed=6, return_trace=True, ttft_tail=True)
    log("service: " + ", ".join(f"{r['label']} {r['mean']:.3f} p99 {r['ttft_p99_s']:.3f}s" for r in rows))
    ref = O.sim_trace([c.point for c in cells], tr, threads=16)
    for i, (o, st, gg, met) in ref.items():
        sl = slice(int(tr["offsets"][i]), int(tr["offsets"][i + 1]))
        assert np.array_equal(o["i_pre"], out["i_pre"][sl]) and np.array_equal(o["i_dec"], out["i_dec"][sl]), i
        assert np.array_equal(o["ttft_ns"], out["ttft_ns"][sl]) and np.array_equal(o["decode_span_ns"],
                                                                                   out["decode_span_ns"][sl]), i
        assert gg == g[i], i
    by = {r["label"]: r for r in rows}
    for pol in ("learned", "round_robin"):
        assert by[f"{pol} batched"]["mean"] >= by[f"{pol} serial"]["mean"]
    pt = W.make_point(2, 4, n_classes=3)
    scales = tuple(np.geomspace(0.25, 1024.0, 13))
    ser = E.saturation_scale(dict(pt, service="serial"), traf, scales=scales, replicas=8, requests=2000, seed=2)
    bat = E.saturation_scale(dict(pt, service="batched", beta_pre=W.BATCH_BETA, beta_dec=W.BATCH_BETA,
                                  batch_cap=E.BATCH_ROOM), traf, scales=scales, replicas=8, requests=2000, seed=2)
    log(f"round robin collapse scale: serial {ser['scale']}, batched {bat['scale']}; batched probes {bat['probes']}")
    # Section VI: under continuous batching (a batch of eight costs 2.9 % per
    # token) the simulator's round robin holds its goodput at arrival rates
    # three orders of magnitude above where the serial model collapses
    assert ser["scale"] is not None and ser["scale"] < 2.0
    assert bat["scale"] is None or bat["scale"] > 1000 * ser["scale"]
    assert min(g for _, g in bat["probes"]) > 0.5
