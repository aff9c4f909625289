"""Host-side parts of the experiment drivers (CPU): the calibration fit
(Section III-B) and the batch layout of a grid."""
import numpy as np

from paper_2609_16206_amd import experiments as E
from paper_2609_16206_amd import workload as W


def test_fit_recovers_noiseless_constants():
    pt = W.make_point(2, 4)
    fit = E.fit_service_constants(**E.latency_curves(pt, n=300))
    assert abs(fit["pre_base_ns"] - pt["pre_base_ns"]) < 1e-3 * pt["pre_base_ns"]
    assert abs(fit["pre_tok_ns"] - pt["pre_tok_ns"]) < 1e-6 * pt["pre_tok_ns"]
    assert abs(fit["dec_tok_ns"] - pt["dec_tok_ns"]) < 1e-9 * pt["dec_tok_ns"]
    # the calibrated router prices are the physics' own (Section III-B)
    q = E.calibrated_point(pt, fit)
    assert q["tau_dec_s"] == pt["tau_dec_s"] and q["tau_pre_s"] == pt["tau_pre_s"]


def test_fit_under_noise_is_close():
    pt = W.make_point(2, 4)
    fit = E.fit_service_constants(**E.latency_curves(pt, n=4000, noise=0.05, seed=3))
    assert abs(fit["dec_tok_ns"] / pt["dec_tok_ns"] - 1) < 0.01
    assert abs(fit["pre_tok_ns"] / pt["pre_tok_ns"] - 1) < 0.05


def test_mispriced_fit_is_detectable():
    """A point whose physics differs from the router's prices (the paper's
    7.4x decode mismatch) is repaired by fitting to the physics."""
    pt = W.make_point(2, 4, tau_dec_scale=1 / 7.4)
    assert pt["tau_dec_s"] < pt["dec_tok_ns"] * 1e-9 / 7
    q = E.calibrated_point(pt, E.fit_service_constants(**E.latency_curves(pt)))
    assert abs(q["tau_dec_s"] / (pt["dec_tok_ns"] * 1e-9) - 1) < 1e-6


def test_grid_trace_layout_and_streams():
    cells = E.policy_cells(2, 3, W.mixed_bursty())
    tr = E.build_trace(cells, replicas=3, requests=50, seed=5)
    assert tr["offsets"][-1] == len(cells) * 3 * 50
    assert list(tr["param_point"]) == [c for c in range(len(cells)) for _ in range(3)]
    assert tr["sample_bits"].shape == (len(cells) * 3 * 50, 4)
    # cells draw disjoint streams, the same cell draws the same ones
    a = tr["arrival_ns"][:50]
    assert not np.array_equal(a, tr["arrival_ns"][150:200])
    tr2 = E.build_trace(cells, replicas=3, requests=50, seed=5)
    assert np.array_equal(tr["prompt_len"], tr2["prompt_len"])


def test_noise_cells_change_only_the_prediction():
    cells = E.noise_cells(2, 3, W.mixed_bursty(), sigmas=(0.0, 1.5))
    t0 = E.build_trace(cells[:1], 1, 200, seed=2)
    t1 = E.build_trace(cells[1:], 1, 200, seed=2)
    for k in ("arrival_ns", "prompt_len", "out_len", "slo_class"):
        assert np.array_equal(t0[k], t1[k]), k
    assert np.array_equal(t0["pred_out_len"], np.maximum(1, t0["out_len"]))
    assert not np.array_equal(t1["pred_out_len"], t0["pred_out_len"])


def test_service_cells_pair_each_policy():
    """The service study pairs every policy's serial cell with its batched
    cell at the same traffic and betas (Section VI's correction)."""
    traf = W.mixed_bursty()
    cells = E.service_cells(2, 4, traf, policies=("learned", "round_robin"), beta=0.01)
    assert [c.label for c in cells] == ["learned serial", "learned batched", "round_robin serial",
                                        "round_robin batched"]
    for a, b in zip(cells[0::2], cells[1::2]):
        assert a.point["service"] == "serial" and b.point["service"] == "batched"
        assert b.point["beta_pre"] == b.point["beta_dec"] == 0.01
        assert a.traffic is b.traffic
        assert {k: v for k, v in a.point.items() if k != "service"} == {k: v for k, v in b.point.items()
                                                                       if k != "service"}


def _fake_runner(fn):
    """A cell runner whose mean goodput is fn(scale), the scale read back
    from the cell's traffic."""
    base = W.mixed_bursty()

    def run(cells, replicas, requests, seed, device):
        return [dict(label=c.label, mean=float(fn(c.traffic.mean_rate() / base.mean_rate()))) for c in cells]
    return run


def test_saturation_search_linear_curve_is_exact():
    """On a goodput curve that is linear in the scale the interpolation
    returns the exact crossing (0.5 at scale 1.3)."""
    res = E.saturation_scale(W.make_point(2, 4), W.mixed_bursty(), run=_fake_runner(lambda s: 1.15 - 0.5 * s))
    assert abs(res["scale"] - 1.3) < 1e-9
    s0, s1 = res["bracket"]
    assert s0 <= 1.3 <= s1 and s1 - s0 < 0.2 / 4


def test_saturation_search_bracket_uses_every_probe():
    """The bracket is taken over all probes so far: a refinement round whose
    four interior probes all lie above the target still narrows it (a
    bracket kept from the previous round would ignore them), and no probe
    lies strictly inside the final bracket."""
    fn = lambda s: 1.0 if s < 1.78 else 0.0  # noqa: E731
    res = E.saturation_scale(W.make_point(2, 4), W.mixed_bursty(), run=_fake_runner(fn), rounds=3)
    s0, s1 = res["bracket"]
    assert s0 < 1.78 <= s1
    inside = [s for s, _ in res["probes"] if s0 < s < s1]
    assert not inside
    assert s1 - s0 < 0.2 / 5 / 5 * 1.01  # two refinements of the 0.2-wide first bracket
    above = [s for s, g in res["probes"] if g >= 0.5]
    assert s0 == max(above)


def test_oracle_cell_runner_means():
    """The oracle's cell runner (used to check the GPU search) returns, per
    cell, the mean of the oracle goodput of its replicas."""
    from oracle import oracle as O
    from tests.parity import oracle_run_cells
    cells = E.policy_cells(2, 3, W.mixed_bursty(), policies=("round_robin", "least_loaded"))
    rows = oracle_run_cells(cells, replicas=2, requests=300, seed=9, threads=2)
    tr = E.build_trace(cells, 2, 300, 9)
    ref = O.sim_trace([c.point for c in cells], tr)
    for c in range(2):
        assert rows[c]["mean"] == float(np.mean([ref[2 * c][2], ref[2 * c + 1][2]]))
