"""Simulation experiments on the HIP simulator.

Each experiment is a grid of cells (a parameter point plus the traffic it
sees), simulated as one batch: every cell gets its own replicas, all cells
go through a single rt_sim_run_replicas call, and the result is the goodput
of each cell (mean and spread over its replicas).  This is the batched
form of the studies of Section V (policy grid, feature ablation, predictor
noise, pool width), plus the two host-side steps the method wraps around
the router:

  * saturation_scale: the protocol's saturation search (Section IV-B): the
    arrival-rate scale at which a reference policy, round robin by default,
    is mid-collapse (its goodput crosses a target), found by probing a grid
    of scales in one batch and refining inside the bracketing interval;
  * fit_service_constants: the calibration step (Section III-B): prices
    per prompt and per output token fitted to latency curves by least
    squares;
  * service_cells / the `service` study: the serial-service model next to
    continuous batching at the prefill and the decode stage alike (Section VI's correction), per
    policy at one arrival rate, with goodput and tail TTFT, and the
    saturation scale under each model.

Replica streams: cell c's replica k draws from replica index
c * stride + k of the workload seed, so cells never share draws.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import rt_router as R
from . import workload as W


@dataclass
class Cell:
    label: str
    point: Dict
    traffic: W.Traffic


def build_trace(cells: Sequence[Cell], replicas: int, requests: int, seed: int,
                stride: int = 1 << 20) -> Dict[str, np.ndarray]:
    """SoA trace with `replicas` replicas per cell (cell c uses point c)."""
    parts, pp = [], []
    for c, cell in enumerate(cells):
        for k in range(replicas):
            parts.append(W.replica_arrays(seed, c * stride + k, cell.traffic, requests))
            pp.append(c)
    keys = ("arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class")
    tr = {k: np.concatenate([q[k] for q in parts]) for k in keys}
    tr["offsets"] = np.arange(len(parts) + 1, dtype=np.int64) * requests
    tr["param_point"] = np.array(pp, np.int32)
    if any(cell.point["policy"] == "learned_sampled" for cell in cells):
        W.add_sample_words(tr, seed, [c * stride + k for c in range(len(cells)) for k in range(replicas)])
    return tr


def run_cells(cells: Sequence[Cell], replicas: int = 32, requests: int = 5000, seed: int = 0,
              device: int = 0, return_trace: bool = False, ttft_tail: bool = False):
    """Goodput per cell: a list of dicts (label, mean, std, min, max; with
    `ttft_tail` also the median and 99th-percentile TTFT in seconds over
    the cell's requests), and optionally the trace and per-replica
    goodput."""
    import torch

    tr = build_trace(cells, replicas, requests, seed)
    sim = R.Simulator([c.point for c in cells], device=device)
    try:
        dtr = R.to_device(tr, f"cuda:{device}")
        out = sim.run(dtr)
        g, _ = sim.goodput(dtr, out)
        flags = sim.data_status()
        g = g.cpu().numpy()
        outs = {k: v.cpu().numpy() for k, v in out.items()} if (return_trace or ttft_tail) else None
        torch.cuda.synchronize(device)
    finally:
        sim.close()
    if flags:
        raise RuntimeError(f"simulation reported data flags {flags:#x}")
    rows = []
    for c, cell in enumerate(cells):
        x = g[c * replicas:(c + 1) * replicas]
        row = dict(label=cell.label, mean=float(x.mean()), std=float(x.std()), min=float(x.min()),
                   max=float(x.max()))
        if ttft_tail:
            t = outs["ttft_ns"][c * replicas * requests:(c + 1) * replicas * requests]
            t = t[t >= 0] * 1e-9
            row["ttft_p50_s"] = float(np.percentile(t, 50)) if t.size else None
            row["ttft_p99_s"] = float(np.percentile(t, 99)) if t.size else None
        rows.append(row)
    if return_trace:
        return rows, tr, outs, g
    return rows


def saturation_scale(point: Dict, traffic: W.Traffic, target: float = 0.5, policy: str = "round_robin",
                     scales: Sequence[float] = tuple(np.linspace(0.4, 2.0, 9)), rounds: int = 2,
                     replicas: int = 32, requests: int = 4000, seed: int = 0, device: int = 0,
                     run=None) -> Dict:
    """Arrival-rate scale (relative to `traffic`) at which `policy` reaches
    goodput `target`.  Each round simulates a grid of scales in one batch;
    the bracket is then taken over every probe so far: its low end is the
    largest probed scale whose mean goodput is still >= target, its high end
    the smallest larger probed scale below the target, and the next round
    probes four scales inside it.  The answer interpolates linearly inside
    the last bracket.  `run(cells, replicas, requests, seed, device)` returns
    one row (with "mean") per cell; the default simulates on the GPU.
    Returns the scale, the bracket and the probed (scale, goodput) pairs."""
    run = run_cells if run is None else run
    pt = dict(point, policy=policy)
    probes: List[Tuple[float, float]] = []
    grid = [float(s) for s in scales]
    lo = hi = None
    for k in range(max(1, rounds)):
        rows = run([Cell(f"x{s:.4f}", pt, traffic.scaled(s)) for s in grid], replicas, requests, seed, device)
        probes.extend(zip(grid, [r["mean"] for r in rows]))
        allp = sorted(probes)
        above = [q for q in allp if q[1] >= target]
        if not above:
            lo = hi = None
            break
        lo = max(above)  # the largest probed scale still at or above the target
        cand = [q for q in allp if q[0] > lo[0] and q[1] < target]
        if not cand:
            hi = None
            break
        hi = min(cand)
        grid = [float(x) for x in np.linspace(lo[0], hi[0], 6)[1:-1]]
    probes.sort()
    if lo is None or hi is None:
        return dict(scale=None, probes=probes)
    (s0, g0), (s1, g1) = lo, hi
    s = s0 if g0 == g1 else s0 + (target - g0) * (s1 - s0) / (g1 - g0)
    return dict(scale=float(s), bracket=(s0, s1), probes=probes)


def fit_service_constants(prompt_len: np.ndarray, prefill_ns: np.ndarray, out_len: np.ndarray,
                          decode_ns: np.ndarray) -> Dict:
    """Least-squares prices from latency curves: prefill latency = base +
    p * pre_tok (a line in p); decode time = (o - 1) * dec_tok (a line
    through the origin in o - 1).  Returns nanoseconds and the router's
    float32 seconds per token."""
    p = np.asarray(prompt_len, np.float64)
    t = np.asarray(prefill_ns, np.float64)
    A = np.stack([np.ones_like(p), p], axis=1)
    (base, pre_tok), *_ = np.linalg.lstsq(A, t, rcond=None)
    k = np.asarray(out_len, np.float64) - 1.0
    d = np.asarray(decode_ns, np.float64)
    dec_tok = float((k * d).sum() / (k * k).sum())
    return dict(pre_base_ns=float(base), pre_tok_ns=float(pre_tok), dec_tok_ns=dec_tok,
                tau_pre_s=float(np.float32(pre_tok * 1e-9)), tau_dec_s=float(np.float32(dec_tok * 1e-9)),
                pre_base_s=float(np.float32(base * 1e-9)))


def latency_curves(point: Dict, n: int = 400, noise: float = 0.0, seed: int = 0) -> Dict[str, np.ndarray]:
    """Synthetic benchmark of the simulated hardware (the calibration's
    input): prefill latency over prompt lengths spread to 8k tokens and
    decode time over output lengths spread to 4k, from the point's physics,
    with optional multiplicative log-normal noise."""
    rng = np.random.default_rng([int(seed), 7])
    p = np.rint(np.exp(rng.uniform(np.log(16), np.log(8192), n))).astype(np.int64)
    o = np.rint(np.exp(rng.uniform(np.log(2), np.log(4096), n))).astype(np.int64)
    pre = point["pre_base_ns"] + p * point["pre_tok_ns"]
    dec = (o - 1) * point["dec_tok_ns"]
    if noise > 0:
        pre = pre * np.exp(noise * rng.standard_normal(n))
        dec = dec * np.exp(noise * rng.standard_normal(n))
    return dict(prompt_len=p, prefill_ns=pre.astype(np.float64), out_len=o, decode_ns=dec.astype(np.float64))


def calibrated_point(point: Dict, fit: Dict) -> Dict:
    """The point with its router prices replaced by fitted ones."""
    q = dict(point)
    q["tau_pre_s"], q["tau_dec_s"], q["pre_base_s"] = fit["tau_pre_s"], fit["tau_dec_s"], fit["pre_base_s"]
    return q


# --------------------------------------------------------------------------
# Grids of Section V
# --------------------------------------------------------------------------
def policy_cells(P: int, D: int, traffic: W.Traffic, policies=("learned", "round_robin", "least_loaded",
                                                                 "length_threshold", "learned_sampled"),
                 **kw) -> List[Cell]:
    return [Cell(pol, W.make_point(P, D, n_classes=3, policy=pol, **kw), traffic) for pol in policies]


def ablation_cells(P: int, D: int, traffic: W.Traffic, **kw) -> List[Cell]:
    """The learned router with one signal removed at a time (Section V-G):
    no backlog (w_b = 0), no length (w_s = 0), no cache pressure (rho = 0),
    no SLO class (sigma = 1), no queue term (w_q = 0)."""
    base = dict(n_classes=3, **kw)
    variants = [("full", {}), ("no backlog", dict(w_b=0.0)), ("no length", dict(w_s=0.0)),
                ("no pressure", dict(rho=0.0)), ("no class", dict(sigma=[1.0] * 8)), ("no queue", dict(w_q=0.0))]
    return [Cell(name, W.make_point(P, D, **dict(base, **v)), traffic) for name, v in variants]


def noise_cells(P: int, D: int, traffic: W.Traffic, sigmas=(0.0, 0.3, 0.6, 0.9, 1.2, 1.5), **kw) -> List[Cell]:
    """The learned router under output-length predictor error (Section V-H):
    o^ = o * exp(sigma * z)."""
    pt = W.make_point(P, D, n_classes=3, **kw)
    return [Cell(f"sigma {s:g}", pt, W.with_predictor_sigma(traffic, s)) for s in sigmas]


# Room per instance for batch members and KV transfers in flight in the
# service study: near saturation a batched instance holds hundreds.
BATCH_ROOM = 4096


def service_cells(P: int, D: int, traffic: W.Traffic, policies=("learned", "round_robin", "least_loaded"),
                  beta: float = W.BATCH_BETA, **kw) -> List[Cell]:
    """Each policy under the serial-service model and with both stages
    batched continuously (Section VI), at the same arrival rate."""
    cells = []
    for pol in policies:
        for sv in ("serial", "batched"):
            pt = W.make_point(P, D, n_classes=3, policy=pol, service=sv, beta_pre=beta, beta_dec=beta, **kw)
            pt["batch_cap"] = BATCH_ROOM
            cells.append(Cell(f"{pol} {sv}", pt, traffic))
    return cells


def width_cells(P: int, widths: Sequence[int], traffic: W.Traffic, policies=("learned", "round_robin"),
                **kw) -> List[Cell]:
    """Decode-pool widths at a fixed arrival rate (Section V-D)."""
    return [Cell(f"{pol} D={d}", W.make_point(P, d, n_classes=3, policy=pol, **kw), traffic)
            for d in widths for pol in policies]


# --------------------------------------------------------------------------
# Command line: python -m paper_2609_16206_amd.experiments <study> [options]
# --------------------------------------------------------------------------
TRAFFIC = {"mixed": lambda: W.mixed_bursty(), "chat": lambda: W.chat(4.0), "document": lambda: W.document(4.0),
           "reasoning": lambda: W.reasoning(1.0)}


def main(argv=None) -> None:
    import argparse
    import json

    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("study", choices=["saturation", "policies", "ablation", "noise", "width", "calibrate",
                                      "service"])
    ap.add_argument("--traffic", default="mixed", choices=sorted(TRAFFIC))
    ap.add_argument("--prefill", type=int, default=2)
    ap.add_argument("--decode", type=int, default=4)
    ap.add_argument("--scale", type=float, default=None,
                    help="arrival-rate scale; default: the saturation scale of round robin")
    ap.add_argument("--replicas", type=int, default=32)
    ap.add_argument("--requests", type=int, default=5000)
    ap.add_argument("--seed", type=int, default=0)
    a = ap.parse_args(argv)
    traf = TRAFFIC[a.traffic]()
    pt = W.make_point(a.prefill, a.decode, n_classes=3)
    if a.study == "calibrate":
        fit = fit_service_constants(**latency_curves(pt, noise=0.05, seed=a.seed))
        print(json.dumps(fit))
        return
    if a.study == "service":
        # round robin's saturation scale under each model, then every
        # policy under both at the serial model's saturation scale
        sat = {sv: saturation_scale(dict(pt, service=sv, beta_pre=W.BATCH_BETA, beta_dec=W.BATCH_BETA,
                                         batch_cap=BATCH_ROOM), traf,
                                    scales=tuple(np.geomspace(0.25, 1024.0, 13)), replicas=a.replicas,
                                    requests=a.requests, seed=a.seed)["scale"]
               for sv in ("serial", "batched")}
        print(json.dumps(dict(saturation_scale=sat, note="None: no collapse within the probed scales 0.25-1024")))
        scale = a.scale if a.scale is not None else sat["serial"]
        for r in run_cells(service_cells(a.prefill, a.decode, traf.scaled(scale)), a.replicas, a.requests, a.seed,
                           ttft_tail=True):
            print(json.dumps(dict(r, scale=scale)))
        return
    scale = a.scale
    if scale is None or a.study == "saturation":
        sat = saturation_scale(pt, traf, replicas=a.replicas, requests=a.requests, seed=a.seed)
        if a.study == "saturation":
            print(json.dumps(dict(scale=sat["scale"], probes=sat["probes"])))
            return
        scale = sat["scale"]
    traf = traf.scaled(scale)
    cells = {"policies": lambda: policy_cells(a.prefill, a.decode, traf),
             "ablation": lambda: ablation_cells(a.prefill, a.decode, traf),
             "noise": lambda: noise_cells(a.prefill, a.decode, traf),
             "width": lambda: width_cells(a.prefill, (3, 4, 6, 8), traf)}[a.study]()
    for r in run_cells(cells, a.replicas, a.requests, a.seed):
        print(json.dumps(dict(r, scale=scale)))


if __name__ == "__main__":
    main()
