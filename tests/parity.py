"""GPU-vs-oracle parity helpers (test infrastructure).

The oracle runs in follow mode: at every decision it computes its own float32
costs; where the GPU placed a request elsewhere, the divergence is accepted
only if the GPU's choice costs at most 1e-6 relative more than the oracle's
best (a near tie), and the oracle then adopts the GPU's choice so the two
trajectories stay aligned.  Anything else is a failure.  On the aligned
trajectory every per-request TTFT and decode span (int64 ns) and every
replica's goodput must be bitwise equal.
"""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor
from typing import Dict, Iterable, Optional

import numpy as np

from oracle import oracle as O

TIE_REL = 1e-6
KEYS = ("arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class")


def follow_replicas(points, trace: Dict[str, np.ndarray], gpu: Dict[str, np.ndarray], replicas: Iterable[int],
                    prefix: Optional[int] = None, gpu_goodput: Optional[np.ndarray] = None,
                    gpu_met: Optional[np.ndarray] = None, threads: int = 16) -> Dict:
    """Check the listed replicas (optionally only their first `prefix`
    requests, which a causal simulation fixes on their own).  `gpu` holds the
    GPU outputs aligned with the trace.  Returns a report; raises
    AssertionError on the first failing replica."""
    off = trace["offsets"]
    pp = trace["param_point"]
    reps = list(replicas)

    def one(i):
        lo, hi = int(off[i]), int(off[i + 1])
        if prefix is not None:
            hi = min(hi, lo + prefix)
        sl = slice(lo, hi)
        pt = points[int(pp[i])]
        args = [trace[k][sl] for k in KEYS]
        sb = trace["sample_bits"][sl] if "sample_bits" in trace else None
        out, st = O.sim_replica(pt, *args, follow_pre=gpu["i_pre"][sl], follow_dec=gpu["i_dec"][sl], tie_rel=TIE_REL,
                                sample_bits=sb)
        res = dict(rep=i, n=hi - lo, near_tie=st["near_tie_pre"] + st["near_tie_dec"],
                   mismatch=st["mismatch_pre"] + st["mismatch_dec"], first=st["first_mismatch"],
                   close=st["close_pre"] + st["close_dec"], invalid=st["invalid"])
        res["ttft_eq"] = bool(np.array_equal(out["ttft_ns"], gpu["ttft_ns"][sl]))
        res["span_eq"] = bool(np.array_equal(out["decode_span_ns"], gpu["decode_span_ns"][sl]))
        res["place_eq"] = bool(np.array_equal(out["i_pre"], gpu["i_pre"][sl]) and
                               np.array_equal(out["i_dec"], gpu["i_dec"][sl]))
        if prefix is None or hi == int(off[i + 1]):
            g, met = O.goodput(pt, args[2], args[4], out["ttft_ns"], out["decode_span_ns"])
            res["goodput"] = g
            if gpu_met is not None:
                res["met_eq"] = int(gpu_met[i]) == met
            if gpu_goodput is not None:
                res["goodput_eq"] = float(gpu_goodput[i]) == g
        return res

    with ThreadPoolExecutor(max_workers=threads) as ex:
        results = list(ex.map(one, reps))
    bad = [r for r in results if r["mismatch"] or not (r["ttft_eq"] and r["span_eq"] and r["place_eq"])
           or r.get("met_eq") is False or r.get("goodput_eq") is False]
    report = dict(replicas=len(results), requests=int(sum(r["n"] for r in results)),
                  near_ties=int(sum(r["near_tie"] for r in results)),
                  close_decisions=int(sum(r["close"] for r in results)),
                  invalid=int(sum(r["invalid"] for r in results)), failures=len(bad))
    assert not bad, f"parity failure: {bad[:3]} (report {report})"
    return report


def check_properties(points, trace: Dict[str, np.ndarray], gpu: Dict[str, np.ndarray]) -> None:
    """Properties every replica must satisfy, checked vectorised over the
    whole batch: placements in range, TTFT at least the prefill service, decode
    span at least transfer + decode service, rejected requests only where the
    data checks reject."""
    pp = trace["param_point"]
    off = trace["offsets"]
    counts = np.diff(off)
    pid = np.repeat(pp, counts)
    P = np.array([p["n_prefill"] for p in points], np.int64)[pid]
    D = np.array([p["n_decode"] for p in points], np.int64)[pid]
    base = np.array([p["pre_base_ns"] for p in points], np.int64)[pid]
    ptok = np.array([p["pre_tok_ns"] for p in points], np.int64)[pid]
    dtok = np.array([p["dec_tok_ns"] for p in points], np.int64)[pid]
    xtok = np.array([p["xfer_tok_ns"] for p in points], np.int64)[pid]
    lo, hi = int(off[0]), int(off[-1])
    p = trace["prompt_len"][lo:hi].astype(np.int64)
    o = trace["out_len"][lo:hi].astype(np.int64)
    ip, idd = gpu["i_pre"][lo:hi], gpu["i_dec"][lo:hi]
    tt, sp = gpu["ttft_ns"][lo:hi], gpu["decode_span_ns"][lo:hi]
    valid = tt >= 0
    assert np.all((ip[valid] >= 0) & (ip[valid] < P[valid]))
    assert np.all((idd[valid] >= 0) & (idd[valid] < D[valid]))
    assert np.all(tt[valid] >= base[valid] + p[valid] * ptok[valid])
    assert np.all(sp[valid] >= p[valid] * xtok[valid] + (o[valid] - 1) * dtok[valid])
    assert np.all(ip[~valid] == -1) and np.all(idd[~valid] == -1) and np.all(sp[~valid] == -1)


def goodput_recount(points, trace, gpu) -> np.ndarray:
    """Met counts recomputed in numpy from the GPU outputs (independent of
    both implementations' goodput code)."""
    off = trace["offsets"]
    pp = trace["param_point"]
    counts = np.diff(off)
    pid = np.repeat(pp, counts)
    lo, hi = int(off[0]), int(off[-1])
    c = trace["slo_class"][lo:hi].astype(np.int64)
    o = trace["out_len"][lo:hi].astype(np.int64)
    ttft_t = np.array([p["slo_ttft_ns"] for p in points], np.int64)[pid, c]
    tpot_t = np.array([p["slo_tpot_ns"] for p in points], np.int64)[pid, c]
    tt, sp = gpu["ttft_ns"][lo:hi], gpu["decode_span_ns"][lo:hi]
    met = (tt >= 0) & (tt <= ttft_t) & ((o <= 1) | (sp <= tpot_t * (o - 1)))
    rep = np.repeat(np.arange(len(counts)), counts)
    return np.bincount(rep, weights=met, minlength=len(counts)).astype(np.int64)


def oracle_run_cells(cells, replicas: int, requests: int, seed: int, device: int = 0, threads: int = 16):
    """The experiment drivers' cell runner with the oracle in place of the
    GPU: the same trace (experiments.build_trace), every replica simulated by
    the oracle, and each cell's mean goodput over its replicas computed as
    the GPU runner computes it."""
    from paper_2609_16206_amd import experiments as E
    tr = E.build_trace(cells, replicas, requests, seed)
    ref = O.sim_trace([c.point for c in cells], tr, threads=threads)
    g = np.array([ref[i][2] for i in range(len(cells) * replicas)], np.float64)
    rows = []
    for c, cell in enumerate(cells):
        x = g[c * replicas:(c + 1) * replicas]
        rows.append(dict(label=cell.label, mean=float(x.mean()), std=float(x.std()), min=float(x.min()),
                         max=float(x.max())))
    return rows
