"""ctypes front end of the CPU oracle (test infrastructure only).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg use
this module.  It loads ``librt_oracle.so`` (built by ``oracle/build.py``) and
takes plain numpy arrays plus parameter-point dictionaries (the keys produced
by the workload generator).  It imports nothing from the GPU package.
"""
from __future__ import annotations

import ctypes as C
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("RT_ORACLE_LIB") or os.path.join(HERE, "librt_oracle.so")
MAX_CLASSES = 8
POLICY = {"learned": 0, "round_robin": 1, "least_loaded": 2, "learned_sampled": 3, "length_threshold": 4}
BACKLOG = {"true": 0, "proxy": 1}
POOL = {"prefill": 0, "decode": 1}
SERVICE = {"serial": 0, "batched": 1}


class Router(C.Structure):
    _fields_ = [("w_b", C.c_float), ("w_s", C.c_float), ("w_q", C.c_float), ("rho", C.c_float),
                ("tau_pre_s", C.c_float), ("tau_dec_s", C.c_float), ("pre_base_s", C.c_float),
                ("sigma", C.c_float * MAX_CLASSES)]


class Point(C.Structure):
    _fields_ = [("n_prefill", C.c_int32), ("n_decode", C.c_int32), ("n_classes", C.c_int32),
                ("policy", C.c_int32), ("backlog_mode", C.c_int32), ("router", Router),
                ("pre_base_ns", C.c_int64), ("pre_tok_ns", C.c_int64), ("dec_tok_ns", C.c_int64),
                ("xfer_tok_ns", C.c_int64), ("kv_cap_pre", C.c_int64), ("kv_cap_dec", C.c_int64),
                ("slo_ttft_ns", C.c_int64 * MAX_CLASSES), ("slo_tpot_ns", C.c_int64 * MAX_CLASSES),
                ("len_threshold", C.c_int32), ("service", C.c_int32), ("beta_pre", C.c_double),
                ("beta_dec", C.c_double)]


STAT_FIELDS = ["invalid", "near_tie_pre", "near_tie_dec", "mismatch_pre", "mismatch_dec", "first_mismatch",
               "tie_pre", "tie_dec", "close_pre", "close_dec", "over_cap_pre", "over_cap_dec", "max_queue_pre", "max_queue_dec",
               "retired_pre", "retired_dec", "violations", "end_inflight_pre", "end_inflight_dec"]


class Stats(C.Structure):
    _fields_ = [(f, C.c_int64) for f in STAT_FIELDS]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"oracle library not built: {LIB_PATH} (run oracle/build.py)")
        L = C.CDLL(LIB_PATH)
        P = C.c_void_p
        L.orc_score.argtypes = [C.POINTER(Router), C.c_int32, C.c_int32, P, P, P, C.c_int64, C.c_int64,
                                C.c_int64, P, P, P, P, P, P, P]
        L.orc_score.restype = C.c_int
        L.orc_candidates.argtypes = [C.c_uint32, C.c_uint32, C.c_int32, C.POINTER(C.c_int32), C.POINTER(C.c_int32)]
        L.orc_candidates.restype = None
        L.orc_sim_replica.argtypes = [C.POINTER(Point), C.c_int64, P, P, P, P, P, P, P, P, C.c_double,
                                      P, P, P, P, C.POINTER(Stats)]
        L.orc_sim_replica.restype = C.c_int
        L.orc_sim_replica_batched.argtypes = L.orc_sim_replica.argtypes
        L.orc_sim_replica_batched.restype = C.c_int
        L.orc_goodput.argtypes = [C.POINTER(Point), C.c_int64, P, P, P, P, C.POINTER(C.c_double)]
        L.orc_goodput.restype = C.c_int64
        _lib = L
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def router_struct(d: Dict) -> Router:
    r = Router()
    for k in ("w_b", "w_s", "w_q", "rho", "tau_pre_s", "tau_dec_s", "pre_base_s"):
        setattr(r, k, float(d[k]))
    sg = list(d["sigma"]) + [1.0] * (MAX_CLASSES - len(d["sigma"]))
    for i in range(MAX_CLASSES):
        r.sigma[i] = float(sg[i])
    return r


def point_struct(d: Dict) -> Point:
    p = Point()
    p.n_prefill, p.n_decode, p.n_classes = int(d["n_prefill"]), int(d["n_decode"]), int(d["n_classes"])
    p.policy = POLICY[d["policy"]] if isinstance(d["policy"], str) else int(d["policy"])
    p.backlog_mode = BACKLOG[d["backlog_mode"]] if isinstance(d["backlog_mode"], str) else int(d["backlog_mode"])
    p.router = router_struct(d)
    for k in ("pre_base_ns", "pre_tok_ns", "dec_tok_ns", "xfer_tok_ns", "kv_cap_pre", "kv_cap_dec"):
        setattr(p, k, int(d[k]))
    for i in range(MAX_CLASSES):
        p.slo_ttft_ns[i] = int(d["slo_ttft_ns"][i])
        p.slo_tpot_ns[i] = int(d["slo_tpot_ns"][i])
    p.len_threshold = int(d.get("len_threshold", 1))
    sv = d.get("service", "serial")
    p.service = SERVICE[sv] if isinstance(sv, str) else int(sv)
    p.beta_pre = float(d.get("beta_pre", 0.0))
    p.beta_dec = float(d.get("beta_dec", 0.0))
    return p


def candidates(u: int, v: int, n: int):
    """The two sampled candidates of a pool of n instances for words u, v."""
    c1, c2 = C.c_int32(), C.c_int32()
    lib().orc_candidates(int(u) & 0xFFFFFFFF, int(v) & 0xFFFFFFFF, int(n), C.byref(c1), C.byref(c2))
    return c1.value, c2.value


def score(router: Dict, pool: str, backlog_s, queue, kv_occ, kv_cap: int, n_inst: int, inst_stride: int,
          prompt_len, pred_out_len, slo_class, sample_bits=None):
    """Standalone scorer: (idx i32, score f32, second-best f32) per request.
    ``sample_bits`` ([n, 2] uint32, optional) restricts each request to its
    two sampled candidates."""
    b = np.ascontiguousarray(backlog_s, np.float32)
    q = np.ascontiguousarray(queue, np.int32)
    k = np.ascontiguousarray(kv_occ, np.int32)
    p = np.ascontiguousarray(prompt_len, np.int32)
    oh = np.ascontiguousarray(pred_out_len, np.int32)
    c = np.ascontiguousarray(slo_class, np.uint8)
    n = p.size
    idx = np.empty(n, np.int32)
    sc = np.empty(n, np.float32)
    sec = np.empty(n, np.float32)
    r = router_struct(router)
    sb = None if sample_bits is None else np.ascontiguousarray(sample_bits, np.uint32).reshape(n, 2)
    rc = lib().orc_score(C.byref(r), POOL[pool], n_inst, _ptr(b), _ptr(q), _ptr(k), kv_cap, inst_stride, n,
                         _ptr(p), _ptr(oh), _ptr(c), _ptr(sb), _ptr(idx), _ptr(sc), _ptr(sec))
    if rc != 0:
        raise ValueError(f"orc_score rejected its arguments (rc={rc})")
    return idx, sc, sec


def sim_replica(point: Dict, arrival_ns, prompt_len, out_len, pred_out_len, slo_class,
                follow_pre=None, follow_dec=None, tie_rel: float = 1e-6, sample_bits=None):
    """One replica; returns (dict of outputs, dict of stats).  ``sample_bits``
    ([n, 4] uint32) is required for the sampled policy.  The point's
    ``service`` ("serial", the default, or "batched") picks the service
    model."""
    a = np.ascontiguousarray(arrival_ns, np.int64)
    n = a.size
    arrs = [np.ascontiguousarray(x, t) for x, t in ((prompt_len, np.int32), (out_len, np.int32),
                                                    (pred_out_len, np.int32), (slo_class, np.uint8))]
    fp = None if follow_pre is None else np.ascontiguousarray(follow_pre, np.int32)
    fd = None if follow_dec is None else np.ascontiguousarray(follow_dec, np.int32)
    out = dict(i_pre=np.empty(n, np.int32), i_dec=np.empty(n, np.int32),
               ttft_ns=np.empty(n, np.int64), decode_span_ns=np.empty(n, np.int64))
    sb = None if sample_bits is None else np.ascontiguousarray(sample_bits, np.uint32).reshape(n, 4)
    st = Stats()
    pst = point_struct(point)
    fn = lib().orc_sim_replica_batched if pst.service == SERVICE["batched"] else lib().orc_sim_replica
    rc = fn(C.byref(pst), n, _ptr(a), *[_ptr(x) for x in arrs], _ptr(sb), _ptr(fp), _ptr(fd),
            float(tie_rel), _ptr(out["i_pre"]), _ptr(out["i_dec"]), _ptr(out["ttft_ns"]),
            _ptr(out["decode_span_ns"]), C.byref(st))
    if rc != 0:
        raise ValueError(f"{fn.__name__} failed (rc={rc})")
    return out, {f: int(getattr(st, f)) for f in STAT_FIELDS}


def goodput(point: Dict, out_len, slo_class, ttft_ns, span_ns):
    """(goodput, met) of one replica."""
    o = np.ascontiguousarray(out_len, np.int32)
    c = np.ascontiguousarray(slo_class, np.uint8)
    t = np.ascontiguousarray(ttft_ns, np.int64)
    s = np.ascontiguousarray(span_ns, np.int64)
    g = C.c_double()
    pst = point_struct(point)
    met = lib().orc_goodput(C.byref(pst), o.size, _ptr(o), _ptr(c), _ptr(t), _ptr(s), C.byref(g))
    return g.value, int(met)


def sim_trace(points: Sequence[Dict], trace: Dict[str, np.ndarray], replicas: Optional[Sequence[int]] = None,
              follow: Optional[Dict[str, np.ndarray]] = None, tie_rel: float = 1e-6, threads: int = 1):
    """Run (a subset of) the replicas of an SoA trace.

    Returns {replica: (outputs, stats, goodput, met)}.  ``follow`` holds full
    i_pre / i_dec arrays aligned with the trace (placements to adopt).
    Replicas are independent; ``threads`` > 1 runs them concurrently (the
    library call releases the GIL), each replica still strictly sequential.
    """
    off = trace["offsets"]
    pp = trace["param_point"]
    reps = range(len(off) - 1) if replicas is None else replicas

    def one(i):
        lo, hi = int(off[i]), int(off[i + 1])
        pt = points[int(pp[i])]
        sl = slice(lo, hi)
        fpre = None if follow is None else follow["i_pre"][sl]
        fdec = None if follow is None else follow["i_dec"][sl]
        sb = trace.get("sample_bits")
        out, st = sim_replica(pt, trace["arrival_ns"][sl], trace["prompt_len"][sl], trace["out_len"][sl],
                              trace["pred_out_len"][sl], trace["slo_class"][sl], fpre, fdec, tie_rel,
                              None if sb is None else sb[sl])
        g, met = goodput(pt, trace["out_len"][sl], trace["slo_class"][sl], out["ttft_ns"], out["decode_span_ns"])
        return i, (out, st, g, met)

    if threads <= 1:
        return dict(one(i) for i in reps)
    with ThreadPoolExecutor(max_workers=threads) as ex:
        return dict(ex.map(one, list(reps)))
