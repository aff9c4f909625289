"""Python binding of librt_router (include/rt_router.h): argument marshalling only.

Every entry point of the C ABI is exposed under the same name.  Device buffers
are torch tensors on the GPU; the library receives their data pointers and the
current torch stream.  Every step of the simulation and scoring runs in the
HIP kernels of librt_router.so; there is no fallback: importing this module
raises if the library has not been built (``python -m
paper_2609_16206_amd.build``).
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, Optional, Sequence

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("RT_ROUTER_LIB") or os.path.join(HERE, "librt_router.so")

RT_OK, RT_EINVAL, RT_ENOMEM, RT_EDEVICE, RT_ERANGE, RT_EUNSUPPORTED, RT_EDATA = 0, -1, -2, -3, -4, -5, -6
RT_POLICY = {"learned": 0, "round_robin": 1, "least_loaded": 2, "learned_sampled": 3, "length_threshold": 4}
RT_BACKLOG = {"true": 0, "proxy": 1}
RT_POOL = {"prefill": 0, "decode": 1}
RT_SERVICE = {"serial": 0, "batched": 1}
RT_MAX_CLASSES = 8
RT_MAX_POOL = 1024

EXPORTS = ("rt_sim_create", "rt_sim_destroy", "rt_sim_run_replicas", "rt_sim_run_replicas_noalloc", "rt_goodput",
           "rt_sim_data_status", "rt_sim_timing", "rt_sim_kernel_time", "rt_score_argmin", "rt_last_error")


class RtError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"rt_router status {status}: {msg}")
        self.status = status


class rt_router_params(C.Structure):
    _fields_ = [("w_b", C.c_float), ("w_s", C.c_float), ("w_q", C.c_float), ("rho", C.c_float),
                ("tau_pre_s", C.c_float), ("tau_dec_s", C.c_float), ("pre_base_s", C.c_float),
                ("sigma", C.c_float * RT_MAX_CLASSES)]


class rt_physics(C.Structure):
    _fields_ = [("pre_base_ns", C.c_int64), ("pre_tok_ns", C.c_int64), ("dec_tok_ns", C.c_int64),
                ("xfer_tok_ns", C.c_int64), ("kv_cap_pre", C.c_int64), ("kv_cap_dec", C.c_int64),
                ("slo_ttft_ns", C.c_int64 * RT_MAX_CLASSES), ("slo_tpot_ns", C.c_int64 * RT_MAX_CLASSES)]


class rt_point(C.Structure):
    _fields_ = [("n_prefill", C.c_int32), ("n_decode", C.c_int32), ("n_classes", C.c_int32),
                ("policy", C.c_int32), ("backlog_mode", C.c_int32), ("router", rt_router_params),
                ("phys", rt_physics), ("len_threshold", C.c_int32), ("service", C.c_int32),
                ("beta_pre", C.c_double), ("beta_dec", C.c_double), ("batch_cap", C.c_int32),
                ("reserved", C.c_int32)]


class rt_trace(C.Structure):
    _fields_ = [("n_replicas", C.c_int64), ("n_requests", C.c_int64), ("offsets", C.c_void_p),
                ("param_point", C.c_void_p), ("arrival_ns", C.c_void_p), ("prompt_len", C.c_void_p),
                ("out_len", C.c_void_p), ("pred_out_len", C.c_void_p), ("slo_class", C.c_void_p),
                ("sample_bits", C.c_void_p)]


class rt_sim_out(C.Structure):
    _fields_ = [("i_pre", C.c_void_p), ("i_dec", C.c_void_p), ("ttft_ns", C.c_void_p),
                ("decode_span_ns", C.c_void_p)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"librt_router.so is missing at {LIB_PATH}: build it with "
                          "`python -m paper_2609_16206_amd.build`")
    L = C.CDLL(LIB_PATH)
    P = C.c_void_p
    L.rt_sim_create.argtypes = [C.POINTER(rt_point), C.c_int32, C.c_int32, C.POINTER(C.c_void_p)]
    L.rt_sim_destroy.argtypes = [P]
    L.rt_sim_run_replicas.argtypes = [P, C.POINTER(rt_trace), C.POINTER(rt_sim_out), P]
    L.rt_sim_run_replicas_noalloc.argtypes = [P, C.POINTER(rt_trace), C.POINTER(rt_sim_out), P]
    L.rt_goodput.argtypes = [P, C.POINTER(rt_trace), C.POINTER(rt_sim_out), P, P, P]
    L.rt_sim_data_status.argtypes = [P, P, C.POINTER(C.c_uint32)]
    L.rt_sim_timing.argtypes = [P, C.c_int32]
    L.rt_sim_kernel_time.argtypes = [P, C.POINTER(C.c_double), C.POINTER(C.c_int64)]
    L.rt_score_argmin.argtypes = [C.POINTER(rt_router_params), C.c_int32, C.c_int32, P, P, P, C.c_int32,
                                  C.c_int64, C.c_int64, P, P, P, P, P, P]
    L.rt_last_error.argtypes = []
    L.rt_last_error.restype = C.c_char_p
    for name in EXPORTS[:-1]:
        getattr(L, name).restype = C.c_int
    return L


_lib = _load()


def library_path() -> str:
    return LIB_PATH


def rt_last_error() -> str:
    return _lib.rt_last_error().decode()


def _check(status: int):
    if status != RT_OK:
        raise RtError(status, rt_last_error())


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return stream


def _dptr(t: Optional[torch.Tensor], dtype: torch.dtype, name: str):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr() if t.numel() > 0 else None


def router_params(d: Dict) -> rt_router_params:
    r = rt_router_params()
    for k in ("w_b", "w_s", "w_q", "rho", "tau_pre_s", "tau_dec_s", "pre_base_s"):
        setattr(r, k, float(d[k]))
    sg = list(d["sigma"]) + [1.0] * (RT_MAX_CLASSES - len(d["sigma"]))
    for i in range(RT_MAX_CLASSES):
        r.sigma[i] = float(sg[i])
    return r


def point(d: Dict) -> rt_point:
    """rt_point from a parameter-point dictionary (workload.make_point keys)."""
    p = rt_point()
    p.n_prefill, p.n_decode, p.n_classes = int(d["n_prefill"]), int(d["n_decode"]), int(d["n_classes"])
    p.policy = RT_POLICY[d["policy"]] if isinstance(d["policy"], str) else int(d["policy"])
    p.backlog_mode = RT_BACKLOG[d["backlog_mode"]] if isinstance(d["backlog_mode"], str) else int(d["backlog_mode"])
    p.router = router_params(d)
    for k in ("pre_base_ns", "pre_tok_ns", "dec_tok_ns", "xfer_tok_ns", "kv_cap_pre", "kv_cap_dec"):
        setattr(p.phys, k, int(d[k]))
    for i in range(RT_MAX_CLASSES):
        p.phys.slo_ttft_ns[i] = int(d["slo_ttft_ns"][i])
        p.phys.slo_tpot_ns[i] = int(d["slo_tpot_ns"][i])
    p.len_threshold = int(d.get("len_threshold", 1))
    sv = d.get("service", "serial")
    p.service = RT_SERVICE[sv] if isinstance(sv, str) else int(sv)
    p.beta_pre = float(d.get("beta_pre", 0.0))
    p.beta_dec = float(d.get("beta_dec", 0.0))
    p.batch_cap = int(d.get("batch_cap", 0))
    p.reserved = 0
    return p


def rt_sim_create(points: Sequence[Dict], device: int = 0) -> int:
    arr = (rt_point * len(points))(*[point(d) for d in points])
    h = C.c_void_p()
    _check(_lib.rt_sim_create(arr, len(points), int(device), C.byref(h)))
    return h.value


def rt_sim_destroy(sim: int) -> None:
    _check(_lib.rt_sim_destroy(sim))


def _trace_struct(tr: Dict[str, torch.Tensor]) -> rt_trace:
    t = rt_trace()
    t.n_replicas = int(tr["offsets"].numel()) - 1
    t.n_requests = int(tr["arrival_ns"].numel())
    t.offsets = _dptr(tr["offsets"], torch.int64, "offsets")
    t.param_point = _dptr(tr.get("param_point"), torch.int32, "param_point")
    t.arrival_ns = _dptr(tr["arrival_ns"], torch.int64, "arrival_ns")
    t.prompt_len = _dptr(tr["prompt_len"], torch.int32, "prompt_len")
    t.out_len = _dptr(tr["out_len"], torch.int32, "out_len")
    t.pred_out_len = _dptr(tr["pred_out_len"], torch.int32, "pred_out_len")
    t.slo_class = _dptr(tr["slo_class"], torch.uint8, "slo_class")
    # [n_requests, 4] candidate words; torch has no general uint32 tensor, so
    # they travel as int32 with the same bits
    sb = tr.get("sample_bits")
    if sb is not None and sb.dim() != 2:
        raise ValueError("sample_bits must have shape [n_requests, 4]")
    if sb is not None and (sb.shape[1] != 4 or sb.shape[0] != t.n_requests):
        raise ValueError("sample_bits must have shape [n_requests, 4]")
    t.sample_bits = _dptr(sb, torch.int32, "sample_bits")
    return t


def _out_struct(out: Dict[str, torch.Tensor]) -> rt_sim_out:
    o = rt_sim_out()
    o.i_pre = _dptr(out["i_pre"], torch.int32, "i_pre")
    o.i_dec = _dptr(out["i_dec"], torch.int32, "i_dec")
    o.ttft_ns = _dptr(out["ttft_ns"], torch.int64, "ttft_ns")
    o.decode_span_ns = _dptr(out["decode_span_ns"], torch.int64, "decode_span_ns")
    return o


def rt_sim_run_replicas(sim: int, trace: Dict[str, torch.Tensor], out: Dict[str, torch.Tensor], stream=None) -> None:
    t, o = _trace_struct(trace), _out_struct(out)
    _check(_lib.rt_sim_run_replicas(sim, C.byref(t), C.byref(o), _stream(stream)))


def rt_sim_run_replicas_noalloc(sim: int, trace: Dict[str, torch.Tensor], out: Dict[str, torch.Tensor],
                                stream=None) -> None:
    t, o = _trace_struct(trace), _out_struct(out)
    _check(_lib.rt_sim_run_replicas_noalloc(sim, C.byref(t), C.byref(o), _stream(stream)))


def rt_goodput(sim: int, trace: Dict[str, torch.Tensor], out: Dict[str, torch.Tensor], goodput: torch.Tensor,
               met: Optional[torch.Tensor] = None, stream=None) -> None:
    t, o = _trace_struct(trace), _out_struct(out)
    _check(_lib.rt_goodput(sim, C.byref(t), C.byref(o), _dptr(goodput, torch.float64, "goodput"),
                           _dptr(met, torch.int64, "met"), _stream(stream)))


def rt_sim_data_status(sim: int, stream=None, raise_on_data: bool = False) -> int:
    f = C.c_uint32()
    st = _lib.rt_sim_data_status(sim, _stream(stream), C.byref(f))
    if st not in (RT_OK, RT_EDATA) or (st == RT_EDATA and raise_on_data):
        _check(st)
    return int(f.value)


def rt_sim_timing(sim: int, enable: bool) -> None:
    _check(_lib.rt_sim_timing(sim, 1 if enable else 0))


def rt_sim_kernel_time(sim: int):
    """(total milliseconds, timed calls) of the simulation kernels since
    timing was enabled."""
    ms, n = C.c_double(), C.c_int64()
    _check(_lib.rt_sim_kernel_time(sim, C.byref(ms), C.byref(n)))
    return ms.value, n.value


def rt_score_argmin(params: Dict, pool: str, n_inst: int, backlog_s: torch.Tensor, queue: torch.Tensor,
                    kv_occ: torch.Tensor, kv_cap: int, inst_stride: int, n_req: int, prompt_len: torch.Tensor,
                    pred_out_len: Optional[torch.Tensor], slo_class: torch.Tensor, out_idx: torch.Tensor,
                    out_score: torch.Tensor, stream=None) -> None:
    prm = router_params(params)
    _check(_lib.rt_score_argmin(
        C.byref(prm), RT_POOL[pool] if isinstance(pool, str) else int(pool), int(n_inst),
        _dptr(backlog_s, torch.float32, "backlog_s"), _dptr(queue, torch.int32, "queue"),
        _dptr(kv_occ, torch.int32, "kv_occ"), int(kv_cap), int(inst_stride), int(n_req),
        _dptr(prompt_len, torch.int32, "prompt_len"), _dptr(pred_out_len, torch.int32, "pred_out_len"),
        _dptr(slo_class, torch.uint8, "slo_class"), _dptr(out_idx, torch.int32, "out_idx"),
        _dptr(out_score, torch.float32, "out_score"), _stream(stream)))


# ---------------------------------------------------------------------------
# Conveniences (memory handling around the ABI calls; no computation)
# ---------------------------------------------------------------------------
TRACE_KEYS = ("offsets", "param_point", "arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class")
OUT_KEYS = ("i_pre", "i_dec", "ttft_ns", "decode_span_ns")


def to_device(trace_np: Dict, device="cuda") -> Dict[str, torch.Tensor]:
    """Copy a numpy SoA trace to GPU tensors (the candidate words of the
    sampled policy, if present, as int32 with the same bits)."""
    out = {k: torch.from_numpy(trace_np[k]).to(device) for k in TRACE_KEYS if k in trace_np}
    if "sample_bits" in trace_np:
        out["sample_bits"] = torch.from_numpy(trace_np["sample_bits"].view(np.int32)).to(device)
    return out


def alloc_outputs(n_requests: int, device="cuda") -> Dict[str, torch.Tensor]:
    return dict(i_pre=torch.empty(n_requests, dtype=torch.int32, device=device),
                i_dec=torch.empty(n_requests, dtype=torch.int32, device=device),
                ttft_ns=torch.empty(n_requests, dtype=torch.int64, device=device),
                decode_span_ns=torch.empty(n_requests, dtype=torch.int64, device=device))


class Simulator:
    """Owns an rt_sim handle for a list of parameter points."""

    def __init__(self, points: Sequence[Dict], device: int = 0):
        self.points = list(points)
        self.device = device
        self.handle = rt_sim_create(self.points, device)

    def close(self):
        if self.handle:
            rt_sim_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def run(self, trace: Dict[str, torch.Tensor], out: Optional[Dict[str, torch.Tensor]] = None, stream=None):
        if out is None:
            out = alloc_outputs(trace["arrival_ns"].numel(), trace["arrival_ns"].device)
        rt_sim_run_replicas(self.handle, trace, out, stream)
        return out

    def goodput(self, trace, out, stream=None):
        n = trace["offsets"].numel() - 1
        g = torch.empty(n, dtype=torch.float64, device=trace["offsets"].device)
        met = torch.empty(n, dtype=torch.int64, device=trace["offsets"].device)
        rt_goodput(self.handle, trace, out, g, met, stream)
        return g, met

    def data_status(self, stream=None) -> int:
        return rt_sim_data_status(self.handle, stream)
