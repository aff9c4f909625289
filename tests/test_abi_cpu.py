"""The C-ABI library without a GPU: it loads, exports every symbol the header
declares, the binding's structs match the header's layout, and argument
errors are returned synchronously, before anything touches the device."""
import ctypes as C
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rt_router.h")


@pytest.fixture(scope="module")
def rt():
    from paper_2609_16206_amd import build as b
    if not os.path.exists(b.LIB):
        b.build()
    from paper_2609_16206_amd import rt_router
    return rt_router


def _declared():
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:rt_status|const char\*)\s+(rt_\w+)\s*\(", txt, re.M)))


def test_every_declared_symbol_is_exported(rt):
    names = _declared()
    assert set(names) == set(rt.EXPORTS)
    lib = C.CDLL(rt.library_path())
    for n in names:
        assert hasattr(lib, n), n


def test_struct_layout_matches_header(rt, tmp_path):
    src = tmp_path / "layout.c"
    fields = {
        "rt_router_params": ["w_b", "tau_pre_s", "pre_base_s", "sigma"],
        "rt_physics": ["pre_base_ns", "kv_cap_dec", "slo_ttft_ns", "slo_tpot_ns"],
        "rt_point": ["n_prefill", "backlog_mode", "router", "phys", "len_threshold", "service", "beta_pre",
                     "beta_dec", "batch_cap", "reserved"],
        "rt_trace": ["n_replicas", "n_requests", "offsets", "param_point", "slo_class", "sample_bits"],
        "rt_sim_out": ["i_pre", "decode_span_ns"],
    }
    lines = ['#include <stdio.h>', '#include <stddef.h>', f'#include "{HEADER}"', "int main(void){"]
    for s, fs in fields.items():
        lines.append(f'printf("{s} %zu\\n", sizeof({s}));')
        for f in fs:
            lines.append(f'printf("{s}.{f} %zu\\n", offsetof({s}, {f}));')
    lines.append("return 0;}")
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", str(src), "-o", str(exe)], check=True)
    got = dict(l.split() for l in subprocess.run([str(exe)], capture_output=True, text=True).stdout.splitlines())
    for s, fs in fields.items():
        cls = getattr(rt, s)
        assert int(got[s]) == C.sizeof(cls), s
        for f in fs:
            assert int(got[f"{s}.{f}"]) == getattr(cls, f).offset, (s, f)


def _score(rt, prm, pool=1, n_inst=4, stride=0, n_req=0, kv_cap=100, arrays=False):
    p = C.c_void_p(1) if arrays else None
    return rt._lib.rt_score_argmin(prm, pool, n_inst, p, p, p, kv_cap, stride, n_req, p, p, p, p, p, None)


def test_scorer_argument_errors(rt):
    good = rt.router_params(dict(w_b=1, w_s=1, w_q=1e-3, rho=1, tau_pre_s=1e-5, tau_dec_s=1.8e-3,
                                 pre_base_s=5e-3, sigma=[2, 1.5]))
    prm = C.byref(good)
    assert _score(rt, None) == rt.RT_EINVAL
    assert "null params" in rt.rt_last_error()
    assert _score(rt, prm, pool=7) == rt.RT_EINVAL
    assert _score(rt, prm, n_inst=0) == rt.RT_EINVAL
    assert _score(rt, prm, n_inst=rt.RT_MAX_POOL + 1) == rt.RT_ERANGE
    assert _score(rt, prm, kv_cap=0) == rt.RT_EINVAL
    assert _score(rt, prm, n_inst=5, stride=3) == rt.RT_EINVAL
    assert _score(rt, prm, n_req=-1) == rt.RT_EINVAL
    assert _score(rt, prm, n_req=10) == rt.RT_EINVAL  # null arrays
    for field, bad in (("w_b", float("nan")), ("rho", -1.0), ("tau_dec_s", float("inf"))):
        b = rt.router_params(dict(w_b=1, w_s=1, w_q=1e-3, rho=1, tau_pre_s=1e-5, tau_dec_s=1.8e-3,
                                  pre_base_s=5e-3, sigma=[2, 1.5]))
        setattr(b, field, bad)
        assert _score(rt, C.byref(b)) == rt.RT_EINVAL, field
    b = rt.router_params(dict(w_b=1, w_s=1, w_q=1e-3, rho=1, tau_pre_s=1e-5, tau_dec_s=1.8e-3, pre_base_s=5e-3,
                              sigma=[2, -1.0]))
    assert _score(rt, C.byref(b)) == rt.RT_EINVAL
    # zero requests with valid arguments: nothing to do, nothing launched
    assert _score(rt, prm, n_req=0) == rt.RT_OK


def test_sim_argument_errors(rt):
    L = rt._lib
    h = C.c_void_p()
    assert L.rt_sim_create(None, 1, 0, C.byref(h)) == rt.RT_EINVAL
    pt = (rt.rt_point * 1)()
    assert L.rt_sim_create(pt, 0, 0, C.byref(h)) == rt.RT_EINVAL
    assert L.rt_sim_run_replicas(None, None, None, None) == rt.RT_EINVAL
    assert L.rt_sim_run_replicas_noalloc(None, None, None, None) == rt.RT_EINVAL
    assert L.rt_goodput(None, None, None, None, None, None) == rt.RT_EINVAL
    assert L.rt_sim_data_status(None, None, None) == rt.RT_EINVAL
    assert L.rt_sim_timing(None, 1) == rt.RT_EINVAL
    assert L.rt_sim_kernel_time(None, None, None) == rt.RT_EINVAL
    assert L.rt_sim_destroy(None) == rt.RT_OK


def test_binding_fails_loudly_without_library(tmp_path):
    """Importing the binding with the library absent raises (no fallback)."""
    code = "import sys; sys.path.insert(0, %r); import paper_2609_16206_amd.rt_router" % ROOT
    env = dict(os.environ, RT_ROUTER_LIB=str(tmp_path / "absent.so"))
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env)
    assert r.returncode != 0 and "librt_router.so is missing" in r.stderr


def test_pool_limit_agrees_with_header(rt):
    """The binding's pool limit is the header's: 1,024 instances per pool
    (the widest workload's decode pool; wider pools are rejected)."""
    m = re.search(r"#define\s+RT_MAX_POOL\s+(\d+)", open(HEADER).read())
    assert m and int(m.group(1)) == rt.RT_MAX_POOL == 1024
