"""The allocation-free entry point (rt_sim_run_replicas_noalloc) against
rt_sim_run_replicas through the C ABI: outputs bit for bit on two calls in a
row, the second on a smaller input (the fixed scratch then holds the first
call's records), with every scoring mode and a multi-wave pool in each call;
and its limits, returned before anything is launched."""
import ctypes as C

import numpy as np
import pytest
import torch

from paper_2609_16206_amd import rt_router as R
from paper_2609_16206_amd import workload as W
from tests.gpu_common import log

pytestmark = pytest.mark.gpu

OUT_KEYS = ("i_pre", "i_dec", "ttft_ns", "decode_span_ns")


def _points():
    return [W.make_point(2, 6, n_classes=3),
            W.make_point(3, 9, n_classes=3, backlog_mode="proxy"),
            W.make_point(2, 4, n_classes=3, policy="round_robin"),
            W.make_point(4, 12, n_classes=3, policy="learned_sampled"),
            W.make_point(40, 300, n_classes=3),
            W.make_point(1, 1, n_classes=3, policy="length_threshold")]


def _trace(pts, lengths, seed):
    parts, pp = [], []
    tr0 = W.mixed_bursty()
    for i, n in enumerate(lengths):
        pid = i % len(pts)
        traf = tr0.scaled(W.capacity_rps(pts[pid], tr0) / tr0.mean_rate())
        parts.append(W.replica_arrays(seed, i, traf, n))
        pp.append(pid)
    keys = ("arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class")
    tr = {k: np.concatenate([q[k] for q in parts]) for k in keys}
    tr["offsets"] = np.concatenate(([0], np.cumsum(lengths))).astype(np.int64)
    tr["param_point"] = np.array(pp, np.int32)
    W.add_sample_words(tr, seed)
    return tr


def _run(sim, dtr, fn):
    out = R.alloc_outputs(int(dtr["arrival_ns"].numel()), "cuda")
    for v in out.values():
        v.fill_(-7)
    fn(sim.handle, dtr, out)
    g, met = sim.goodput(dtr, out)
    flags = sim.data_status()
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}, g.cpu().numpy(), met.cpu().numpy(), flags


def test_noalloc_matches_run_replicas_on_two_calls():
    pts = _points()
    sim = R.Simulator(pts)
    try:
        for call, (lengths, seed) in enumerate((([0, 1, 63, 64, 65, 3000, 4097, 7000, 2, 1500] * 12, 41),
                                                ([5, 300, 0, 1000, 17, 2500] * 3, 42))):
            tr = _trace(pts, lengths, seed)
            dtr = R.to_device(tr, "cuda")
            ref, gr, mr, fr = _run(sim, dtr, R.rt_sim_run_replicas)
            got, gg, mg, fg = _run(sim, dtr, R.rt_sim_run_replicas_noalloc)
            assert fr == 0 and fg == 0
            for k in OUT_KEYS:
                assert np.array_equal(ref[k], got[k]), (call, k)
            assert np.array_equal(gr, gg) and np.array_equal(mr, mg), call
            assert np.all(got["ttft_ns"] >= 0)
            log(f"no-alloc call {call + 1}: {len(lengths)} replicas, {tr['arrival_ns'].size} requests, "
                f"identical to rt_sim_run_replicas (mean goodput {gg.mean():.4f})")
    finally:
        sim.close()


def test_noalloc_limits_are_returned_before_launch():
    pts = _points()
    sim = R.Simulator(pts)
    bsim = R.Simulator([dict(W.make_point(2, 4, n_classes=3), service="batched", beta_pre=W.BATCH_BETA,
                             beta_dec=W.BATCH_BETA)])
    try:
        # more scratch than the fixed array holds: 2^20 requests of a call
        # that holds both record sizes need 192 MiB
        n = 1 << 20
        tr = _trace(pts[:2], [n // 2, n // 2], 43)
        dtr = R.to_device(tr, "cuda")
        out = R.alloc_outputs(n, "cuda")
        with pytest.raises(R.RtError) as ei:
            R.rt_sim_run_replicas_noalloc(sim.handle, dtr, out)
        assert ei.value.status == R.RT_ERANGE and "scratch" in str(ei.value)
        # too many replicas (one request each)
        many = 65537
        tr = dict(arrival_ns=np.zeros(many, np.int64), prompt_len=np.full(many, 10, np.int32),
                  out_len=np.full(many, 10, np.int32), pred_out_len=np.full(many, 10, np.int32),
                  slo_class=np.zeros(many, np.uint8), offsets=np.arange(many + 1, dtype=np.int64),
                  param_point=np.zeros(many, np.int32))
        dtr = R.to_device(tr, "cuda")
        out = R.alloc_outputs(many, "cuda")
        with pytest.raises(R.RtError) as ei:
            R.rt_sim_run_replicas_noalloc(sim.handle, dtr, out)
        assert ei.value.status == R.RT_ERANGE
        # continuous batching is not served by this entry point
        tr = _trace([W.make_point(2, 4, n_classes=3)], [100], 45)
        dtr = R.to_device(tr, "cuda")
        out = R.alloc_outputs(100, "cuda")
        with pytest.raises(R.RtError) as ei:
            R.rt_sim_run_replicas_noalloc(bsim.handle, dtr, out)
        assert ei.value.status == R.RT_EUNSUPPORTED
        # nothing was launched by the refused calls: the simulator still works
        ref, _, _, fr = _run(sim, R.to_device(_trace(pts, [500] * 6, 46), "cuda"), R.rt_sim_run_replicas_noalloc)
        assert fr == 0 and np.all(ref["ttft_ns"] >= 0)
    finally:
        sim.close()
        bsim.close()
