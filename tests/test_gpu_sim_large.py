"""Full-size sweep (65,536 replicas x 5,000 requests over 1,225 points) and
large pool (256 replicas x 1,000,000 requests, 128 prefill + 1,024 decode)
on the GPU, each in the launch the benchmark times (every replica in one
call).  The oracle checks one replica of every sweep point in full, and 64 of
the 256 large-pool replicas in full (every fourth, 1,000,000 requests each);
properties and goodput recounts cover every replica."""
import numpy as np
import pytest

from paper_2609_16206_amd import workload as W
from tests.gpu_common import log, run_sim
from tests.parity import check_properties, follow_replicas, goodput_recount

pytestmark = pytest.mark.gpu


def test_sweep_full_size():
    wl = W.param_sweep()
    tr = W.make_trace(wl)
    log(f"sweep trace: {tr['arrival_ns'].size} requests")
    gpu, g, met, flags = run_sim(wl.points, tr)
    assert flags == 0
    check_properties(wl.points, tr, gpu)
    assert np.array_equal(goodput_recount(wl.points, tr, gpu), met)
    rep = follow_replicas(wl.points, tr, gpu, range(1225), gpu_goodput=g, gpu_met=met)
    rep2 = follow_replicas(wl.points, tr, gpu, range(65536 - 64, 65536), gpu_goodput=g, gpu_met=met)
    log(f"sweep 65536x5000: first 1225 {rep}; last 64 {rep2}")


def test_large_pool_full_size():
    wl = W.large_pool_wl()
    tr = W.make_trace(wl)
    log(f"large trace: {tr['arrival_ns'].size} requests")
    gpu, g, met, flags = run_sim(wl.points, tr)
    assert flags == 0
    check_properties(wl.points, tr, gpu)
    assert np.array_equal(goodput_recount(wl.points, tr, gpu), met)
    sample = list(range(0, wl.n_replicas, 4))
    assert len(sample) == 64
    total = dict(replicas=0, requests=0, near_ties=0, close_decisions=0)
    for k in range(0, len(sample), 16):
        rep = follow_replicas(wl.points, tr, gpu, sample[k:k + 16], gpu_goodput=g, gpu_met=met)
        for key in total:
            total[key] += rep[key]
        log(f"large 256x1e6: replicas {sample[k]}..{sample[min(k + 15, len(sample) - 1)]} in full: {rep}")
    log(f"large 256x1e6: {total['replicas']} full replicas ({total['requests']} requests) bitwise in follow mode, "
        f"{total['near_ties']} near ties, {total['close_decisions']} close decisions; mean goodput {g.mean():.4f}")
