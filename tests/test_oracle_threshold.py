"""Pins of the oracle's predicted-length threshold baseline (Section IV-C
names it without a rule; the reading is size-interval assignment: the
decode pool's lower part serves requests predicted short, its upper part
those predicted long, least loaded within the part).  CPU only.

What fixes it, beyond the oracle's own code:
  * with two decode instances the decode placement is exactly
    [o^_r >= threshold] (closed form);
  * prefill placements do not depend on decode placements in this model,
    so they equal the least-loaded policy's exactly;
  * every decode placement lies in the part its predicted length picks;
  * the event-heap simulation agrees on random tiny traces (in
    test_oracle_sim.test_event_heap_bruteforce_agrees).
"""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2609_16206_amd import workload as W

KEYS = ("arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class")


def _replicas(P, D, n=3000, reps=2, seed=11, scale=1.2, **kw):
    pt = W.make_point(P, D, n_classes=3, **kw)
    wl = W.Workload("t", seed, reps, n, [pt], [W.mixed_bursty().scaled(scale)])
    tr = W.make_trace(wl)
    for i in range(reps):
        sl = slice(int(tr["offsets"][i]), int(tr["offsets"][i + 1]))
        yield [tr[k][sl] for k in KEYS]


@pytest.mark.parametrize("thr", [1, 64, 300, 1 << 30])
def test_two_decode_instances_closed_form(thr):
    pt = W.make_point(2, 2, n_classes=3, policy="length_threshold", len_threshold=thr)
    for args in _replicas(2, 2):
        out, st = O.sim_replica(pt, *args)
        assert st["violations"] == 0
        assert np.array_equal(out["i_dec"], (args[3] >= thr).astype(np.int32))


def test_one_decode_instance_takes_everything():
    pt = W.make_point(3, 1, n_classes=3, policy="length_threshold", len_threshold=100)
    for args in _replicas(3, 1):
        out, _ = O.sim_replica(pt, *args)
        assert np.all(out["i_dec"] == 0)


@pytest.mark.parametrize("P,D", [(2, 6), (3, 5), (1, 9)])
def test_prefill_is_least_loaded_and_parts_hold(P, D):
    thr = 256
    pt = W.make_point(P, D, n_classes=3, policy="length_threshold", len_threshold=thr)
    jsq = W.make_point(P, D, n_classes=3, policy="least_loaded")
    half = (D + 1) // 2
    for args in _replicas(P, D):
        out, st = O.sim_replica(pt, *args)
        ref, _ = O.sim_replica(jsq, *args)
        assert st["violations"] == 0
        assert np.array_equal(out["i_pre"], ref["i_pre"])
        assert np.array_equal(out["ttft_ns"], ref["ttft_ns"])   # prefill side is the same system
        lng = args[3] >= thr
        assert np.all(out["i_dec"][lng] >= half) and np.all(out["i_dec"][~lng] < half)
        assert lng.any() and (~lng).any()


def test_threshold_must_be_positive():
    pt = W.make_point(2, 3, policy="length_threshold", len_threshold=0)
    z = np.zeros(2, np.int64)
    o = np.ones(2, np.int32)
    with pytest.raises(ValueError):
        O.sim_replica(pt, z, o, o, o, np.zeros(2, np.uint8))
