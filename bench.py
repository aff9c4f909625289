"""Throughput of the replica-batched router simulation on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
rt_sim_run_replicas (every replica: release, score both pools, argmin,
serve, record) followed by rt_goodput (per-replica SLO attainment).  The
default workload is the largest single-GPU configuration, the large pool:
256 replicas x 1,000,000 requests, 128 prefill + 1,024 decode instances,
Poisson arrivals at 0.95 of capacity, Pareto output lengths, learned router
with the simulation-clock backlog (294.9 G scored pairs per step).

Prints one JSON line: simulated requests/s over K timed steps (inputs
resident in HBM), the dominant kernel's roofline position measured with HIP
events on its own stream, and the CPU oracle's rate on the host cores.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

METRIC = "simulated requests/sec and scored pairs/sec (1 GPU); % of roofline"
HBM_PEAK = 8.0e12  # B/s, MI355X HBM3E
# Plain VALU lane-op peak: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz (one
# non-fused, non-packed op per lane per clock).
ALU_PEAK = 256 * 4 * 16 * 2.4e9
# Algorithmic work per unit, as the scope analysis counts it: about 12 VALU
# lane-ops per scored pair (int add, 2 conversions, 7 fp32 ops,
# compare/select, the release compare) and about 40 of bookkeeping per
# request; 10 per pair for the standalone scorer, whose backlog is given.
SIM_BYTES_PER_REQ = 21 + 24  # trace in (i64 + 3 x i32 + u8), outputs out (2 x i32 + 2 x i64)
SAMPLE_BYTES_PER_REQ = 16  # the sampled policy's four candidate words
SIM_OPS_PER_PAIR = 12
SIM_OPS_PER_REQ = 40
SCORE_OPS_PER_PAIR = 10
SCORE_OPS_PER_REQ = 0
# The design notes' own recount of the written arithmetic (reported beside
# the fraction above, labelled): backlog 4, press 3, factor 2, size 2, load 2,
# queue 2, sums 2, argmin 1, release 1 = 19 per pair and 25 per request; the
# scorer 14 per pair and 4 per request.
RECOUNT_SIM = (19, 25)
RECOUNT_SCORE = (14, 4)
SCORE_BYTES_PER_REQ = 4 + 4 + 1 + 4 + 4  # p, o^, class in; index, score out
SCORE_BYTES_PER_PAIR_ROWS = 4 + 4 + 4  # per-request snapshot rows: backlog, queue, occupancy


def _workload(name):
    from paper_2609_16206_amd import workload as W
    if name == "tiny":
        return W.tiny_sim()
    if name == "cluster":
        return W.paper_cluster()
    if name == "cluster_sampled":
        return W.paper_cluster(policy="learned_sampled")
    if name == "cluster_batched":
        return W.paper_cluster(service="batched")
    if name == "cluster_batched_wide":
        return W.paper_cluster(n_replicas=65536, requests=2000, service="batched")
    if name == "sweep":
        return W.param_sweep()
    if name == "large":
        return W.large_pool_wl()
    if name == "batched_wide_pool":
        return W.batched_wide_pool()
    raise SystemExit(f"unknown workload {name}")


def _source_hash(files):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


SIM_SOURCES = ["paper_2609_16206_amd/csrc/" + f for f in (
    "seg_kernel.h", "wseg_kernel.h", "seg_true.hip", "seg_proxy.hip", "seg_base.hip", "seg_true_s.hip", "seg_proxy_s.hip", "seg_classes.hip",
    "lane_ops.h", "rt_internal.h", "api.hip")]
BAT_SOURCES = ["paper_2609_16206_amd/csrc/" + f for f in ("bat_kernel.hip", "lane_ops.h", "rt_internal.h", "api.hip", "seg_classes.hip")]
SCORE_SOURCES = ["paper_2609_16206_amd/csrc/score_kernel.hip", "paper_2609_16206_amd/csrc/rt_internal.h"]


def _traffic(kernel_tag, workload_name, sources):
    """HBM bytes per launch from the committed counter summary, if it was
    taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel_tag}_{workload_name}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("source_sha") != _source_hash(sources):
        return None
    return d.get("bytes_per_launch")


def _valu_busy(kernel_tag, workload_name, sources):
    """Measured VALU issue share of the dominant kernel(s) from the committed
    counter summary (VALUBusy, percent, one entry per kernel class the call
    launches), if it was taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"valu_{kernel_tag}_{workload_name}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("source_sha") != _source_hash(sources):
        return None
    return d.get("valu_busy_pct")


def cpu_threads():
    """Threads for the oracle's baseline: the cores this process may run on,
    capped by OMP_NUM_THREADS where the host sets the job's CPU share."""
    n = len(os.sched_getaffinity(0))
    share = os.environ.get("OMP_NUM_THREADS")
    if share and share.isdigit() and int(share) > 0:
        n = min(n, int(share))
    return max(1, n)


def _cpu_baseline_sim(wl, tr, budget_s):
    from oracle import oracle as O
    threads = cpu_threads()
    off = tr["offsets"]
    n_rep = len(off) - 1
    done_req = 0
    done_rep = 0
    pairs = 0
    t0 = time.perf_counter()
    chunk = max(1, threads)
    while done_rep < n_rep and time.perf_counter() - t0 < budget_s:
        reps = list(range(done_rep, min(n_rep, done_rep + chunk)))
        O.sim_trace(wl.points, tr, replicas=reps, threads=threads)
        for i in reps:
            n = int(off[i + 1] - off[i])
            pt = wl.points[int(tr["param_point"][i])]
            done_req += n
            pairs += n * (pt["n_prefill"] + pt["n_decode"])
        done_rep += len(reps)
        chunk = min(4 * chunk, 1024)
    dt = time.perf_counter() - t0
    return dict(value=done_req / dt, unit="requests/s", cores=threads, kind="oracle",
                pairs_per_s=pairs / dt,
                sample=f"{done_rep} of {n_rep} replicas ({done_req} requests), {threads} threads "
                       f"(affinity {len(os.sched_getaffinity(0))} cores), {dt:.1f} s")


def bench_sim(args):
    import torch
    from paper_2609_16206_amd import rt_router as R
    from paper_2609_16206_amd import workload as W

    wl = _workload(args.workload)
    t_gen = time.perf_counter()
    tr = W.make_trace(wl)
    t_gen = time.perf_counter() - t_gen
    n_req = int(tr["arrival_ns"].size)
    counts = np.diff(tr["offsets"])
    widths = np.array([p["n_prefill"] + p["n_decode"] for p in wl.points], np.int64)
    n_pairs = int(np.sum(counts * widths[tr["param_point"]]))

    torch.cuda.set_device(0)
    dev = "cuda:0"
    sim = R.Simulator(wl.points, device=0)
    dtr = R.to_device(tr, dev)
    out = R.alloc_outputs(n_req, dev)
    g = torch.empty(wl.n_replicas, dtype=torch.float64, device=dev)
    met = torch.empty(wl.n_replicas, dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        R.rt_sim_run_replicas(sim.handle, dtr, out, stream)
        R.rt_goodput(sim.handle, dtr, out, g, met, stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    R.rt_sim_timing(sim.handle, True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    kern_ms, calls = R.rt_sim_kernel_time(sim.handle)
    R.rt_sim_timing(sim.handle, False)
    flags = sim.data_status()
    mean_goodput = float(g.mean().item())
    sim.close()

    ms_step = dt * 1e3 / args.steps
    value = n_req * args.steps / dt
    kernel_s = kern_ms * 1e-3 / max(1, calls)
    alg_bytes = n_req * (SIM_BYTES_PER_REQ + (SAMPLE_BYTES_PER_REQ if "sample_bits" in tr else 0))
    alg_ops = n_pairs * SIM_OPS_PER_PAIR + n_req * SIM_OPS_PER_REQ
    t_hbm, t_alu = alg_bytes / HBM_PEAK, alg_ops / ALU_PEAK
    if t_hbm >= t_alu:
        roof = dict(bound="hbm", achieved=alg_bytes / kernel_s / 1e9, peak=HBM_PEAK / 1e9, unit="GB/s")
    else:
        roof = dict(bound="alu", achieved=alg_ops / kernel_s / 1e12, peak=ALU_PEAK / 1e12, unit="Tlane-op/s")
    roof["frac"] = roof["achieved"] / roof["peak"]
    rc_ops = n_pairs * RECOUNT_SIM[0] + n_req * RECOUNT_SIM[1]
    roof["frac_alu_recount"] = rc_ops / kernel_s / ALU_PEAK
    batched = any(p.get("service") == "batched" for p in wl.points)
    roof["traffic"] = _traffic("bat", args.workload, BAT_SOURCES) if batched else _traffic("sim", args.workload,
                                                                                          SIM_SOURCES)
    roof["valu_busy_pct"] = (_valu_busy("bat", args.workload, BAT_SOURCES) if batched else
                             _valu_busy("sim", args.workload, SIM_SOURCES))
    roof["kernel"] = ("rt::bat::bseg_kernel / bat_kernel (the batched classes the call launches)" if batched else
                      "rt::seg::seg_kernel / wseg_kernel (every class one rt_sim_run_replicas call launches)")
    roof["per_unit"] = (f"{SIM_BYTES_PER_REQ} B/request; {SIM_OPS_PER_PAIR} lane-ops/pair + {SIM_OPS_PER_REQ}/request "
                        f"(recount {RECOUNT_SIM[0]}/pair + {RECOUNT_SIM[1]}/request)")
    roof["kernel_ms"] = kernel_s * 1e3
    roof["alg_bytes"] = alg_bytes
    roof["alg_lane_ops"] = alg_ops

    pt = wl.points[0]
    res = dict(metric=METRIC, value=value, unit="requests/s", n_gpus=1, steps=args.steps, warmup=args.warmup,
               ms_per_step=ms_step, higher_is_better=True, scaling="weak", vs_baseline=None, dtype="f32",
               data="synthetic",
               config=dict(workload=wl.name, replicas=wl.n_replicas, requests_per_replica=wl.requests,
                           points=len(wl.points), prefill=pt["n_prefill"] if len(wl.points) == 1 else "mixed",
                           decode=pt["n_decode"] if len(wl.points) == 1 else "mixed",
                           policy=pt["policy"], backlog=pt["backlog_mode"], service=pt.get("service", "serial")),
               pairs_per_s=n_pairs * args.steps / dt, requests=n_req, pairs=n_pairs, mean_goodput=mean_goodput,
               data_flags=flags, roofline=roof, trace_gen_s=t_gen)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = _cpu_baseline_sim(wl, tr, args.cpu_budget)
    return res


def bench_scorer(args, rows=False):
    """The standalone scorer: 2^20 requests x 64 decode instances against one
    shared snapshot (ALU-bound), or with a snapshot row per request
    (``rows``: 12 B per pair read, HBM-bound)."""
    import torch
    from oracle import oracle as O
    from paper_2609_16206_amd import rt_router as R
    from paper_2609_16206_amd import workload as W

    n_req, n_inst = 1 << 20, 64
    d = W.scorer_inputs(n_req=n_req, n_inst=n_inst, seed=1, per_request=rows)
    stride = d["inst_stride"]
    prm = W.scorer_params()
    torch.cuda.set_device(0)
    t = {k: torch.from_numpy(d[k]).cuda() for k in ("backlog_s", "queue", "kv_occ", "prompt_len", "pred_out_len",
                                                   "slo_class")}
    idx = torch.empty(n_req, dtype=torch.int32, device="cuda")
    sc = torch.empty(n_req, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()

    def step():
        R.rt_score_argmin(prm, "decode", n_inst, t["backlog_s"], t["queue"], t["kv_occ"], d["kv_cap"], stride, n_req,
                          t["prompt_len"], t["pred_out_len"], t["slo_class"], idx, sc, stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    kernel_s = ev0.elapsed_time(ev1) * 1e-3 / args.steps
    pairs = n_req * n_inst
    alg_bytes = n_req * SCORE_BYTES_PER_REQ + (pairs * SCORE_BYTES_PER_PAIR_ROWS if rows else 0)
    alg_ops = pairs * SCORE_OPS_PER_PAIR + n_req * SCORE_OPS_PER_REQ
    if rows:
        roof = dict(bound="hbm", achieved=alg_bytes / kernel_s / 1e9, peak=HBM_PEAK / 1e9, unit="GB/s")
        roof["traffic"] = _traffic("score", "scorer_rows", SCORE_SOURCES)
        roof["valu_busy_pct"] = _valu_busy("score", "scorer_rows", SCORE_SOURCES)
        roof["kernel"] = "rt::score_rows16_kernel"
        roof["per_unit"] = (f"{SCORE_BYTES_PER_PAIR_ROWS} B/pair + {SCORE_BYTES_PER_REQ} B/request")
    else:
        roof = dict(bound="alu", achieved=alg_ops / kernel_s / 1e12, peak=ALU_PEAK / 1e12, unit="Tlane-op/s")
        roof["traffic"] = _traffic("score", "scorer", SCORE_SOURCES)
        roof["valu_busy_pct"] = _valu_busy("score", "scorer", SCORE_SOURCES)
        roof["kernel"] = "rt::score_shared_kernel"
        roof["per_unit"] = (f"{SCORE_OPS_PER_PAIR} lane-ops/pair (recount {RECOUNT_SCORE[0]}/pair + "
                            f"{RECOUNT_SCORE[1]}/request)")
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["frac_alu_recount"] = (pairs * RECOUNT_SCORE[0] + n_req * RECOUNT_SCORE[1]) / kernel_s / ALU_PEAK
    roof["kernel_ms"] = kernel_s * 1e3
    wname = f"scorer-{n_req}x{n_inst}-" + ("per-request" if rows else "shared")
    res = dict(metric=METRIC, value=n_req * args.steps / dt, unit="requests/s", n_gpus=1, steps=args.steps,
               warmup=args.warmup, ms_per_step=dt * 1e3 / args.steps, higher_is_better=True, scaling="weak",
               vs_baseline=None, dtype="f32", data="synthetic",
               config=dict(workload=wname, requests=n_req, instances=n_inst, inst_stride=stride),
               pairs_per_s=pairs * args.steps / dt, roofline=roof)
    if not args.no_cpu_baseline:
        threads = 1
        m = 1 << 17
        t0 = time.perf_counter()
        rl = slice(0, m * stride if rows else None)
        O.score(prm, "decode", d["backlog_s"][rl], d["queue"][rl], d["kv_occ"][rl], d["kv_cap"], n_inst, stride,
                d["prompt_len"][:m], d["pred_out_len"][:m], d["slo_class"][:m])
        dtc = time.perf_counter() - t0
        res["cpu_baseline"] = dict(value=m / dtc, unit="requests/s", cores=threads, kind="oracle",
                                   pairs_per_s=m * n_inst / dtc,
                                   sample=f"first {m} of {n_req} requests x {n_inst} instances, 1 thread")
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="large",
                    choices=["large", "tiny", "cluster", "cluster_sampled", "cluster_batched", "cluster_batched_wide",
                             "batched_wide_pool", "sweep", "scorer", "scorer_rows"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle time for the CPU baseline")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="first copy MIB MiB device-to-device (a plain copy of known size that scales the "
                         "hardware byte counters when the run is profiled)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps(dict(error="bench.py measures one GPU: replicas are independent and would shard "
                                    "across GPUs with no exchange, but only --gpus 1 is run")), flush=True)
        sys.exit(2)
    if args.calibrate_copy > 0:
        import torch
        n = args.calibrate_copy << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if args.workload in ("scorer", "scorer_rows"):
        res = bench_scorer(args, rows=args.workload == "scorer_rows")
    else:
        res = bench_sim(args)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
