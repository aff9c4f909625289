"""Seeded synthetic inputs for the disaggregated prefill/decode routing simulation.

This module only builds *inputs*: request traces (structure-of-arrays), the
per-point parameter records (cost constants, physics, SLO targets) and the
standalone-scorer snapshots.  It contains none of the routing method's
arithmetic (no scoring, no argmin, no queue simulation), so both the HIP path
and the CPU oracle can consume what it produces.

The paper evaluates on internal arrival traces that are not published
(Section IV-B, "three arrival traces"; Table I lists the four workload
families).  The generators here stand in for them with the shapes the study
describes: chat (short in / short out), reasoning (short in / long out), a
mixed bursty mixture driven by a two-state Markov-modulated Poisson process,
and heavy-tailed large-pool traffic.

Conventions
-----------
* all simulated times are integer nanoseconds (``int64``);
* lengths are ``int32`` tokens, ``clip(rint(x), lo, hi)`` of a continuous draw;
* the predicted output length stands in for the paper's swappable predictor
  (Section III-C): ``max(1, rint(o * exp(0.3 z)))``, i.e. true length times a
  lognormal(0, 0.3) error, as in the predictor-noise study (Section V-H);
* each replica draws from ``numpy.random.default_rng([config_seed, replica])``
  in a fixed order: mixture uniform, prompt normal, output draw, prediction
  normal, class uniform, then the arrival-process draws.  A replica can thus be
  regenerated alone, which is what range-resume and sampled parity rely on.
* every float parameter is stored already rounded to float32 (as a Python
  float holding an exactly representable value) so that any consumer that
  converts it to float32 obtains the same bits.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ProcessPoolExecutor
from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

MAX_CLASSES = 8

POLICIES = ("learned", "round_robin", "least_loaded", "learned_sampled", "length_threshold")
BACKLOG_MODES = ("true", "proxy")
SERVICES = ("serial", "batched")


def f32(x: float) -> float:
    """Round a Python float to the nearest float32 and return it as a float."""
    return float(np.float32(x))


# --------------------------------------------------------------------------
# Physics constant sets (Section VI, simulator vs measured A40 constants)
# --------------------------------------------------------------------------
# The simulator set: decode 0.0018 s/token, prefill base 0.005 s, 2048 KV
# bytes/token.  The paper gives neither a prefill per-token time nor a link
# bandwidth; the values below (1e-5 s/token, 25 GB/s) are readings of this
# library, not the paper's.
LINK_BYTES_PER_S = 25e9

SIM_PHYSICS = dict(
    pre_base_ns=5_000_000,
    pre_tok_ns=10_000,
    dec_tok_ns=1_800_000,
    kv_bytes_per_token=2048,
)
# The measured A40 set: decode 0.013237 s/token, prefill base 0.0667 s,
# 36864 KV bytes/token; prefill per-token 1e-4 s is again a reading.
A40_PHYSICS = dict(
    pre_base_ns=66_700_000,
    pre_tok_ns=100_000,
    dec_tok_ns=13_237_000,
    kv_bytes_per_token=36864,
)


# Continuous batching (Section VI): the measured decode curve is nearly flat,
# a batch of eight costing each request 2.9 % more per token, i.e. a factor
# 1 + beta (b - 1) with beta = 0.029 / 7 per extra batch member.  The paper
# gives no prefill curve; the same beta for prefill is a reading of this
# library.
BATCH_BETA = 0.029 / 7


def xfer_tok_ns(kv_bytes_per_token: int, link_bytes_per_s: float = LINK_BYTES_PER_S) -> int:
    """KV transfer delay per prompt token in ns (bytes/token over the link)."""
    return int(round(kv_bytes_per_token / link_bytes_per_s * 1e9))


def slo_targets(dec_tok_ns: int, n_classes: int):
    """Per-class (TTFT, TPOT) targets in ns.

    The tight targets are TTFT 175 ms / TPOT 39.7 ms and loose ones are 3x
    (Section IV-B, Protocol), derived from the same calibration as the router
    constants.  39.7 ms is three measured A40 decode steps (3 x 13.237 ms,
    Section VI), so the targets are expressed relative to the decode step:
    TPOT_c = 3 * dec_tok * 3^c and TTFT_c = round(175/39.7 * TPOT_0) * 3^c.
    Class 0 is the tightest class.
    """
    tpot0 = 3 * dec_tok_ns
    ttft0 = int(round(175.0 / 39.7 * tpot0))
    ttft = [0] * MAX_CLASSES
    tpot = [0] * MAX_CLASSES
    for c in range(n_classes):
        ttft[c] = ttft0 * 3 ** c
        tpot[c] = tpot0 * 3 ** c
    return ttft, tpot


def sigma_table(n_classes: int) -> List[float]:
    """SLO amplifier sigma(s) (Section III-A): larger for tighter classes.

    The paper gives no values; this library reads sigma_c = 1 + 3^-c, rounded to
    float32 once (2, 1.3333334, 1.1111112, 1.0370370, ...).
    """
    out = [1.0] * MAX_CLASSES
    for c in range(n_classes):
        out[c] = f32(1.0 + 3.0 ** (-c))
    return out


def make_point(
    n_prefill: int,
    n_decode: int,
    n_classes: int = 2,
    policy: str = "learned",
    backlog_mode: str = "true",
    physics: Optional[dict] = None,
    kv_cap: int = 200_000,
    kv_cap_pre: Optional[int] = None,
    w_b: float = 1.0,
    w_s: float = 1.0,
    w_q: float = 1e-3,
    rho: float = 1.0,
    tau_pre_scale: float = 1.0,
    tau_dec_scale: float = 1.0,
    sigma: Optional[Sequence[float]] = None,
    link_bytes_per_s: float = LINK_BYTES_PER_S,
    len_threshold: int = 256,
    service: str = "serial",
    beta_pre: Optional[float] = None,
    beta_dec: Optional[float] = None,
) -> Dict:
    """One parameter point: pool shape, router constants, physics and SLOs.

    Router constants are the priced view (float32 seconds); physics is the
    true service model (int64 ns).  ``tau_*_scale`` multiplies the router's
    per-token prices relative to the physics (1.0 = calibrated, Section III-B).
    ``service`` is "serial" (one request at a time per instance) or "batched"
    (continuous batching at the prefill and the decode stage alike: each of b requests sharing an
    instance runs at 1 / (1 + beta (b - 1)) of its stand-alone speed);
    both betas default to BATCH_BETA, the measured decode curve of Section VI.
    """
    ph = dict(SIM_PHYSICS if physics is None else physics)
    ttft, tpot = slo_targets(ph["dec_tok_ns"], n_classes)
    sg = list(sigma) + [1.0] * (MAX_CLASSES - len(sigma)) if sigma is not None else sigma_table(n_classes)
    return dict(
        n_prefill=int(n_prefill),
        n_decode=int(n_decode),
        n_classes=int(n_classes),
        policy=policy,
        len_threshold=int(len_threshold),
        backlog_mode=backlog_mode,
        w_b=f32(w_b),
        w_s=f32(w_s),
        w_q=f32(w_q),
        rho=f32(rho),
        tau_pre_s=f32(ph["pre_tok_ns"] * 1e-9 * tau_pre_scale),
        tau_dec_s=f32(ph["dec_tok_ns"] * 1e-9 * tau_dec_scale),
        pre_base_s=f32(ph["pre_base_ns"] * 1e-9),
        sigma=[f32(s) for s in sg],
        pre_base_ns=int(ph["pre_base_ns"]),
        pre_tok_ns=int(ph["pre_tok_ns"]),
        dec_tok_ns=int(ph["dec_tok_ns"]),
        xfer_tok_ns=xfer_tok_ns(ph["kv_bytes_per_token"], link_bytes_per_s),
        kv_cap_pre=int(kv_cap if kv_cap_pre is None else kv_cap_pre),
        kv_cap_dec=int(kv_cap),
        slo_ttft_ns=[int(v) for v in ttft],
        slo_tpot_ns=[int(v) for v in tpot],
        service=service,
        beta_pre=float(BATCH_BETA if beta_pre is None else beta_pre),
        beta_dec=float(BATCH_BETA if beta_dec is None else beta_dec),
    )


# --------------------------------------------------------------------------
# Length and arrival distributions
# --------------------------------------------------------------------------
@dataclass(frozen=True)
class LogNormal:
    mu: float
    sigma: float
    lo: int
    hi: int

    def from_normal(self, z: np.ndarray) -> np.ndarray:
        return np.clip(np.rint(np.exp(self.mu + self.sigma * z)), self.lo, self.hi).astype(np.int32)

    def clipped_mean(self) -> float:
        """E[clip(X, lo, hi)] for the continuous lognormal X (rounding ignored)."""
        m, s = self.mu, self.sigma

        def phi(x):
            return 0.5 * (1.0 + math.erf(x / math.sqrt(2.0)))

        la, lb = math.log(self.lo), math.log(self.hi)
        p_lo = phi((la - m) / s)
        p_hi = 1.0 - phi((lb - m) / s)
        mid = math.exp(m + s * s / 2) * (phi((lb - m - s * s) / s) - phi((la - m - s * s) / s))
        return self.lo * p_lo + self.hi * p_hi + mid


@dataclass(frozen=True)
class Pareto:
    alpha: float
    xm: float
    lo: int
    hi: int

    def from_uniform(self, u: np.ndarray) -> np.ndarray:
        x = self.xm / np.power(1.0 - u, 1.0 / self.alpha)
        return np.clip(np.rint(x), self.lo, self.hi).astype(np.int32)

    def clipped_mean(self) -> float:
        """E[min(X, hi)] for lo <= xm (closed form of the integral of the tail)."""
        a, xm, c = self.alpha, self.xm, float(self.hi)
        return xm + (xm ** a * c ** (1.0 - a) - xm) / (1.0 - a)


@dataclass(frozen=True)
class Traffic:
    """Request mixture + arrival process of one parameter point."""

    prompt: tuple  # per component: LogNormal
    output: tuple  # per component: LogNormal or Pareto
    mix: tuple  # component probabilities (sum 1)
    class_probs: tuple
    arrival: str  # "poisson" or "mmpp"
    rates: tuple  # poisson: (rate,), mmpp: (calm, burst) in req/s
    dwell_mean_s: float = 20.0
    pred_sigma: float = 0.3

    def mean_prompt(self) -> float:
        return sum(w * d.clipped_mean() for w, d in zip(self.mix, self.prompt))

    def mean_output(self) -> float:
        return sum(w * d.clipped_mean() for w, d in zip(self.mix, self.output))

    def mean_rate(self) -> float:
        if self.arrival == "poisson":
            return self.rates[0]
        return 0.5 * (self.rates[0] + self.rates[1])  # equal mean dwell in both states

    def scaled(self, k: float) -> "Traffic":
        return Traffic(self.prompt, self.output, self.mix, self.class_probs, self.arrival,
                       tuple(r * k for r in self.rates), self.dwell_mean_s, self.pred_sigma)


def capacity_rps(point: Dict, traffic: Traffic) -> float:
    """Saturation arrival rate of a pool shape under serial service.

    min(P / E[S_pre], D / E[S_dec]) with E[S_pre] = base + E[p] * pre_tok and
    E[S_dec] = (E[o] - 1) * dec_tok, the means taken over the clipped length
    distributions.  Used only to place workloads at a chosen load factor.
    """
    ep, eo = traffic.mean_prompt(), traffic.mean_output()
    s_pre = (point["pre_base_ns"] + ep * point["pre_tok_ns"]) * 1e-9
    s_dec = (eo - 1.0) * point["dec_tok_ns"] * 1e-9
    return min(point["n_prefill"] / s_pre, point["n_decode"] / s_dec)


# Workload families (Table I).  Chat: short in / short out.  Reasoning: short
# in / long out.  Mixed bursty: an 80/20 chat/reasoning mixture under MMPP.
CHAT_PROMPT = LogNormal(5.5, 0.8, 16, 8192)
CHAT_OUTPUT = LogNormal(4.5, 0.8, 1, 4096)
REASON_PROMPT = LogNormal(7.0, 0.7, 16, 8192)
REASON_OUTPUT = LogNormal(7.0, 0.6, 1, 4096)


def mixed_bursty(calm: float = 3.0, burst: float = 12.0) -> Traffic:
    return Traffic(
        prompt=(CHAT_PROMPT, REASON_PROMPT),
        output=(CHAT_OUTPUT, REASON_OUTPUT),
        mix=(0.8, 0.2),
        class_probs=(0.5, 0.3, 0.2),
        arrival="mmpp",
        rates=(calm, burst),
    )


# The other workload families of Table I as Poisson streams (the lengths are
# our proposal; the paper characterizes them only qualitatively).
DOC_PROMPT = LogNormal(7.6, 0.5, 256, 4096)  # long documents, up to 4k in
DOC_OUTPUT = LogNormal(4.5, 0.8, 1, 4096)    # short answers


def chat(rate: float) -> Traffic:
    return Traffic((CHAT_PROMPT,), (CHAT_OUTPUT,), (1.0,), (0.5, 0.3, 0.2), "poisson", (rate,))


def document(rate: float) -> Traffic:
    return Traffic((DOC_PROMPT,), (DOC_OUTPUT,), (1.0,), (0.5, 0.3, 0.2), "poisson", (rate,))


def reasoning(rate: float) -> Traffic:
    return Traffic((REASON_PROMPT,), (REASON_OUTPUT,), (1.0,), (0.5, 0.3, 0.2), "poisson", (rate,))


def with_predictor_sigma(traffic: Traffic, sigma: float) -> Traffic:
    """The same traffic with the output-length predictor's log-normal error
    sigma (o^ = o * exp(sigma * z))."""
    return Traffic(traffic.prompt, traffic.output, traffic.mix, traffic.class_probs, traffic.arrival,
                   traffic.rates, traffic.dwell_mean_s, float(sigma))


def tiny_poisson(rate: float = 4.0) -> Traffic:
    return Traffic(
        prompt=(LogNormal(6.0, 1.0, 16, 8192),),
        output=(LogNormal(5.0, 1.2, 1, 4096),),
        mix=(1.0,),
        class_probs=(0.7, 0.3),
        arrival="poisson",
        rates=(rate,),
    )


def large_pool(rate: float) -> Traffic:
    return Traffic(
        prompt=(LogNormal(6.5, 1.2, 16, 131072),),
        output=(Pareto(1.5, 100.0, 1, 32768),),
        mix=(1.0,),
        class_probs=(0.4, 0.3, 0.2, 0.1),
        arrival="poisson",
        rates=(rate,),
    )


# --------------------------------------------------------------------------
# Per-replica generation
# --------------------------------------------------------------------------
def _arrivals(rng: np.random.Generator, traffic: Traffic, n: int) -> np.ndarray:
    if n == 0:
        return np.zeros(0, np.int64)
    if traffic.arrival == "poisson":
        t = np.cumsum(rng.standard_exponential(n) / traffic.rates[0])
    elif traffic.arrival == "mmpp":
        # Two-state MMPP starting in the calm state, exponential dwell times.
        # Time rescaling: unit-rate Poisson points u_i mapped through the
        # inverse of the piecewise-linear cumulative intensity.
        u = np.cumsum(rng.standard_exponential(n))
        dwell: List[np.ndarray] = []
        lam_end = 0.0
        total = 0
        while lam_end < u[-1]:
            d = rng.exponential(traffic.dwell_mean_s, 64)
            dwell.append(d)
            total += 64
            rate = np.where(np.arange(total) % 2 == 0, traffic.rates[0], traffic.rates[1])
            lam_end = float(np.sum(np.concatenate(dwell) * rate))
        d = np.concatenate(dwell)
        rate = np.where(np.arange(d.size) % 2 == 0, traffic.rates[0], traffic.rates[1])
        t_start = np.concatenate(([0.0], np.cumsum(d)[:-1]))
        l_start = np.concatenate(([0.0], np.cumsum(d * rate)[:-1]))
        seg = np.searchsorted(l_start, u, side="right") - 1
        t = t_start[seg] + (u - l_start[seg]) / rate[seg]
    else:
        raise ValueError(f"unknown arrival process {traffic.arrival!r}")
    return np.rint(t * 1e9).astype(np.int64)


def replica_arrays(seed: int, replica: int, traffic: Traffic, n: int) -> Dict[str, np.ndarray]:
    """All request arrays of one replica, drawn in the fixed order."""
    rng = np.random.default_rng([int(seed), int(replica)])
    ncomp = len(traffic.mix)
    u_mix = rng.random(n)
    comp = np.searchsorted(np.cumsum(traffic.mix)[:-1], u_mix, side="right") if ncomp > 1 else np.zeros(n, np.int64)
    zp = rng.standard_normal(n)
    p = np.empty(n, np.int32)
    for c in range(ncomp):
        m = comp == c
        p[m] = traffic.prompt[c].from_normal(zp[m])
    out_kind = type(traffic.output[0])
    if out_kind is Pareto:
        uo = rng.random(n)
        o = np.empty(n, np.int32)
        for c in range(ncomp):
            m = comp == c
            o[m] = traffic.output[c].from_uniform(uo[m])
    else:
        zo = rng.standard_normal(n)
        o = np.empty(n, np.int32)
        for c in range(ncomp):
            m = comp == c
            o[m] = traffic.output[c].from_normal(zo[m])
    zq = rng.standard_normal(n)
    oh = np.maximum(1, np.rint(o.astype(np.float64) * np.exp(traffic.pred_sigma * zq))).astype(np.int32)
    u_cls = rng.random(n)
    cls = np.searchsorted(np.cumsum(traffic.class_probs)[:-1], u_cls, side="right").astype(np.uint8)
    arr = _arrivals(rng, traffic, n)
    return dict(arrival_ns=arr, prompt_len=p, out_len=o, pred_out_len=oh, slo_class=cls)


def sample_words(seed: int, replica: int, n: int) -> np.ndarray:
    """[n, 4] uint32 random words of one replica for the sampled policy (two
    per pool), from a stream of their own so that the other arrays do not
    depend on whether they are drawn."""
    rng = np.random.default_rng([int(seed), int(replica), 1])
    return rng.integers(0, 1 << 32, size=(n, 4), dtype=np.uint32)


def add_sample_words(trace: Dict[str, np.ndarray], seed: int, replicas: Optional[Sequence[int]] = None) -> None:
    """Attach ``sample_bits`` ([n_requests, 4] uint32) to an SoA trace: the
    words of trace replica k are those of workload replica replicas[k]."""
    off = trace["offsets"]
    reps = range(len(off) - 1) if replicas is None else replicas
    parts = [sample_words(seed, int(r), int(off[k + 1] - off[k])) for k, r in enumerate(reps)]
    trace["sample_bits"] = np.concatenate(parts) if parts else np.zeros((0, 4), np.uint32)


# --------------------------------------------------------------------------
# Workloads
# --------------------------------------------------------------------------
@dataclass
class Workload:
    """A batch of replicas over one or more parameter points."""

    name: str
    seed: int
    n_replicas: int
    requests: int  # per replica
    points: List[Dict]
    traffic: List[Traffic]  # per point
    point_of: Callable[[int], int] = field(default=lambda i: 0)
    meta: Dict = field(default_factory=dict)

    def param_point(self) -> np.ndarray:
        return np.array([self.point_of(i) for i in range(self.n_replicas)], np.int32)


def _gen_range(args):
    wl_seed, lo, hi, pts, trafs, n = args
    parts = [replica_arrays(wl_seed, i, trafs[pts[i - lo]], n) for i in range(lo, hi)]
    return lo, {k: np.concatenate([q[k] for q in parts]) for k in parts[0]}


def make_trace(wl: Workload, replicas: Optional[Sequence[int]] = None, workers: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Structure-of-arrays trace for ``replicas`` (default: all) of a workload.

    Returns arrival_ns i64, prompt_len/out_len/pred_out_len i32, slo_class u8
    (concatenated per replica), offsets i64[n+1] and param_point i32[n].
    """
    if replicas is None:
        reps = np.arange(wl.n_replicas)
    else:
        reps = np.asarray(replicas, dtype=np.int64)
    pts_all = np.array([wl.point_of(int(i)) for i in reps], np.int32)
    n = wl.requests
    contiguous = reps.size > 0 and np.all(np.diff(reps) == 1)
    if workers is None:
        workers = min(16, os.cpu_count() or 1)
    if contiguous and reps.size * n >= 2_000_000 and workers > 1:
        lo0 = int(reps[0])
        chunk = max(1, reps.size // (workers * 4))
        jobs = [(wl.seed, lo0 + a, lo0 + min(reps.size, a + chunk), pts_all[a:a + chunk], wl.traffic, n)
                for a in range(0, reps.size, chunk)]
        cols = {k: [] for k in ("arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class")}
        import multiprocessing as mp
        with ProcessPoolExecutor(max_workers=workers, mp_context=mp.get_context("fork")) as ex:
            for _, d in ex.map(_gen_range, jobs):
                for k in cols:
                    cols[k].append(d[k])
        out = {k: np.concatenate(v) for k, v in cols.items()}
    else:
        parts = [replica_arrays(wl.seed, int(i), wl.traffic[int(pt)], n) for i, pt in zip(reps, pts_all)]
        keys = ("arrival_ns", "prompt_len", "out_len", "pred_out_len", "slo_class")
        if parts:
            out = {k: np.concatenate([q[k] for q in parts]) for k in keys}
        else:
            out = dict(arrival_ns=np.zeros(0, np.int64), prompt_len=np.zeros(0, np.int32),
                       out_len=np.zeros(0, np.int32), pred_out_len=np.zeros(0, np.int32),
                       slo_class=np.zeros(0, np.uint8))
    out["offsets"] = np.arange(reps.size + 1, dtype=np.int64) * n
    out["param_point"] = pts_all
    if any(p["policy"] == "learned_sampled" for p in wl.points):
        add_sample_words(out, wl.seed, reps)
    return out


def tiny_sim(seed: int = 0) -> Workload:
    """1 replica, 3 prefill + 3 decode, 2,000 Poisson requests at 4 req/s."""
    return Workload("tiny-sim-3p3d-2k", seed, 1, 2000,
                    [make_point(3, 3, n_classes=2)], [tiny_poisson(4.0)])


def paper_cluster(n_replicas: int = 4096, requests: int = 10_000, seed: int = 2,
                  policy: str = "learned", service: str = "serial") -> Workload:
    """2 prefill + 6 decode, mixed bursty MMPP (3 / 12 req/s, 20 s dwell);
    ``service="batched"`` serves it under continuous batching (BATCH_BETA)."""
    tag = "" if policy == "learned" else "-" + policy.replace("_", "-")
    tag += "" if service == "serial" else "-" + service
    return Workload(f"cluster-2p6d-mmpp-{n_replicas}x{requests}{tag}", seed, n_replicas, requests,
                    [make_point(2, 6, n_classes=3, policy=policy, service=service)], [mixed_bursty()])


SWEEP_WIDTHS = (3, 4, 6, 8, 16, 32, 64)
SWEEP_LOADS = (0.6, 0.7, 0.8, 0.9, 1.0, 1.1, 1.2)
SWEEP_SCALES = (0.25, 0.5, 1.0, 2.0, 4.0)


def sweep_points():
    """The 7 x 7 x 25 = 1225 points of the parameter sweep and their traffic.

    Point index = (width * 7 + load) * 25 + (prefill-scale * 5 + decode-scale).
    Each point's MMPP rates are scaled so that its mean rate is load x the
    pool's serial-service capacity; the router prices per-token work at
    scale x the physics (mis-calibration), with the in-flight ledger as the
    backlog signal (Section VI: the proxy estimates backlog from its own
    constants).
    """
    base = mixed_bursty()
    points, trafs = [], []
    for w in SWEEP_WIDTHS:
        for ld in SWEEP_LOADS:
            for sp in SWEEP_SCALES:
                for sd in SWEEP_SCALES:
                    pt = make_point(2, w, n_classes=3, backlog_mode="proxy",
                                    tau_pre_scale=sp, tau_dec_scale=sd)
                    k = ld * capacity_rps(pt, base) / base.mean_rate()
                    points.append(pt)
                    trafs.append(base.scaled(k))
    return points, trafs


def param_sweep(n_replicas: int = 65536, requests: int = 5000, seed: int = 3) -> Workload:
    pts, trafs = sweep_points()
    npt = len(pts)
    return Workload(f"sweep-1225pt-{n_replicas}x{requests}", seed, n_replicas, requests, pts, trafs,
                    point_of=lambda i: i % npt)


def large_pool_wl(n_replicas: int = 256, requests: int = 1_000_000, seed: int = 4, load: float = 0.95) -> Workload:
    """128 prefill + 1,024 decode, Pareto outputs, Poisson at 0.95 of capacity."""
    pt = make_point(128, 1024, n_classes=4, kv_cap=2_000_000)
    tr0 = large_pool(1.0)
    rate = load * capacity_rps(pt, tr0)
    return Workload(f"large-128p1024d-{n_replicas}x{requests}", seed, n_replicas, requests, [pt],
                    [large_pool(rate)], meta=dict(rate=rate))


def batched_wide_pool(n_replicas: int = 16384, requests: int = 1000, seed: int = 5, n_prefill: int = 8,
                      n_decode: int = 64, load: float = 0.8) -> Workload:
    """Continuous batching at the prefill and the decode stage alike on a pool too wide for one segment
    of lanes (8 prefill + 64 decode = 72 instances): mixed bursty traffic at
    ``load`` x the serial-service capacity."""
    pt = make_point(n_prefill, n_decode, n_classes=3, service="batched")
    base = mixed_bursty()
    k = load * capacity_rps(pt, base) / base.mean_rate()
    return Workload(f"batched-{n_prefill}p{n_decode}d-mmpp-{n_replicas}x{requests}", seed, n_replicas, requests, [pt],
                    [base.scaled(k)])


# --------------------------------------------------------------------------
# Standalone scorer inputs
# --------------------------------------------------------------------------
def scorer_inputs(n_req: int = 1 << 20, n_inst: int = 64, seed: int = 1, per_request: bool = False,
                  kv_cap: int = 200_000) -> Dict[str, np.ndarray]:
    """Requests with the tiny-sim feature distributions and one decode-pool snapshot.

    Snapshot: queue ~ U{0..256}, kv_occ = floor(U[0,1) * cap), backlog (busy
    until, with now = 0) ~ U[0, 10) s.  ``per_request`` draws an independent
    snapshot row per request (layout [n_req][n_inst]).
    """
    tr = tiny_poisson()
    rng = np.random.default_rng([int(seed)])
    zp = rng.standard_normal(n_req)
    zo = rng.standard_normal(n_req)
    zq = rng.standard_normal(n_req)
    p = tr.prompt[0].from_normal(zp)
    o = tr.output[0].from_normal(zo)
    oh = np.maximum(1, np.rint(o.astype(np.float64) * np.exp(tr.pred_sigma * zq))).astype(np.int32)
    cls = np.searchsorted(np.cumsum(tr.class_probs)[:-1], rng.random(n_req), side="right").astype(np.uint8)
    rows = n_req if per_request else 1
    queue = rng.integers(0, 257, size=(rows, n_inst)).astype(np.int32)
    kv = np.floor(rng.random((rows, n_inst)) * kv_cap).astype(np.int32)
    backlog = rng.uniform(0.0, 10.0, size=(rows, n_inst)).astype(np.float32)
    return dict(prompt_len=p, pred_out_len=oh, slo_class=cls, queue=queue.reshape(-1),
                kv_occ=kv.reshape(-1), backlog_s=backlog.reshape(-1),
                n_inst=n_inst, inst_stride=(n_inst if per_request else 0), kv_cap=kv_cap)


def scorer_params(n_classes: int = 2) -> Dict:
    """Router parameters for the standalone scorer (simulator constants)."""
    pt = make_point(1, 64, n_classes=n_classes)
    return {k: pt[k] for k in ("w_b", "w_s", "w_q", "rho", "tau_pre_s", "tau_dec_s", "pre_base_s", "sigma")}


WORKLOADS = {
    "tiny": tiny_sim,
    "cluster": paper_cluster,
    "sweep": param_sweep,
    "large": large_pool_wl,
}
