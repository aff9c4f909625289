// Replica-batched simulation of the learned prefill/decode router on gfx950.
//
// Method: Algorithm 1 per admission (score both pools with the Section III-A
// cost equation, take each argmin, prefill, transfer KV, decode, record),
// on the serial-service simulator of Section III-D / Section VI.
//
// Mapping.  A replica is a sequential chain of admissions; replicas are
// independent.  One replica occupies a segment of S lanes (S a power of two):
// S <= 64 packs 64/S replicas into each wave; S > 64 spreads one replica over
// the S/64 waves of a workgroup.  Instance j of a pool lives in lane j / M,
// slot j % M (blocked layout, M instances per lane), so the lowest lane that
// holds the minimum cost also holds the lowest index.  All per-instance state
// (busy-until, queue, cache occupancy, ledger tokens, FIFO head) is in
// registers; every lane of a segment computes the per-request quantities
// redundantly, so no broadcast is needed for them.
//
// FIFO of in-flight requests per instance.  Service is in admission order,
// so each instance releases its requests in admission order and only the
// head's release time matters for retiring.  The list is kept as successor
// records in HBM scratch: when request y is appended behind x, y's record
// (release time, index, cache tokens, ledger tokens) is stored in x's slot.
// The head and the second element are cached in registers; after a pop the
// record behind the new head is loaded into a pending register set and
// merged at the start of the next step, so a single pop per step never waits
// for memory.  The same lane always writes and reads an instance's slots.
//
// Arithmetic: the cost is evaluated exactly as the equation is written, left
// to right in float32, one rounding per operation (built with
// -ffp-contract=off); integer-to-float conversions round to nearest even.
#include "rt_internal.h"

namespace rt {
namespace {

struct Rec {
  int64_t t;    // release time
  int32_t idx;  // index within the replica
  int32_t fp;   // cache tokens held until release
  int32_t pt;   // tokens the ledger prices
};

// Per-instance state.  Plain scalars only, copied field by field with value
// selects, so that everything stays in registers.
struct Inst {
  int64_t busy;  // end of everything admitted so far
  int64_t kv;    // cache tokens in flight
  int64_t pend;  // ledger tokens in flight
  int32_t q;     // requests in flight
  int32_t tail;  // index of the last admitted request
  // head of the FIFO (valid if q >= 1)
  int64_t h_t;
  int32_t h_idx, h_fp, h_pt;
  // second element (valid if q >= 2 and lp == 0)
  int64_t n_t;
  int32_t n_idx, n_fp, n_pt;
  // load target for the second element (valid if lp != 0)
  int64_t l_t;
  int32_t l_idx, l_fp, l_pt;
  int32_t lp;
};

__device__ __forceinline__ void merge_pending(Inst& s) {
  const bool c = s.lp != 0;
  s.n_t = c ? s.l_t : s.n_t;
  s.n_idx = c ? s.l_idx : s.n_idx;
  s.n_fp = c ? s.l_fp : s.n_fp;
  s.n_pt = c ? s.l_pt : s.n_pt;
  s.lp = 0;
}

__device__ __forceinline__ int64_t shfl64(int64_t v, int src) {
  int lo = __shfl((int)(uint32_t)(uint64_t)v, src, 64);
  int hi = __shfl((int)(uint32_t)((uint64_t)v >> 32), src, 64);
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint64_t)(uint32_t)lo);
}

template <int S>
__device__ __forceinline__ uint32_t seg_min(uint32_t v) {
#pragma unroll
  for (int m = 1; m < S && m < 64; m <<= 1) v = min(v, (uint32_t)__shfl_xor((int)v, m, 64));
  return v;
}

template <int S>
__device__ __forceinline__ int32_t seg_max_i32(int32_t v) {
#pragma unroll
  for (int m = 1; m < S && m < 64; m <<= 1) v = max(v, __shfl_xor(v, m, 64));
  return v;
}

__device__ __forceinline__ int32_t wave_max_i32(int32_t v) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) v = max(v, __shfl_xor(v, m, 64));
  return v;
}

// Pop the head of an instance's FIFO (caller checked q >= 1).  kDec selects
// the decode record layout {idx, cache tokens, ledger tokens, 0}; prefill
// records are {idx, prompt tokens} (cache and ledger tokens are both p).
__device__ __forceinline__ void pop_common(Inst& s) {
  s.q -= 1;
  s.kv -= s.h_fp;
  s.pend -= s.h_pt;
}

// The successor slot read after a pop is clamped into the replica's range:
// with correct bookkeeping it always is in range; the clamp only guarantees
// that no load can leave the scratch buffer.
__device__ __forceinline__ int64_t slot_of(int64_t base, int32_t idx, int32_t R) {
  idx = idx < 0 ? 0 : idx;
  idx = idx >= R ? R - 1 : idx;
  return base + idx;
}

__device__ __forceinline__ void pop_pre(Inst& s, const int64_t* __restrict__ succ_t,
                                        const int2* __restrict__ succ_m, int64_t base, int32_t R) {
  pop_common(s);
  if (s.q >= 1) {
    merge_pending(s);  // only does work on a second pop within one step
    s.h_t = s.n_t;
    s.h_idx = s.n_idx;
    s.h_fp = s.n_fp;
    s.h_pt = s.n_pt;
    if (s.q >= 2) {
      const int64_t g = slot_of(base, s.h_idx, R);
      const int2 m = succ_m[g];
      s.l_t = succ_t[g];
      s.l_idx = m.x;
      s.l_fp = m.y;
      s.l_pt = m.y;
      s.lp = 1;
    }
  }
}

__device__ __forceinline__ void pop_dec(Inst& s, const int64_t* __restrict__ succ_t,
                                        const int4* __restrict__ succ_m, int64_t base, int32_t R) {
  pop_common(s);
  if (s.q >= 1) {
    merge_pending(s);
    s.h_t = s.n_t;
    s.h_idx = s.n_idx;
    s.h_fp = s.n_fp;
    s.h_pt = s.n_pt;
    if (s.q >= 2) {
      const int64_t g = slot_of(base, s.h_idx, R);
      const int4 m = succ_m[g];
      s.l_t = succ_t[g];
      s.l_idx = m.x;
      s.l_fp = m.y;
      s.l_pt = m.z;
      s.lp = 1;
    }
  }
}

// Append request r (release t, index idx, cache tokens fp, ledger tokens pt).
__device__ __forceinline__ void append_common(Inst& s, int64_t t, int32_t idx, int32_t fp, int32_t pt) {
  const bool first = s.q == 0, second = s.q == 1;
  s.h_t = first ? t : s.h_t;
  s.h_idx = first ? idx : s.h_idx;
  s.h_fp = first ? fp : s.h_fp;
  s.h_pt = first ? pt : s.h_pt;
  s.n_t = second ? t : s.n_t;
  s.n_idx = second ? idx : s.n_idx;
  s.n_fp = second ? fp : s.n_fp;
  s.n_pt = second ? pt : s.n_pt;
  s.tail = idx;
  s.q += 1;
  s.kv += fp;
  s.pend += pt;
}

__device__ __forceinline__ void append_pre(Inst& s, int64_t t, int32_t idx, int32_t p, int64_t* __restrict__ succ_t,
                                           int2* __restrict__ succ_m, int64_t base) {
  if (s.q >= 1) {
    succ_t[base + s.tail] = t;
    succ_m[base + s.tail] = make_int2(idx, p);
  }
  append_common(s, t, idx, p, p);
}

__device__ __forceinline__ void append_dec(Inst& s, int64_t t, int32_t idx, int32_t fp, int32_t pt,
                                           int64_t* __restrict__ succ_t, int4* __restrict__ succ_m, int64_t base) {
  if (s.q >= 1) {
    succ_t[base + s.tail] = t;
    succ_m[base + s.tail] = make_int4(idx, fp, pt, 0);
  }
  append_common(s, t, idx, fp, pt);
}

__device__ __forceinline__ void init_inst(Inst& s) {
  s.busy = 0;
  s.kv = 0;
  s.pend = 0;
  s.q = 0;
  s.tail = -1;
  s.h_t = s.n_t = s.l_t = 0;
  s.h_idx = s.h_fp = s.h_pt = 0;
  s.n_idx = s.n_fp = s.n_pt = 0;
  s.l_idx = s.l_fp = s.l_pt = 0;
  s.lp = 0;
}

// The cost equation for one candidate (Section III-A), in written order.
__device__ __forceinline__ float cost_eq(float w_b, float rho, float w_q, float backlog_s, float work,
                                         float sg, int64_t kv, int64_t need, float inv_cap, int32_t q) {
  const float press = (float)(kv + need) * inv_cap;
  const float load = w_b * backlog_s * sg;
  const float size = work * (1.0f + rho * press) * sg;
  return load + size + w_q * (float)q;
}

struct Winner {
  int32_t idx;
  int64_t busy;
};

struct Partial {
  uint32_t key;
  int32_t idx;
  int64_t busy;
};

template <int S, int MP, int MD>
__global__ void __launch_bounds__(S > 64 ? S : 256) sim_kernel(SimArgs a) {
  constexpr int kSegs = S >= 64 ? 1 : 64 / S;  // replicas per wave
  constexpr int kW = S > 64 ? S / 64 : 1;      // waves per replica
  const int lane = threadIdx.x & 63;
  // Wave index as a wave-uniform value, so that for S >= 64 everything
  // derived from it (replica, point parameters) lives in scalar registers.
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  int sl;        // lane within the replica's segment
  int64_t item;  // position in the work list
  int seg_base;  // first lane of the segment within the wave
  if constexpr (S <= 64) {
    sl = lane % S;
    seg_base = lane - sl;
    item = ((int64_t)blockIdx.x * (blockDim.x >> 6) + wave) * kSegs + lane / S;
  } else {
    sl = threadIdx.x;
    seg_base = 0;
    item = blockIdx.x;
  }
  const bool live = item < a.n_work;
  const int rep = live ? a.work[item] : 0;
  const int64_t base = live ? a.offsets[rep] : 0;
  const int32_t R = live ? (int32_t)(a.offsets[rep + 1] - base) : 0;
  const int pid = (live && a.param_point) ? a.param_point[rep] : 0;
  const DevPoint& pp = a.points[pid];
  const int32_t P = pp.P, D = pp.D, ncls = pp.n_classes, policy = pp.policy, mode = pp.mode;
  const float w_b = pp.w_b, w_s = pp.w_s, w_q = pp.w_q, rho = pp.rho;
  const float tau_pre = pp.tau_pre, tau_dec = pp.tau_dec, pre_base = pp.pre_base;
  const float inv_pre = pp.inv_cap_pre, inv_dec = pp.inv_cap_dec;
  float sigma[kMaxClasses];
#pragma unroll
  for (int c = 0; c < kMaxClasses; ++c) sigma[c] = pp.sigma[c];
  const int64_t pre_base_ns = pp.pre_base_ns, pre_tok_ns = pp.pre_tok_ns;
  const int64_t dec_tok_ns = pp.dec_tok_ns, xfer_tok_ns = pp.xfer_tok_ns;

  __shared__ Partial part[S > 64 ? 2 * 2 * kW : 1];

  Inst pre[MP], dec[MD];
#pragma unroll
  for (int m = 0; m < MP; ++m) init_inst(pre[m]);
#pragma unroll
  for (int m = 0; m < MD; ++m) init_inst(dec[m]);

  int32_t Rmax;
  if constexpr (S <= 64)
    Rmax = wave_max_i32(R);
  else
    Rmax = R;  // one replica per workgroup

  // Prefetched features of the next request.
  int64_t nx_arr = 0;
  int32_t nx_p = 0, nx_o = 0, nx_oh = 0;
  uint32_t nx_c = 0;
  if (R > 0) {
    nx_arr = a.arrival[base];
    nx_p = a.plen[base];
    nx_o = a.olen[base];
    nx_oh = a.ohat[base];
    nx_c = a.cls[base];
  }
  int64_t last_arr = 0;
  bool have_arr = false;
  int32_t rr_pre = 0, rr_dec = 0;  // round-robin counters: t mod P, t mod D

  for (int32_t t = 0; t < Rmax; ++t) {
    const bool act = t < R;
    const int64_t now = nx_arr;
    const int32_t p = nx_p, o = nx_o, oh = nx_oh;
    const uint32_t c = nx_c;
    if (t + 1 < R) {
      const int64_t g = base + t + 1;
      nx_arr = a.arrival[g];
      nx_p = a.plen[g];
      nx_o = a.olen[g];
      nx_oh = a.ohat[g];
      nx_c = a.cls[g];
    }
    const bool bad = act && (p < 1 || o < 1 || oh < 1 || (int64_t)p + o > INT32_MAX ||
                             (int64_t)p + oh > INT32_MAX || c >= (uint32_t)ncls || now < 0 ||
                             (have_arr && now < last_arr));
    const bool go = act && !bad;
    if (go) {
      last_arr = now;
      have_arr = true;
    }

    // Merge the successor records loaded during the previous step.
#pragma unroll
    for (int m = 0; m < MP; ++m) merge_pending(pre[m]);
#pragma unroll
    for (int m = 0; m < MD; ++m) merge_pending(dec[m]);

    // 1. Release everything that finished at or before now.
    while (true) {
      bool want = false;
#pragma unroll
      for (int m = 0; m < MP; ++m) want |= go && pre[m].q > 0 && pre[m].h_t <= now;
#pragma unroll
      for (int m = 0; m < MD; ++m) want |= go && dec[m].q > 0 && dec[m].h_t <= now;
      if (!__any(want)) break;
#pragma unroll
      for (int m = 0; m < MP; ++m)
        if (go && pre[m].q > 0 && pre[m].h_t <= now) pop_pre(pre[m], a.sp_t, a.sp_m, base, R);
#pragma unroll
      for (int m = 0; m < MD; ++m)
        if (go && dec[m].q > 0 && dec[m].h_t <= now) pop_dec(dec[m], a.sd_t, a.sd_m, base, R);
    }

    // 2. Keys of every candidate under the point's policy.
    float sg = sigma[0];
#pragma unroll
    for (int k = 1; k < kMaxClasses; ++k) sg = (c == (uint32_t)k) ? sigma[k] : sg;
    const float work_pre = w_s * (float)p * tau_pre;
    const float work_dec = w_s * (float)oh * tau_dec;
    const int64_t need_pre = p;
    const int64_t need_dec = (int64_t)p + oh;

    uint32_t bk_pre = 0xffffffffu, bk_dec = 0xffffffffu;
    int32_t bj_pre = 0, bj_dec = 0;
    int64_t bb_pre = 0, bb_dec = 0;
#pragma unroll
    for (int m = 0; m < MP; ++m) {
      const int j = sl * MP + m;
      uint32_t key;
      if (policy == 0) {
        float bl;
        if (mode == 0) {
          int64_t d = pre[m].busy - now;
          d = d < 0 ? 0 : d;
          bl = (float)d * 1e-9f;
        } else {
          bl = tau_pre * (float)pre[m].pend + pre_base * (float)pre[m].q;
        }
        key = cost_key(cost_eq(w_b, rho, w_q, bl, work_pre, sg, pre[m].kv, need_pre, inv_pre, pre[m].q));
      } else if (policy == 2) {
        key = (uint32_t)pre[m].q;
      } else {
        key = (j == rr_pre) ? 0u : 1u;
      }
      key = (go && j < P) ? key : 0xffffffffu;
      if (key < bk_pre) {
        bk_pre = key;
        bj_pre = j;
        bb_pre = pre[m].busy;
      }
    }
#pragma unroll
    for (int m = 0; m < MD; ++m) {
      const int j = sl * MD + m;
      uint32_t key;
      if (policy == 0) {
        float bl;
        if (mode == 0) {
          int64_t d = dec[m].busy - now;
          d = d < 0 ? 0 : d;
          bl = (float)d * 1e-9f;
        } else {
          bl = tau_dec * (float)dec[m].pend;
        }
        key = cost_key(cost_eq(w_b, rho, w_q, bl, work_dec, sg, dec[m].kv, need_dec, inv_dec, dec[m].q));
      } else if (policy == 2) {
        key = (uint32_t)dec[m].q;
      } else {
        key = (j == rr_dec) ? 0u : 1u;
      }
      key = (go && j < D) ? key : 0xffffffffu;
      if (key < bk_dec) {
        bk_dec = key;
        bj_dec = j;
        bb_dec = dec[m].busy;
      }
    }

    // 3. Argmin over the segment (lowest index on equal keys).
    Winner wp, wd;
    {
      const uint32_t mp = seg_min<S>(bk_pre);
      const uint32_t md = seg_min<S>(bk_dec);
      const uint64_t bp = __ballot(bk_pre == mp);
      const uint64_t bd = __ballot(bk_dec == md);
      const uint64_t segmask = (S >= 64) ? ~0ull : ((1ull << (S < 64 ? S : 0)) - 1ull);
      const uint64_t sp = (bp >> seg_base) & segmask;
      const uint64_t sd = (bd >> seg_base) & segmask;
      const int src_p = seg_base + (__ffsll((unsigned long long)sp) - 1);
      const int src_d = seg_base + (__ffsll((unsigned long long)sd) - 1);
      wp.idx = __shfl(bj_pre, src_p, 64);
      wd.idx = __shfl(bj_dec, src_d, 64);
      wp.busy = shfl64(bb_pre, src_p);
      wd.busy = shfl64(bb_dec, src_d);
      if constexpr (S > 64) {
        // Combine the per-wave winners through LDS (double-buffered by step
        // parity, so one barrier per step suffices).
        Partial* buf = part + (t & 1) * 2 * kW;
        if (lane == 0) {
          buf[wave] = Partial{mp, wp.idx, wp.busy};
          buf[kW + wave] = Partial{md, wd.idx, wd.busy};
        }
        __syncthreads();
        Partial bp0 = buf[0], bd0 = buf[kW];
#pragma unroll
        for (int w = 1; w < kW; ++w) {
          const Partial x = buf[w], y = buf[kW + w];
          if (x.key < bp0.key) bp0 = x;  // waves hold increasing index ranges
          if (y.key < bd0.key) bd0 = y;
        }
        wp = Winner{bp0.idx, bp0.busy};
        wd = Winner{bd0.idx, bd0.busy};
      }
    }

    // 4. Serve: prefill, KV transfer, decode, each FIFO in admission order.
    const int64_t s_pre = pre_base_ns + (int64_t)p * pre_tok_ns;
    const int64_t s_dec = (int64_t)(o - 1) * dec_tok_ns;
    const int64_t xfer = (int64_t)p * xfer_tok_ns;
    const int64_t pf_end = (now > wp.busy ? now : wp.busy) + s_pre;
    const int64_t kv_at = pf_end + xfer;
    const int64_t dec_end = (kv_at > wd.busy ? kv_at : wd.busy) + s_dec;
#pragma unroll
    for (int m = 0; m < MP; ++m)
      if (go && sl * MP + m == wp.idx) {
        append_pre(pre[m], pf_end, t, p, a.sp_t, a.sp_m, base);
        pre[m].busy = pf_end;
      }
#pragma unroll
    for (int m = 0; m < MD; ++m)
      if (go && sl * MD + m == wd.idx) {
        append_dec(dec[m], dec_end, t, p + o, oh, a.sd_t, a.sd_m, base);
        dec[m].busy = dec_end;
      }

    // 5. Record the outcome.
    if (act && sl == 0) {
      const int64_t g = base + t;
      a.i_pre[g] = go ? wp.idx : -1;
      a.i_dec[g] = go ? wd.idx : -1;
      a.ttft[g] = go ? pf_end - now : -1;
      a.span[g] = go ? dec_end - pf_end : -1;
      if (bad) atomicOr(a.flag, kFlagRejected);
    }
    rr_pre = (rr_pre + 1 == P) ? 0 : rr_pre + 1;
    rr_dec = (rr_dec + 1 == D) ? 0 : rr_dec + 1;
  }
}

template <int S, int MP, int MD>
hipError_t launch_one(const SimArgs& a, hipStream_t stream) {
  if (a.n_work <= 0) return hipSuccess;
  int64_t blocks;
  int threads;
  if constexpr (S <= 64) {
    threads = 256;
    const int64_t per_block = (256 / 64) * (64 / S);
    blocks = (a.n_work + per_block - 1) / per_block;
  } else {
    threads = S;
    blocks = a.n_work;
  }
  hipLaunchKernelGGL((sim_kernel<S, MP, MD>), dim3((unsigned)blocks), dim3(threads), 0, stream, a);
  return hipGetLastError();
}

struct ClassEntry {
  SimClass c;
  hipError_t (*fn)(const SimArgs&, hipStream_t);
};

// Cheapest first: the host picks the first class that fits a point.
const ClassEntry kClasses[] = {
    {{1, 1, 1}, launch_one<1, 1, 1>},       {{2, 1, 1}, launch_one<2, 1, 1>},
    {{4, 1, 1}, launch_one<4, 1, 1>},       {{8, 1, 1}, launch_one<8, 1, 1>},
    {{16, 1, 1}, launch_one<16, 1, 1>},     {{32, 1, 1}, launch_one<32, 1, 1>},
    {{64, 1, 1}, launch_one<64, 1, 1>},     {{64, 2, 2}, launch_one<64, 2, 2>},
    {{256, 1, 4}, launch_one<256, 1, 4>},   {{512, 2, 2}, launch_one<512, 2, 2>},
};

}  // namespace

int sim_class_count() { return (int)(sizeof(kClasses) / sizeof(kClasses[0])); }

SimClass sim_class(int i) { return kClasses[i].c; }

hipError_t launch_sim(const SimClass& c, const SimArgs& a, hipStream_t stream) {
  for (const ClassEntry& e : kClasses)
    if (e.c.S == c.S && e.c.MP == c.MP && e.c.MD == c.MD) return e.fn(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace rt
