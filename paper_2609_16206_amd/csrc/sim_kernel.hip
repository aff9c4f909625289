// Replica-batched simulation of the learned prefill/decode router on gfx950,
// for pools wider than one wave segment holds (the general kernel; narrower
// pools run the segment kernels).
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
// redundantly.  Segment reductions use DPP lane permutations within 16-lane
// rows and readlane across rows (no LDS round trip); S > 64 combines the
// per-wave winners through LDS with one barrier per step.
//
// Number representation.  Simulated times (ns) and token totals are integers;
// inside the kernel they are held as doubles, which represent every integer
// below 2^53 exactly, so sums, differences and maxima are exact and a
// double-to-float conversion rounds the exact integer to nearest even, the
// same float as an int64-to-float conversion.  On gfx950 these are single
// full-rate f64 instructions, where int64 arithmetic takes 2-3 instructions
// and an int64-to-float conversion a long sequence.  Times at or beyond 2^52
// ns (52 days) set a flag bit.
//
// FIFO of in-flight requests per instance.  Service is in admission order,
// so each instance releases its requests in admission order and only the
// head's release time matters for retiring.  The list is kept as successor
// records in HBM scratch: when request y is appended behind x, y's record
// (release time, index, cache tokens, ledger tokens) is stored in x's slot.
// The head and the second element live in registers; a pop promotes the
// second element and loads the record behind it into a pending register set
// that is merged at the top of the next step.
//
// Memory ordering within a step (one wave).  On gfx9 stores and loads share
// one counter, so a wait for a load also waits for every older store.  A step
// therefore places its one wait before its stores:
//   1. the current request (prefetched during the previous step); prefetch
//      the next one (index clamped into the replica);
//   2. release: at most one pop per instance, whose successor load is issued
//      unconditionally (from the wave's dummy slot when nothing was popped),
//      so that it lands in its own registers with no control-flow merge;
//      more pops at one instance in one step take a rare slow path that
//      waits;
//   3. score, argmin, serve (registers only);
//   4. merge the successor records loaded in 2 (the wait: those loads, and
//      stores of the previous step, which by now have long completed);
//   5. stores (outputs, FIFO appends) by the lanes that own them.
// The same lane always writes and reads an instance's slots, in program
// order, so a store is visible to every later load of that slot.
//
// Arithmetic of the cost: evaluated exactly as the equation is written, left
// to right in float32, one rounding per operation (built with
// -ffp-contract=off).
#include "lane_ops.h"
#include "rt_internal.h"

namespace rt {
namespace {

// Per-instance state.  Plain scalars only, copied field by field with value
// selects, so that everything stays in registers.
struct Inst {
  double busy;  // end of everything admitted so far
  double kv;    // cache tokens in flight
  double pend;  // ledger tokens in flight
  int32_t q;    // requests in flight
  int32_t tail; // index of the last admitted request
  // head of the FIFO (valid if q >= 1)
  double h_t;
  int32_t h_idx, h_fp, h_pt;
  // second element (valid if q >= 2 and lp == 0)
  double n_t;
  int32_t n_idx, n_fp, n_pt;
  // load target for the second element (valid if lp != 0)
  double l_t;
  int32_t l_idx, l_fp, l_pt;
  int32_t lp;
};

__device__ __forceinline__ void init_inst(Inst& s) {
  s.busy = 0.0;
  s.kv = 0.0;
  s.pend = 0.0;
  s.q = 0;
  s.tail = -1;
  s.h_t = s.n_t = s.l_t = 0.0;
  s.h_idx = s.h_fp = s.h_pt = 0;
  s.n_idx = s.n_fp = s.n_pt = 0;
  s.l_idx = s.l_fp = s.l_pt = 0;
  s.lp = 0;
}

__device__ __forceinline__ void merge_pending(Inst& s) {
  const bool c = s.lp != 0;
  s.n_t = c ? s.l_t : s.n_t;
  s.n_idx = c ? s.l_idx : s.n_idx;
  s.n_fp = c ? s.l_fp : s.n_fp;
  s.n_pt = c ? s.l_pt : s.n_pt;
  s.lp = 0;
}

// Materializes the merged second element here, ahead of every later memory
// instruction (an empty volatile asm that reads the registers and clobbers
// memory), so that the wait for its load is not pushed past the stores.
__device__ __forceinline__ void pin_record(const Inst& s) {
  asm volatile("" ::"v"(s.n_t), "v"(s.n_idx), "v"(s.n_fp), "v"(s.n_pt) : "memory");
}

// The successor slot read after a pop is clamped into the replica's range:
// with correct bookkeeping it always is in range; the clamp only guarantees
// that no load can leave the scratch buffer.
__device__ __forceinline__ int64_t slot_of(int64_t base, int32_t idx, int32_t R) {
  idx = idx < 0 ? 0 : idx;
  idx = idx >= R ? R - 1 : idx;
  return base + idx;
}

// Records: {release (double bits), successor index, cache tokens} in the
// first entry of the request's pair for the pool; the ledger tokens of a
// decode record in the first entry of its token pair (a prefill record's
// ledger tokens are its cache tokens, the prompt).
template <typename T>
__device__ __forceinline__ T* rec_at(const SimArgs& a, int64_t g, int off) {
  return reinterpret_cast<T*>(a.rec + g * kRecStride + off);
}

__device__ __forceinline__ void read_pre(const int4& m, double& t, int32_t& idx, int32_t& fp, int32_t& pt) {
  t = __hiloint2double(m.y, m.x);
  idx = m.z;
  fp = m.w;
  pt = m.w;
}

// Fast-path pop, applied with selects when `pp`: the second element becomes
// the head.  The record behind the new head is then loaded unconditionally
// (from `dummy` when there is no such record) straight into the pending set.
template <bool kDec>
__device__ __forceinline__ void pop_fast(Inst& s, bool pp, const SimArgs& a, const char* dummy, int64_t base,
                                         int32_t R) {
  s.q -= pp ? 1 : 0;
  s.kv -= pp ? (double)s.h_fp : 0.0;
  s.pend -= pp ? (double)s.h_pt : 0.0;
  s.h_t = pp ? s.n_t : s.h_t;
  s.h_idx = pp ? s.n_idx : s.h_idx;
  s.h_fp = pp ? s.n_fp : s.h_fp;
  s.h_pt = pp ? s.n_pt : s.h_pt;
  const bool ld = pp && s.q >= 2;
  const int64_t g = slot_of(base, s.h_idx, R);
  if constexpr (kDec) {
    const int4* pm = ld ? rec_at<int4>(a, g, kRecPairDec) : reinterpret_cast<const int4*>(dummy);
    const int32_t* pq = ld ? rec_at<int32_t>(a, g, kRecTokDec) : reinterpret_cast<const int32_t*>(dummy + 16);
    const int4 m = *pm;
    s.l_t = __hiloint2double(m.y, m.x);
    s.l_idx = m.z;
    s.l_fp = m.w;
    s.l_pt = *pq;
  } else {
    const int4* pm = ld ? rec_at<int4>(a, g, kRecPairPre) : reinterpret_cast<const int4*>(dummy);
    read_pre(*pm, s.l_t, s.l_idx, s.l_fp, s.l_pt);
  }
  s.lp = ld ? 1 : 0;
}

// Slow-path pop (a further completion at the same instance within one step):
// merges what is pending, pops, and reads the next record synchronously.
template <bool kDec>
__device__ __forceinline__ void pop_slow(Inst& s, const SimArgs& a, int64_t base, int32_t R) {
  merge_pending(s);
  s.q -= 1;
  s.kv -= (double)s.h_fp;
  s.pend -= (double)s.h_pt;
  s.h_t = s.n_t;
  s.h_idx = s.n_idx;
  s.h_fp = s.n_fp;
  s.h_pt = s.n_pt;
  if (s.q >= 2) {
    const int64_t g = slot_of(base, s.h_idx, R);
    if constexpr (kDec) {
      const int4 m = *rec_at<int4>(a, g, kRecPairDec);
      s.n_t = __hiloint2double(m.y, m.x);
      s.n_idx = m.z;
      s.n_fp = m.w;
      s.n_pt = *rec_at<int32_t>(a, g, kRecTokDec);
    } else {
      read_pre(*rec_at<int4>(a, g, kRecPairPre), s.n_t, s.n_idx, s.n_fp, s.n_pt);
    }
  }
}

// Append a request (release t, index idx, cache tokens fp, ledger tokens
// pt).  Returns the scratch slot whose successor record must be stored (the
// previous tail's), or -1.
__device__ __forceinline__ int64_t append(Inst& s, double t, int32_t idx, int32_t fp, int32_t pt, int64_t base) {
  const int64_t slot = s.q >= 1 ? base + s.tail : -1;
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
  s.kv += (double)fp;
  s.pend += (double)pt;
  return slot;
}

// The cost equation for one candidate (Section III-A), in written order.
// `occ_need` is the exact cache occupancy after admission.
__device__ __forceinline__ float cost_eq(float w_b, float rho, float w_q, float backlog_s, float work,
                                         float sg, double occ_need, float inv_cap, int32_t q) {
  const float press = (float)occ_need * inv_cap;
  const float load = w_b * backlog_s * sg;
  const float size = work * (1.0f + rho * press) * sg;
  return load + size + w_q * (float)q;
}

struct Partial {
  uint32_t key_pre, key_dec;
  int32_t idx_pre, idx_dec;
  double busy_pre;
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
  if constexpr (S <= 64) {
    sl = lane % S;
    item = ((int64_t)blockIdx.x * (blockDim.x >> 6) + wave) * kSegs + lane / S;
  } else {
    sl = threadIdx.x;
    item = blockIdx.x;
  }
  const int wl_self = S > 64 ? lane : sl;  // lane index seg_first reports
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
  const double pre_base_ns = (double)pp.pre_base_ns, pre_tok_ns = (double)pp.pre_tok_ns;
  const double dec_tok_ns = (double)pp.dec_tok_ns, xfer_tok_ns = (double)pp.xfer_tok_ns;

  __shared__ Partial part[S > 64 ? 2 * kW : 1];

  Inst pre[MP], dec[MD];
#pragma unroll
  for (int m = 0; m < MP; ++m) init_inst(pre[m]);
#pragma unroll
  for (int m = 0; m < MD; ++m) init_inst(dec[m]);

  // steps of this wave: the longest replica among its segments
  const int32_t Rmax = S <= 64 ? wave_max_nonneg(R) : R;
  // the wave's 64-byte dummy slot (see the memory-ordering note); every lane
  // of the wave reads the same address, which costs one memory request
  char* const dummy =
      a.dummy + (size_t)(((blockIdx.x * blockDim.x + threadIdx.x) >> 6) & (kDummyLanes / 64 - 1)) * 64;

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

  uint32_t flag = 0;  // data-error bits, published once at the end

  for (int32_t t = 0; t < Rmax; ++t) {
    // 1. the current request; prefetch the next (index clamped into the
    // replica, so the same loads are issued at every step)
    const bool act = t < R;
    const int64_t arr = nx_arr;
    const int32_t p = nx_p, o = nx_o, oh = nx_oh;
    const uint32_t c = nx_c;
    {
      const int32_t tn = t + 1 < R ? t + 1 : (R > 0 ? R - 1 : 0);
      const int64_t g = base + tn;
      nx_arr = a.arrival[g];
      nx_p = a.plen[g];
      nx_o = a.olen[g];
      nx_oh = a.ohat[g];
      nx_c = a.cls[g];
    }
    const bool bad = act && (p < 1 || o < 1 || oh < 1 || (int64_t)p + o > INT32_MAX ||
                             (int64_t)p + oh > INT32_MAX || c >= (uint32_t)ncls || arr < 0 ||
                             (have_arr && arr < last_arr));
    const bool go = act && !bad;
    if (go) {
      last_arr = arr;
      have_arr = true;
    }
    const double now = i64_to_f64(arr);

    // 2. release everything that finished at or before now: one pop per
    // instance on the fast path; further pops (several completions between
    // two arrivals at one instance) on the slow path, which waits.
#pragma unroll
    for (int m = 0; m < MP; ++m)
      pop_fast<false>(pre[m], go && pre[m].q > 0 && pre[m].h_t <= now, a, dummy + 32, base, R);
#pragma unroll
    for (int m = 0; m < MD; ++m)
      pop_fast<true>(dec[m], go && dec[m].q > 0 && dec[m].h_t <= now, a, dummy + 32, base, R);
    {
      bool more = false;
#pragma unroll
      for (int m = 0; m < MP; ++m) more |= go && pre[m].q > 0 && pre[m].h_t <= now;
#pragma unroll
      for (int m = 0; m < MD; ++m) more |= go && dec[m].q > 0 && dec[m].h_t <= now;
      while (__any(more)) {
#pragma unroll
        for (int m = 0; m < MP; ++m)
          if (go && pre[m].q > 0 && pre[m].h_t <= now) pop_slow<false>(pre[m], a, base, R);
#pragma unroll
        for (int m = 0; m < MD; ++m)
          if (go && dec[m].q > 0 && dec[m].h_t <= now) pop_slow<true>(dec[m], a, base, R);
        more = false;
#pragma unroll
        for (int m = 0; m < MP; ++m) more |= go && pre[m].q > 0 && pre[m].h_t <= now;
#pragma unroll
        for (int m = 0; m < MD; ++m) more |= go && dec[m].q > 0 && dec[m].h_t <= now;
        // Leave the slow path with nothing of its own in flight, so that the
        // loads and register writes after it keep exact wait counts.
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
      }
    }

    // 3a. keys of every candidate under the point's policy
    float sg = sigma[0];
#pragma unroll
    for (int k = 1; k < kMaxClasses; ++k) sg = (c == (uint32_t)k) ? sigma[k] : sg;
    const float work_pre = w_s * (float)p * tau_pre;
    const float work_dec = w_s * (float)oh * tau_dec;
    const double need_pre = (double)p;
    const double need_dec = (double)p + (double)oh;

    uint32_t bk_pre = 0xffffffffu, bk_dec = 0xffffffffu;
    int32_t bm_pre = 0, bm_dec = 0;
    double bb_pre = 0.0;
#pragma unroll
    for (int m = 0; m < MP; ++m) {
      const int j = sl * MP + m;
      const float bl = mode == 0 ? (float)__builtin_fmax(pre[m].busy - now, 0.0) * 1e-9f
                                 : tau_pre * (float)pre[m].pend + pre_base * (float)pre[m].q;
      uint32_t key = cost_key(cost_eq(w_b, rho, w_q, bl, work_pre, sg, pre[m].kv + need_pre, inv_pre, pre[m].q));
      key = policy == 2 ? (uint32_t)pre[m].q : key;
      key = policy == 1 ? (j == rr_pre ? 0u : 1u) : key;
      key = (go && j < P) ? key : 0xffffffffu;
      if (key < bk_pre) {
        bk_pre = key;
        bm_pre = m;
        bb_pre = pre[m].busy;
      }
    }
#pragma unroll
    for (int m = 0; m < MD; ++m) {
      const int j = sl * MD + m;
      const float bl = mode == 0 ? (float)__builtin_fmax(dec[m].busy - now, 0.0) * 1e-9f
                                 : tau_dec * (float)dec[m].pend;
      uint32_t key = cost_key(cost_eq(w_b, rho, w_q, bl, work_dec, sg, dec[m].kv + need_dec, inv_dec, dec[m].q));
      key = policy == 2 ? (uint32_t)dec[m].q : key;
      key = policy == 1 ? (j == rr_dec ? 0u : 1u) : key;
      key = (go && j < D) ? key : 0xffffffffu;
      if (key < bk_dec) {
        bk_dec = key;
        bm_dec = m;
      }
    }

    // 3b. argmin per pool over the segment (lowest index on equal keys) and
    // the prefill winner's busy-until, known to every lane afterwards.
    int32_t ip, id;
    double busy_ip;
    {
      const uint32_t kp = seg_min<S>(bk_pre, lane);
      const uint32_t kd = seg_min<S>(bk_dec, lane);
      const int32_t wl_p = seg_first<S>(bk_pre == kp, lane);
      const int32_t wl_d = seg_first<S>(bk_dec == kd, lane);
      const bool own_p = wl_self == wl_p;
      const bool own_d = wl_self == wl_d;
      int32_t jp = wl_p * MP, jd = wl_d * MD;
      if constexpr (MP > 1) jp += (int32_t)seg_or<S>(own_p ? (uint32_t)bm_pre : 0u, lane);
      if constexpr (MD > 1) jd += (int32_t)seg_or<S>(own_d ? (uint32_t)bm_dec : 0u, lane);
      double bp = seg_bcast_f64<S>(bb_pre, own_p, lane);
      if constexpr (S > 64) {
        jp += wave * 64 * MP;
        jd += wave * 64 * MD;
        // combine the per-wave winners through LDS (double-buffered by step
        // parity: one barrier per step)
        Partial* buf = part + (t & 1) * kW;
        if (lane == 0) buf[wave] = Partial{kp, kd, jp, jd, bp};
        __syncthreads();
        Partial w0 = buf[0];
#pragma unroll
        for (int w = 1; w < kW; ++w) {
          const Partial x = buf[w];  // waves hold increasing index ranges
          if (x.key_pre < w0.key_pre) {
            w0.key_pre = x.key_pre;
            w0.idx_pre = x.idx_pre;
            w0.busy_pre = x.busy_pre;
          }
          if (x.key_dec < w0.key_dec) {
            w0.key_dec = x.key_dec;
            w0.idx_dec = x.idx_dec;
          }
        }
        jp = w0.idx_pre;
        jd = w0.idx_dec;
        bp = w0.busy_pre;
      }
      ip = jp;
      id = jd;
      busy_ip = bp;
    }

    // 3c. serve: prefill, KV transfer, decode, each FIFO in admission order
    // (every product below is an exact integer below the time limit)
    const double s_pre = __builtin_fma((double)p, pre_tok_ns, pre_base_ns);
    const double s_dec = (double)(o - 1) * dec_tok_ns;
    const double xfer = (double)p * xfer_tok_ns;
    const double pf_end = __builtin_fmax(now, busy_ip) + s_pre;
    const double kv_at = pf_end + xfer;
    int64_t d_out = -1;  // output index this lane writes
    int32_t d_ipre = 0, d_idec = 0;
    int64_t d_ttft = 0, d_span = 0;
    int64_t d_ps = -1;  // prefill successor slot this lane writes, and its record
    double d_pt = 0.0;
    int32_t d_pidx = 0, d_pp = 0;
    int64_t d_ds = -1;  // decode successor slot this lane writes, and its record
    double d_dt = 0.0;
    int32_t d_didx = 0, d_dfp = 0, d_dpt = 0;
#pragma unroll
    for (int m = 0; m < MP; ++m)
      if (go && sl * MP + m == ip) {
        d_ps = append(pre[m], pf_end, t, p, p, base);
        pre[m].busy = pf_end;
        d_pt = pf_end;
        d_pidx = t;
        d_pp = p;
      }
#pragma unroll
    for (int m = 0; m < MD; ++m)
      if (go && sl * MD + m == id) {
        const double dec_end = __builtin_fmax(kv_at, dec[m].busy) + s_dec;
        d_ds = append(dec[m], dec_end, t, p + o, oh, base);
        dec[m].busy = dec_end;
        d_dt = dec_end;
        d_didx = t;
        d_dfp = p + o;
        d_dpt = oh;
        // the decode owner records the outcome
        d_out = base + t;
        d_ipre = ip;
        d_idec = id;
        d_ttft = f64_to_i64(pf_end - now);
        d_span = f64_to_i64(dec_end - pf_end);
        flag |= dec_end >= kTimeLimit ? kFlagTimeRange : 0u;
      }
    if (bad && sl == 0) {
      d_out = base + t;
      d_ipre = d_idec = -1;
      d_ttft = d_span = -1;
      flag |= kFlagRejected;
    }

    // 4. the successor records loaded in 2 (the step's one wait).  The
    // scheduling barriers keep the wait after the step's arithmetic and before
    // its stores.
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int m = 0; m < MP; ++m) {
      merge_pending(pre[m]);
      pin_record(pre[m]);
    }
#pragma unroll
    for (int m = 0; m < MD; ++m) {
      merge_pending(dec[m]);
      pin_record(dec[m]);
    }
    __builtin_amdgcn_sched_barrier(0);

    // 5. stores, by the lanes that own them
    if (d_out >= 0) {
      a.i_pre[d_out] = d_ipre;
      a.i_dec[d_out] = d_idec;
      a.ttft[d_out] = d_ttft;
      a.span[d_out] = d_span;
    }
    if (d_ps >= 0) *rec_at<int4>(a, d_ps, kRecPairPre) = make_int4(__double2loint(d_pt), __double2hiint(d_pt), d_pidx, d_pp);
    if (d_ds >= 0) {
      *rec_at<int4>(a, d_ds, kRecPairDec) = make_int4(__double2loint(d_dt), __double2hiint(d_dt), d_didx, d_dfp);
      *rec_at<int32_t>(a, d_ds, kRecTokDec) = d_dpt;
    }
    rr_pre = (rr_pre + 1 == P) ? 0 : rr_pre + 1;
    rr_dec = (rr_dec + 1 == D) ? 0 : rr_dec + 1;
  }
  if (flag) atomicOr(a.flag, flag);
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

struct WideEntry {
  int S, MP, MD;
  hipError_t (*fn)(const SimArgs&, hipStream_t);
};

// Pools wider than one wave segment holds (the segment kernels take the
// rest); the host picks the first class that fits a point.
const WideEntry kWideTable[] = {
    {256, 1, 4, launch_one<256, 1, 4>},
    {512, 2, 2, launch_one<512, 2, 2>},
};

}  // namespace

int wide_class_count() { return (int)(sizeof(kWideTable) / sizeof(kWideTable[0])); }

SimClass wide_class(int i) {
  const WideEntry& e = kWideTable[i];
  return SimClass{kWide, e.S, e.MP, e.MD, kModeAny};
}

hipError_t launch_wide_class(const SimClass& c, const SimArgs& a, hipStream_t stream) {
  for (const WideEntry& e : kWideTable)
    if (e.S == c.S && e.MP == c.MP && e.MD == c.MD) return e.fn(a, stream);
  return hipErrorInvalidValue;
}

int sim_class_count() { return seg_class_count() + wide_class_count(); }

SimClass sim_class(int i) { return i < seg_class_count() ? seg_class(i) : wide_class(i - seg_class_count()); }

hipError_t launch_sim(const SimClass& c, const SimArgs& a, hipStream_t stream) {
  return c.kind == kWide ? launch_wide_class(c, a, stream) : launch_seg_class(c, a, stream);
}

}  // namespace rt
