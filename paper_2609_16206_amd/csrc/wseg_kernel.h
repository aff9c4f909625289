// Replica-batched simulation of the learned prefill/decode router for pools
// wider than one wave, on gfx950.
//
// Method and per-instance machinery as in seg_kernel.h (Algorithm 1 per
// admission on the serial-service simulator of Section III-D / Section VI;
// Section III-A costs; the register FIFO window with successor records
// written only beyond the window).  Differences for wide pools:
//
// Mapping.  One replica per workgroup of W waves.  Instances are dealt to the
// waves round robin (instance j of a pool to wave j mod W), so that runs of
// low-index instances, which win the ties of idle instances, spread over all
// waves.  In wave w the first LPW lanes hold prefill instances
// w + W * (lane * M + m) and the next LDW lanes decode instances
// w + W * ((lane - LPW) * M + m), m < M.  Everything per request is uniform
// over the workgroup.
//
// Issue model.  A wave issues about one instruction every four cycles,
// vector, scalar, branch or LDS alike, and the step is a chain of dependent
// work ending in a barrier, so the kernel is written for the fewest
// instructions per step rather than for the fewest vector ones; two waves
// per SIMD (eight per workgroup) let one wave's waits overlap the other's
// issue, which pays more than the extra lanes cost (the large pool's 1,152
// instances run at three per lane on eight waves).
//
// Requests.  The terms a step needs from its request (arrival, service
// times, priced work and cache need per pool, sigma, the sampled
// candidates) are derived once per block of 64 requests, lane k of every
// wave working on request (block start + k), and left in LDS; a step reads
// its request's record (96 bytes) from LDS one step ahead.  Admission (valid
// lengths and class, arrival not before the last accepted one) is decided
// for the whole block at once: a request is accepted if valid and its
// arrival equals the running maximum of the valid arrivals so far, a prefix
// maximum taken with DPP across the wave (the last accepted arrival is the
// largest valid one before it, whether accepted or not).  The raw trace of a
// block is loaded two blocks ahead.
//
// Argmin.  Every lane that holds instances folds its best slot (the lowest
// slot of the lane's smallest cost key) into the LDS minimum of its pool,
// packed as (cost key << 32 | instance index << 14 | FIFO position << 12 |
// slot << 9 | cell), and writes that slot's busy-until to its own cell
// (wave * 64 + lane).  The 64-bit minimum keeps the smallest key and, among
// equal keys, the lowest index; the bits below the index never decide
// (indices are unique), and they hand the winner's wave, lane, slot and
// queue length (capped at 3: beyond the window) to the append as scalars.
// No reduction within the wave precedes the fold: a DPP argmin with its
// scalar winner lookup was a chain of vector-to-scalar round trips, and the
// LDS takes a few hundred atomics per step without becoming the bound.  After one barrier per step (it
// orders LDS only: every global access of a wave is to addresses no other
// wave touches) every wave reads both minima and then the two winners'
// busy-until from the cells they name, so all waves form the same prefill
// and decode ends.
// The LDS cells rotate over three step slots: slot t % 3 is filled at step
// t, read after its barrier, and reset by wave 0 after the barrier of step
// t + 1 (every wave has read it by then, and none writes it again before the
// barrier of step t + 2).
//
// Sparse work.  The releases run only when some head of the wave has
// finished (slot by slot, again while a head is still finished), a refill
// from the successor records only where a queue is deeper than the window
// (loaded and merged at once), and the appends, whose FIFO position is the
// winner's queue length read as a scalar, touch scratch only beyond the
// register window.  Each slot keeps its queue term w_q * queue (and,
// pricing the ledger, its ledger backlog), which change only with its
// queue, cached.  The step loop is unrolled by two, so that the request
// records alternate between two register sets.
//
// Outcomes.  Each output array is kept by one wave (wave a keeps array a
// with four or more waves; with two, each keeps two): lane k holds the
// value of step (block start + k), and the block is written with one
// coalesced store per array.
#pragma once

#include "seg_kernel.h"

namespace rt {
namespace seg {

// Lanes per wave holding a pool of n instances, dealt round robin to W waves
// at M per lane.
__host__ __device__ inline int wide_pool_lanes(int n, int M, int W) { return ((n + W - 1) / W + M - 1) / M; }

__device__ __forceinline__ double rl_f64(double v, int lane) {
  return __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(v), lane),
                          __builtin_amdgcn_readlane(__double2loint(v), lane));
}

// One instance of the wide kernel: the state the score reads, and the first
// three positions of its FIFO (t = +inf beyond it).  A refill from the
// successor records is loaded and merged at once (rare: only queues deeper
// than the window need one), so no load is carried between steps.
struct WSlot {
  double busy;   // end of everything admitted so far
  double kv;     // cache tokens in flight
  double pend;   // ledger tokens in flight
  int32_t q;     // requests in flight
  int32_t tail;  // last admitted request
  int32_t tail2; // the one admitted before it
  Elem h, n, n2; // FIFO positions 0, 1, 2
};

__device__ __forceinline__ void init_wslot(WSlot& s) {
  s.busy = s.kv = s.pend = 0.0;
  s.q = 0;
  s.tail = s.tail2 = -1;
  s.h = s.n = s.n2 = none();
}

// The releases of one slot by `now_eff`, on the lanes whose head has
// finished: up to two from the window, then the positions the shift left
// empty refilled from the new head's record (refill_mask), loaded and
// merged here where any lane of the wave needs one.
template <bool kTok, bool kKv>
__device__ __forceinline__ void wrelease(WSlot& x, double now_eff, const char* recr, int32_t R, int64_t dmy) {
  const bool p1 = x.h.t <= now_eff;
  const bool p2 = x.n.t <= now_eff;  // implies p1 (release times do not decrease)
  x.q -= (p1 ? 1 : 0) + (p2 ? 1 : 0);
  if constexpr (kKv) x.kv = x.kv - ((p1 ? (double)x.h.fp : 0.0) + (p2 ? (double)x.n.fp : 0.0));
  if constexpr (kTok) x.pend = x.pend - ((p1 ? (double)x.h.pt : 0.0) + (p2 ? (double)x.n.pt : 0.0));
  const Elem h1 = sel(p2, x.n2, sel(p1, x.n, x.h));
  Elem n1 = sel(p1, x.n2, x.n);
  n1.t = p2 ? kInf : n1.t;
  x.h = h1;
  x.n = n1;
  x.n2.t = p1 ? kInf : x.n2.t;
  const int32_t lq = opaque(refill_mask(p1, p2, x.q));
  if (__any(lq != 0)) {
    const int64_t g = sel_index(lq != 0, min(max(x.h.idx, 0), max(R - 1, 0)), dmy);
    Slot tmp;
    load_pair<kTok>(tmp, rec_at<kTok>(recr, g));
    x.n = sel((lq & 1) != 0, tmp.l1, x.n);
    x.n2 = sel((lq & 2) != 0, tmp.l2, x.n2);
  }
}

template <int M>
__device__ __forceinline__ double head_min_w(const WSlot (&s)[M]) {
  double h = s[0].h.t;
#pragma unroll
  for (int m = 1; m < M; ++m) h = __builtin_fmin(h, s[m].h.t);
  return h;
}

// A request as a step of the wide kernel reads it (96 bytes).
struct alignas(16) WReq {
  double now;             // arrival (ns) if the request is accepted, else -1
  double s_pre;           // prefill service
  double xfer;            // KV transfer delay
  double s_dec;           // decode service
  double need_p, need_d;  // cache tokens it needs on a prefill / decode instance
  float work_p, work_d;   // priced work w_s * tokens * tau of each pool
  float sg;               // sigma of its class
  int32_t p, po, oh;      // prompt, prompt + output, predicted output
  uint32_t cand[4];       // sampled candidates: prefill c1, c2, decode c1, c2
  int32_t pad[2];
};
static_assert(sizeof(WReq) == 96, "six 16-byte words");

// One step of a wave-wide scan of doubles: x = max(x, x of the lane the DPP
// control names); a lane without a source reads +0 (full row mask) or keeps
// its value (partial row mask).
template <int C, int RM>
__device__ __forceinline__ double dpp_max_f64(double x) {
  const int lo = __double2loint(x), hi = __double2hiint(x);
  const int slo = __builtin_amdgcn_update_dpp(RM == 0xF ? 0 : lo, lo, C, RM, 0xF, RM == 0xF);
  const int shi = __builtin_amdgcn_update_dpp(RM == 0xF ? 0 : hi, hi, C, RM, 0xF, RM == 0xF);
  return __builtin_fmax(x, __hiloint2double(shi, slo));
}

// Inclusive prefix maximum over the wave of doubles >= -1 (lanes in order;
// +0 enters as the maximum's floor): shifts of 1, 2, 4, 8 within each row of
// 16 lanes, then the last lane of each row into the rows after it.
__device__ __forceinline__ double wave_prefix_max(double x) {
  x = dpp_max_f64<0x111, 0xF>(x);  // row_shr:1
  x = dpp_max_f64<0x112, 0xF>(x);  // row_shr:2
  x = dpp_max_f64<0x114, 0xF>(x);  // row_shr:4
  x = dpp_max_f64<0x118, 0xF>(x);  // row_shr:8
  x = dpp_max_f64<0x142, 0xA>(x);  // row_bcast:15 into rows 1 and 3
  x = dpp_max_f64<0x143, 0xC>(x);  // row_bcast:31 into rows 2 and 3
  return x;
}

template <int W, int M, int kMode>
__global__ void __launch_bounds__(64 * W) wseg_kernel(SimArgs a) {
  static_assert(W == 2 || W == 4 || W == 8, "workgroups of 2, 4 or 8 waves");
  // (instance indices, below the boundary's pool limit of 1,024, fit the
  // 18 bits above them)
  static_assert(W * 64 <= 512 && M <= 8, "cell and slot fit their bits of the packed minimum");
  constexpr bool kTok = mode_ledger(kMode);    // the ledger is priced
  constexpr bool kKv = kMode != kModeBase;     // occupancy is priced
  constexpr bool kSamp = mode_sampled(kMode);  // two candidates per pool
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int rep = a.work[blockIdx.x];
  const int64_t base = a.offsets[rep];
  const int32_t R = (int32_t)(a.offsets[rep + 1] - base);  // >= 1: empty replicas are not launched
  const int pid = a.param_point ? a.param_point[rep] : 0;
  const DevPoint& pt = a.points[pid];
  const int32_t P = pt.P, D = pt.D, ncls = pt.n_classes, policy = pt.policy;
  const bool thr = policy == kPolicyLengthThreshold;
  const int32_t half_d = (D + 1) / 2;  // first instance of the decode pool's upper part
  const int32_t len_thr = pt.len_thr;
  const int32_t LPW = wide_pool_lanes(P, M, W), LDW = wide_pool_lanes(D, M, W);
  const bool isp = lane < LPW;
  const int32_t lrel = isp ? lane : lane - LPW;  // lane within the pool's lanes of this wave
  // instance m of this lane: wave + W * (lrel * M + m)
  const int32_t npool = isp ? P : D;
  const bool inpool = lane < LPW + LDW;
  const float w_b = pt.w_b, w_q = pt.w_q, rho = pt.rho;
  const float inv = isp ? pt.inv_cap_pre : pt.inv_cap_dec;
  const float tau = isp ? pt.tau_pre : pt.tau_dec;
  const float basec = isp ? pt.pre_base : 0.0f;  // proxy ledger: base per in-flight prefill
  char* const recb = isp ? a.rec[0] : a.rec[1];
  const uint32_t wave_id = (blockIdx.x * W + wave) & (kDummyRecords - 1);
  // the lane's plane at its replica's request 0; the wave's dummy record,
  // indexed relative to it
  char* const recr = recb + rec_off<kTok>(base);
  const int64_t dmy = -1 - (int64_t)wave_id - base;

  __shared__ unsigned long long best[3][2];  // per step slot: packed minimum of each pool
  __shared__ double wbusy[3][W * 64];         // per step slot: each lane's best busy-until
  __shared__ WReq reqs[2][64];               // request records of the current and the next block
  if (threadIdx.x < 6) best[threadIdx.x >> 1][threadIdx.x & 1] = ~0ull;

  WSlot s[M];
  bool ok[M];    // the slot holds an instance of the lane's pool
  float wqq[M];  // w_q * (float)queue of each slot
  float blv[M];  // ledger backlog of each slot (ledger modes)
  // (slot indices compile-time from the start: a loop here left the slot
  // array in scratch memory in the ledger modes)
  static_for<M>([&](auto mc) __attribute__((always_inline)) {
    constexpr int m = decltype(mc)::value;
    init_wslot(s[m]);
    ok[m] = inpool && wave + W * (lrel * M + m) < npool;
  });
  // a slot's cached queue and ledger terms, after its queue or ledger changed
  auto refresh = [&](int m) __attribute__((always_inline)) {
    wqq[m] = w_q * (float)s[m].q;
    if constexpr (kTok) blv[m] = tau * (float)s[m].pend + basec * (float)s[m].q;
  };
  static_for<M>([&](auto mc) __attribute__((always_inline)) { refresh(decltype(mc)::value); });

  // Raw trace of a block, lane k holding request (block start + k) (clamped
  // into the replica; lanes past its end are rejected when the block's
  // records are made).
  struct Raw {
    int64_t arr;
    int32_t p, o, oh;
    uint32_t c;
    uint32_t w[4];  // candidate words (sampled modes)
  };
  auto load_raw = [&](Raw& f, int32_t blk) __attribute__((always_inline)) {
    const int64_t g = base + min(blk + lane, R - 1);
    f.arr = a.arrival[g];
    f.p = a.plen[g];
    f.o = a.olen[g];
    f.oh = a.ohat[g];
    f.c = a.cls[g];
    if constexpr (kSamp) {
      const uint4 w = *reinterpret_cast<const uint4*>(a.samp + 4 * g);
      f.w[0] = w.x;
      f.w[1] = w.y;
      f.w[2] = w.z;
      f.w[3] = w.w;
    } else {
      f.w[0] = f.w[1] = f.w[2] = f.w[3] = 0;
    }
  };
  // The records of block `blk` from its raw trace, into reqs[buf]; `carry`
  // is the largest valid arrival before the block (0 before the first).
  const double pre_base_ns = (double)pt.pre_base_ns, pre_tok_ns = (double)pt.pre_tok_ns;
  const double dec_tok_ns = (double)pt.dec_tok_ns, xfer_tok_ns = (double)pt.xfer_tok_ns;
  const float w_s = pt.w_s, tau_pre = pt.tau_pre, tau_dec = pt.tau_dec;
  const float sig_l = pt.sigma[lane & (kMaxClasses - 1)];  // lane k: sigma of class k mod 8
  double carry = 0.0;
  auto make_block = [&](const Raw& f, int32_t blk, int buf) __attribute__((always_inline)) {
    const int32_t p = f.p, o = f.o, oh = f.oh;
    const int32_t po = (int32_t)((uint32_t)p + (uint32_t)o), poh = (int32_t)((uint32_t)p + (uint32_t)oh);
    const int32_t vm = min(min(min(p, o), min(oh, po)), min(min(poh, ncls - (int32_t)f.c), R - (blk + lane)));
    const bool valid = opaque(vm) >= 1;
    const double x = valid ? i64_to_f64(f.arr) : -1.0;
    const double incl = __builtin_fmax(wave_prefix_max(x), carry);
    carry = rl_f64(incl, 63);
    WReq r;
    r.now = (valid && x == incl) ? x : -1.0;
    r.s_pre = __builtin_fma((double)p, pre_tok_ns, pre_base_ns);
    r.xfer = (double)p * xfer_tok_ns;
    r.s_dec = (double)(o - 1) * dec_tok_ns;
    r.need_p = (double)p;
    r.need_d = (double)poh;
    r.work_p = w_s * (float)p * tau_pre;
    r.work_d = w_s * (float)oh * tau_dec;
    r.sg = __builtin_bit_cast(
        float, __builtin_amdgcn_ds_bpermute((int)((f.c & (kMaxClasses - 1)) << 2), __builtin_bit_cast(int, sig_l)));
    r.p = p;
    r.po = po;
    r.oh = oh;
    if constexpr (kSamp) {
      sample_pair(f.w[0], f.w[1], (uint32_t)P, r.cand[0], r.cand[1]);
      sample_pair(f.w[2], f.w[3], (uint32_t)D, r.cand[2], r.cand[3]);
    } else {
      r.cand[0] = r.cand[1] = r.cand[2] = r.cand[3] = 0;
    }
    r.pad[0] = r.pad[1] = 0;
    reqs[buf][lane] = r;
  };

  Raw raw;
  load_raw(raw, 0);
  make_block(raw, 0, 0);
  load_raw(raw, 64);
  __syncthreads();
  WReq rq = reqs[0][0];  // the current request's record

  // outcomes of the current block kept by this wave (lane k: step block
  // start + k): an int32 array (0 i_pre, 1 i_dec) and an int64 array (0
  // ttft, 1 span), or none (-1)
  const int oi = W == 2 ? wave : (wave < 2 ? wave : -1);
  const int ol = W == 2 ? wave : (wave == 2 ? 0 : (wave == 3 ? 1 : -1));
  int32_t b32 = -1;
  int64_t b64 = -1;
  int32_t rr = 0;     // round robin: t mod (size of this lane's pool)
  double tmax = 0.0;  // latest decode end (time-range check)
  bool rej = false;   // a request was rejected
  int sl3 = 0;        // step slot t % 3 of the LDS cells

  // one step; request t's record is rq, request t+1's is read into rn
  auto step = [&](const int32_t t, WReq& rq, WReq& rn) __attribute__((always_inline)) {
    // at a block boundary: the records of the next block, and the raw trace
    // of the one after it
    if ((t & 63) == 0) {
      make_block(raw, t + 64, ((t >> 6) + 1) & 1);
      load_raw(raw, t + 128);
    }
    const double now = rq.now;
    const bool go = now >= 0.0;

    // 1. score this lane's instances
    const float work = isp ? rq.work_p : rq.work_d;
    const double need = isp ? rq.need_p : rq.need_d;
    const float sg = rq.sg;
    const bool long_req = rq.oh >= len_thr;  // length threshold: the upper part
    uint32_t bkey = 0xffffffffu;
    int32_t bm = 0;
    int32_t bq = s[0].q;
    double bbusy = s[0].busy;
    const uint32_t c1 = isp ? rq.cand[0] : rq.cand[2], c2 = isp ? rq.cand[1] : rq.cand[3];
#pragma unroll
    for (int m = 0; m < M; ++m) {
      const WSlot& x = s[m];
      uint32_t key;
      if constexpr (kMode == kModeBase) {
        // round robin; least loaded; or least loaded within the decode
        // part the request's predicted length picks (length threshold)
        const int32_t j = (wave + W * (lrel * M + m));
        key = policy == kPolicyRoundRobin ? (j == rr ? 0u : 1u) : (uint32_t)x.q;
        const bool part = D == 1 || ((j >= half_d) == long_req);
        key = (thr && !isp && !part) ? 0xffffffffu : key;
      } else {
        float bl;
        if constexpr (!kTok)
          bl = (float)__builtin_fmax(x.busy - now, 0.0) * 1e-9f;
        else
          bl = blv[m];
        const float press = (float)(x.kv + need) * inv;
        const float load = w_b * bl * sg;
        const float size = work * (1.0f + rho * press) * sg;
        const float cost = load + size + wqq[m];
        key = cost != cost ? 0x7fc00000u : __float_as_uint(cost);
      }
      if constexpr (kSamp) {
        const uint32_t j = (uint32_t)(wave + W * (lrel * M + m));
        key = (j == c1 || j == c2) ? key : 0xffffffffu;
      }
      key = ok[m] ? key : 0xffffffffu;
      if (m == 0) {
        bkey = key;
      } else {
        const bool b = key < bkey;
        bkey = b ? key : bkey;
        bm = b ? m : bm;
        bq = b ? x.q : bq;
        bbusy = b ? x.busy : bbusy;
      }
    }

    // 2. every lane holding instances folds its best slot into its pool's
    // LDS minimum and leaves that slot's busy-until in its cell
    if (inpool) {
      const uint32_t cell = (uint32_t)(wave * 64 + lane);
      const uint32_t idx = (uint32_t)(wave + W * (lrel * M + bm));
      const uint32_t wq = (uint32_t)min(bq, 3);  // the FIFO position the request would take
      atomicMin(&best[sl3][isp ? 0 : 1],
                ((unsigned long long)bkey << 32) | (idx << 14) | (wq << 12) | ((uint32_t)bm << 9) | cell);
      wbusy[sl3][cell] = bbusy;
    }
    lds_barrier();
    const uint32_t bpl = (uint32_t)best[sl3][0], bdl = (uint32_t)best[sl3][1];
    const uint32_t bps = (uint32_t)__builtin_amdgcn_readfirstlane((int32_t)bpl);
    const uint32_t bds = (uint32_t)__builtin_amdgcn_readfirstlane((int32_t)bdl);
    const int32_t ip = (int32_t)(bps >> 14), id = (int32_t)(bds >> 14);
    const double busy_ip = wbusy[sl3][bps & 511u];
    const double busy_id = wbusy[sl3][bds & 511u];
    // the cells of step t - 1 are free again (every wave has read them)
    const int sl_prev = sl3 == 0 ? 2 : sl3 - 1;
    if (wave == 0 && lane < 2) best[sl_prev][lane] = ~0ull;
    // the next request's record (read a step ahead)
    rn = reqs[((t + 1) >> 6) & 1][(t + 1) & 63];

    // 3. serve (uniform): prefill, KV transfer, decode (exact integers in
    // doubles)
    const double pf_end = max_f64(now, busy_ip) + rq.s_pre;
    const double kv_at = pf_end + rq.xfer;
    const double de = max_f64(kv_at, busy_id) + rq.s_dec;

    // 5. append the request to the winning slot of each pool (uniform
    // branches: the winner's wave and slot, then its FIFO position)
    if (go) {
      auto append = [&](uint32_t pk, double end, int32_t fp, int32_t tk)
                        __attribute__((always_inline)) {
        const int32_t lw = (int32_t)(pk & 63u);        // lane
        const int32_t mw = (int32_t)((pk >> 9) & 7u);  // slot
        const int32_t w = (int32_t)((pk >> 12) & 3u);  // z's FIFO position (3: beyond the window)
        const bool own = lane == lw;
        const Elem z{end, t, fp, tk};
        static_for<M>([&](auto mc) __attribute__((always_inline)) {
          constexpr int m = decltype(mc)::value;
          if (m != mw) return;
          WSlot& x = s[m];
          x.h = sel(own && w == 0, z, x.h);
          x.n = sel(own && w == 1, z, x.n);
          x.n2 = sel(own && w == 2, z, x.n2);
          if (w >= 3) {
            // beyond the window: z is the first successor of the tail and
            // the second of the request before it
            if (own) {
              char* const r1 = rec_at<kTok>(recr, x.tail);
              char* const r2 = rec_at<kTok>(recr, x.tail2);
              *reinterpret_cast<Entry*>(r1) = Entry{end, t, fp};
              *reinterpret_cast<Entry*>(r2 + 16) = Entry{end, t, fp};
              if constexpr (kTok) {
                *reinterpret_cast<int32_t*>(r1 + kRecTok) = tk;
                *reinterpret_cast<int32_t*>(r2 + kRecTok + 4) = tk;
              }
            }
          }
          const int32_t tl_old = x.tail;
          x.tail2 = own ? tl_old : x.tail2;
          x.tail = own ? t : tl_old;
          x.q = own ? x.q + 1 : x.q;
          if constexpr (kKv) x.kv = x.kv + (own ? (double)fp : 0.0);
          if constexpr (kTok) x.pend = x.pend + (own ? (double)tk : 0.0);
          x.busy = own ? end : x.busy;
          refresh(m);
        });
      };
      if (wave == (ip & (W - 1))) append(bps, pf_end, rq.p, rq.p);
      if (wave == (id & (W - 1))) append(bds, de, rq.po, rq.oh);
    }

    // 6. the outcome: each array kept by its wave, written per block of 64
    {
      const bool keep = lane == (t & 63);
      if (oi >= 0) b32 = keep ? (go ? (oi == 0 ? ip : id) : -1) : b32;
      if (ol >= 0) b64 = keep ? (go ? f64_to_i64(ol == 0 ? pf_end - now : de - pf_end) : -1) : b64;
      if ((t & 63) == 63 || t == R - 1) {
        const int32_t tl = (t & ~63) + lane;
        if (tl <= t) {
          const int64_t gi = base + tl;
          if (oi >= 0) (oi == 0 ? a.i_pre : a.i_dec)[gi] = b32;
          if (ol >= 0) (ol == 0 ? a.ttft : a.span)[gi] = b64;
        }
      }
    }
    tmax = go ? __builtin_fmax(tmax, de) : tmax;
    rej = rej || !go;
    if constexpr (kMode == kModeBase) rr = (rr + 1 == npool) ? 0 : rr + 1;
    sl3 = sl3 == 2 ? 0 : sl3 + 1;

    // 7. the releases for request t+1: slot by slot where some lane's head
    // has finished, again while a head is still finished (more releases
    // than the window holds)
    {
      const double now_eff = rn.now;
      bool done = false;
#pragma unroll
      for (int m = 0; m < M; ++m) done = done || s[m].h.t <= now_eff;
      if (__any(done)) {
        static_for<M>([&](auto mc) __attribute__((always_inline)) {
          constexpr int m = decltype(mc)::value;
          if (__any(s[m].h.t <= now_eff)) {
            wrelease<kTok, kKv>(s[m], now_eff, recr, R, dmy);
            refresh(m);
          }
        });
        if (__builtin_expect(__any(head_min_w(s) <= now_eff), 0)) {
          do {
            static_for<M>([&](auto mc) __attribute__((always_inline)) {
              constexpr int m = decltype(mc)::value;
              if (__any(s[m].h.t <= now_eff)) {
                wrelease<kTok, kKv>(s[m], now_eff, recr, R, dmy);
                refresh(m);
              }
            });
          } while (__any(head_min_w(s) <= now_eff));
        }
      }
    }
  };
  // two steps per trip, so that the records alternate between two register
  // sets instead of being copied
  WReq rb;
  for (int32_t t = 0; t < R; t += 2) {
    step(t, rq, rb);
    if (t + 1 < R) step(t + 1, rb, rq);
  }
  if (wave == 0 && lane == 0) {
    const uint32_t flag = (tmax >= kTimeLimit ? kFlagTimeRange : 0u) | (rej ? kFlagRejected : 0u);
    if (flag) atomicOr(a.flag, flag);
  }
}

template <int W, int M, int kMode>
hipError_t launch_wseg(const SimArgs& a, hipStream_t stream) {
  if (a.n_work <= 0) return hipSuccess;
  hipLaunchKernelGGL((wseg_kernel<W, M, kMode>), dim3((unsigned)a.n_work), dim3(64 * W), 0, stream, a);
  return hipGetLastError();
}

// The workgroup widths (waves) and lane depths compiled for every mode, in
// order of preference: at most one wave per SIMD of a compute unit first
// (then fewer instances per lane), then eight waves.
#define RT_WSEG_FOR_EACH(X) X(2, 2) X(4, 2) X(2, 3) X(4, 3) X(8, 3) X(4, 5) X(8, 2) X(8, 5)

template <int kMode>
hipError_t launch_wide_mode(int W, int M, const SimArgs& a, hipStream_t stream);

}  // namespace seg
}  // namespace rt
