// Replica-batched simulation of the learned prefill/decode router for pools
// that fit one wave, on gfx950.
//
// Method: Algorithm 1 per admission (score every instance of both pools with
// the Section III-A cost equation, take each pool's argmin, prefill, transfer
// the KV cache, decode, record), on the serial-service simulator of Section
// III-D / Section VI.
//
// Mapping.  A replica is a chain of admissions; replicas are independent.
// One replica occupies an aligned segment of S lanes of one wave (64 / S
// replicas per wave).  Lanes [0, LP) hold the prefill instances and lanes
// [LP, LP + LD) the decode instances, M per lane in blocked order (instance
// j of a pool sits in that pool's lane j / M, slot j % M), so every lane
// scores a single pool and the lowest lane holding a pool's minimum also
// holds its lowest index.  Per-instance state (busy-until, queue, cache
// occupancy, ledger tokens, the first three requests of its FIFO) lives in
// registers; the per-request terms are computed by every lane of the
// segment.  The two argmins are DPP reductions within 16-lane rows plus
// readlane across rows.
//
// Issue model.  One wave per SIMD issues one instruction every ~4 cycles; a
// lane mask written by a vector compare and read by the scalar unit, and a
// taken branch, each cost several issue slots more.  The step is therefore
// written so that every condition is a single vector compare feeding vector
// selects (sentinels fold the conditions: a FIFO position beyond the FIFO's
// length has release time +inf, and a rejected request uses now = -1, so
// "the head has finished" is the one compare head <= now), and every record
// load and store is issued unconditionally (a lane with nothing to load or
// store addresses its wave's dummy slot).  The only branches of a step are
// the loop and a rare slow path.
//
// Outcomes.  A store sends one write request per enabled lane, wherever it
// points, so the step does not store outcomes: lane k of a segment keeps the
// outcome of step (block start + k), and every S steps the segment writes
// the block with one coalesced store per output array.
//
// FIFO of in-flight requests per instance.  Service is in admission order,
// so an instance releases its requests in admission order.  The first three
// requests of each FIFO (positions 0, 1, 2) are kept in registers; the rest
// is a list in HBM scratch in which a request's record holds its first and
// second successor (release time, index, cache tokens: one 32-byte sector;
// ledger tokens after them in the modes that price the ledger).  Records are
// written only when a request joins beyond the register window (position
// 3 or later): it is then stored as the first successor of the request
// ahead of it and as the second successor of the one ahead of that.  So the
// record of the request at position p holds a valid first successor when
// p >= 2 and a valid second successor when p >= 1 (where those successors
// exist), and a FIFO that never grows past three requests never touches
// scratch.  Up to two releases per instance between two arrivals shift the
// register window; the positions the shift leaves empty are then filled
// from the new head's record, loaded with one independent access (no chain
// of dependent loads) and merged at the end of the step: after one release
// only position 2 (the new head's second successor), after two releases
// positions 1 and 2.  A third release in one step takes the slow path,
// which waits.
//
// Memory ordering within a step (one wave): on gfx9 loads and stores share
// one counter, so a wait for a load also waits for every older store.  The
// step issues its loads (the next request, the successor pairs) before its
// one wait, which it places after the arithmetic and before its own stores.
// An instance's records are written and read by the one lane that owns it,
// in program order, so a record is visible to every later load of it.
//
// Arithmetic of the cost: evaluated exactly as the equation is written, left
// to right in float32, one rounding per operation (built with
// -ffp-contract=off).  Times and token totals are integers held in doubles
// (exact below 2^53; simulated times are kept below 2^52).
#pragma once

#include <algorithm>

#include "lane_ops.h"
#include "rt_internal.h"

namespace rt {
namespace seg {

constexpr double kInf = __builtin_huge_val();

// One FIFO position: release time, request index, cache tokens, ledger tokens.
struct Elem {
  double t;
  int32_t idx, fp, pt;
};

// A stored entry as it lies in scratch (16 bytes; ledger tokens apart).
struct alignas(16) Entry {
  double t;
  int32_t idx, fp;
};

struct alignas(16) EntryPair {
  Entry a, b;
};

struct Slot {
  double busy;      // end of everything admitted so far
  double kv;        // cache tokens in flight
  double pend;      // ledger tokens in flight
  int32_t q;        // requests in flight
  int32_t tail;     // last admitted request
  int32_t tail2;    // the one admitted before it
  Elem h, n, n2;    // FIFO positions 0, 1, 2 (t = +inf beyond the FIFO)
  Elem l1, l2;      // successors of the head, loaded this step
  int32_t lq;       // positions the loaded pair fills: bit 0 position 1,
                    // bit 1 position 2 (0: nothing loaded)
};

__device__ __forceinline__ Elem none() { return Elem{kInf, 0, 0, 0}; }

__device__ __forceinline__ void init_slot(Slot& s) {
  s.busy = s.kv = s.pend = 0.0;
  s.q = 0;
  s.tail = s.tail2 = -1;
  s.h = s.n = s.n2 = none();
  s.l1 = s.l2 = Elem{0.0, 0, 0, 0};
  s.lq = 0;
}

__device__ __forceinline__ Elem sel(bool c, const Elem& x, const Elem& y) {
  return Elem{c ? x.t : y.t, c ? x.idx : y.idx, c ? x.fp : y.fp, c ? x.pt : y.pt};
}

// The loaded successors fill the positions the last release left empty.
__device__ __forceinline__ void merge_pending(Slot& s) {
  const bool m1 = (s.lq & 1) != 0, m2 = (s.lq & 2) != 0;
  s.n = sel(m1, s.l1, s.n);
  s.n2 = sel(m2, s.l2, s.n2);
  s.lq = 0;
}

// Materializes the merged positions here, ahead of every later memory
// instruction (an empty volatile asm that reads the registers and clobbers
// memory), so that the wait for their load is not pushed past the stores.
// Without a priced ledger the positions' ledger tokens are never read, and
// are not pinned (so their selects are dropped).
template <bool kTok>
__device__ __forceinline__ void pin_window(const Slot& s) {
  if constexpr (kTok)
    asm volatile("" ::"v"(s.n.t), "v"(s.n.idx), "v"(s.n.fp), "v"(s.n.pt), "v"(s.n2.t), "v"(s.n2.idx), "v"(s.n2.fp),
                 "v"(s.n2.pt)
                 : "memory");
  else
    asm volatile("" ::"v"(s.n.t), "v"(s.n.idx), "v"(s.n.fp), "v"(s.n2.t), "v"(s.n2.idx), "v"(s.n2.fp) : "memory");
}

// Byte offset of request g's record in its pool's plane (a shift that folds
// into the address add).
template <bool kTok>
__device__ __forceinline__ int64_t rec_off(int64_t g) {
  return g << rec_shift(kTok);
}

// Address of record g of a plane based at p.  (A single v_lshl_add_u64
// takes shifts of 0..4 only; records are 32 or 64 bytes.)
template <bool kTok>
__device__ __forceinline__ char* rec_at(const char* p, int64_t g) {
  return const_cast<char*>(p) + rec_off<kTok>(g);
}

// The 64-bit index `x` where `c` holds, else `d` (x >= 0): the two halves
// selected apart, with no sign extension of x.
__device__ __forceinline__ int64_t sel_index(bool c, int32_t x, int64_t d) {
  const uint32_t lo = c ? (uint32_t)x : (uint32_t)(uint64_t)d;
  const uint32_t hi = c ? 0u : (uint32_t)((uint64_t)d >> 32);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

template <bool kTok>
__device__ __forceinline__ void load_pair(Slot& s, const char* rp) {
  const EntryPair e = *reinterpret_cast<const EntryPair*>(rp);
  s.l1 = Elem{e.a.t, e.a.idx, e.a.fp, e.a.fp};
  s.l2 = Elem{e.b.t, e.b.idx, e.b.fp, e.b.fp};
  if constexpr (kTok) {
    const int2 k = *reinterpret_cast<const int2*>(rp + kRecTok);
    s.l1.pt = k.x;
    s.l2.pt = k.y;
  }
}

// A request as the step sees it: checked, with its derived token sums.
struct Req {
  double now, now_eff;
  int32_t p, o, oh, po, poh;
  bool go;
};

// Request validity: lengths >= 1, token sums within int32, class in range,
// the step belongs to the replica (rem >= 1), arrival >= 0 and not before
// the last accepted one.  A rejected request is not routed and changes no
// state; it releases nothing (now_eff = -1).
__device__ __forceinline__ Req admit_check(int32_t rem, int32_t ncls, int64_t arr, int32_t p, int32_t o, int32_t oh,
                                           uint32_t c, double& last_now) {
  Req q;
  q.p = p;
  q.o = o;
  q.oh = oh;
  q.po = (int32_t)((uint32_t)p + (uint32_t)o);
  q.poh = (int32_t)((uint32_t)p + (uint32_t)oh);
  const int32_t vm = min(min(min(p, o), min(oh, q.po)), min(min(q.poh, ncls - (int32_t)c), rem));
  q.now = i64_to_f64(arr);
  const double xv = opaque(vm) >= 1 ? q.now : -1.0;
  q.go = xv >= last_now;
  q.now_eff = q.go ? xv : -1.0;
  last_now = __builtin_fmax(last_now, xv);
  return q;
}

// The two sampled candidates of a pool of n instances from the request's two
// words of that pool (the rule rt_sim_run_replicas documents): c1 and c2
// are distinct when n >= 2; with n == 1 both are instance 0.
__device__ __forceinline__ void sample_pair(uint32_t u, uint32_t v, uint32_t n, uint32_t& c1, uint32_t& c2) {
  c1 = __umulhi(u, n);
  const uint32_t x = __umulhi(v, n - 1);
  c2 = n > 1 ? x + (x >= c1 ? 1u : 0u) : c1;
}

// Which window positions the new head's record must fill after a release
// (p1: one request released, p2: two), with q requests left: bit 0 position
// 1 (only after two releases), bit 1 position 2.
__device__ __forceinline__ int32_t refill_mask(bool p1, bool p2, int32_t q) {
  return (p2 && q >= 2 ? 1 : 0) | (p1 && q >= 3 ? 2 : 0);
}

// Release without the refill: up to two completions per instance from the
// register window; records in x.lq which positions the new head's record
// must fill (refill_mask).
template <bool kTok, bool kKv>
__device__ __forceinline__ void release_pop(Slot& x, double now_eff) {
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
  x.lq = opaque(refill_mask(p1, p2, x.q));
}

// The refill load of a released slot: the new head's record where x.lq asks
// for one, else the wave's dummy record `dmy`.  `recr` is the lane's record
// plane at its replica's request 0; indices are relative to it (the
// dummy's too), so that an address is one shift-add.
template <bool kTok>
__device__ __forceinline__ void load_refill(Slot& x, const char* recr, int32_t R, int64_t dmy) {
  const int64_t g = sel_index(x.lq != 0, min(max(x.h.idx, 0), max(R - 1, 0)), dmy);
  load_pair<kTok>(x, rec_at<kTok>(recr, g));
}

// Release with its refill load issued unconditionally, merged later.
template <bool kTok, bool kKv>
__device__ __forceinline__ void release_slot(Slot& x, double now_eff, const char* recr, int32_t R, int64_t dmy) {
  release_pop<kTok, kKv>(x, now_eff);
  load_refill<kTok>(x, recr, R, dmy);
}

// The releases of every slot.  With one slot per lane they run on every
// step, branch-free (a launch of such classes has about one wave per SIMD,
// and a branch costs more than the work it skips).  With two or more, a slot
// whose head has finished on no lane of the wave is skipped, and the refill
// load is issued only where some lane needs one (those classes run several
// waves per SIMD and are bound by instruction issue: sweep 60.3 -> 55.3 ms
// with the matching merge below).
template <int M, bool kTok, bool kKv>
__device__ __forceinline__ void release_fast(Slot (&s)[M], double now_eff, const char* recr, int32_t R, int64_t dmy) {
  static_for<M>([&](auto mc) __attribute__((always_inline)) {
    constexpr int m = decltype(mc)::value;
    if constexpr (M >= 2) {
      if (__any(s[m].h.t <= now_eff)) {
        release_pop<kTok, kKv>(s[m], now_eff);
        if (__any(s[m].lq != 0)) load_refill<kTok>(s[m], recr, R, dmy);
      }
    } else {
      release_slot<kTok, kKv>(s[m], now_eff, recr, R, dmy);
    }
  });
}

template <int M>
__device__ __forceinline__ double head_min(const Slot (&s)[M]) {
  double h = s[0].h.t;
#pragma unroll
  for (int m = 1; m < M; ++m) h = __builtin_fmin(h, s[m].h.t);
  return h;
}

// The earliest third FIFO position of the lane's slots.  Before the fast
// releases, "some lane's third position has finished" is exactly "some head
// has finished after them" (release times do not decrease along a FIFO).
template <int M>
__device__ __forceinline__ double third_min(const Slot (&s)[M]) {
  double h = s[0].n2.t;
#pragma unroll
  for (int m = 1; m < M; ++m) h = __builtin_fmin(h, s[m].n2.t);
  return h;
}

// More completions than the window holds (rare; `more` says that some head
// of the wave has finished after the fast releases): wait for the loaded
// successors and release again, until no head of the wave has finished.
template <int M, bool kTok, bool kKv>
__device__ __forceinline__ void release_more(bool more, Slot (&s)[M], double now_eff, const char* recr, int32_t R,
                                             int64_t dmy) {
  if (__builtin_expect(more, 0)) {
    do {
#pragma unroll
      for (int m = 0; m < M; ++m) merge_pending(s[m]);
      release_fast<M, kTok, kKv>(s, now_eff, recr, R, dmy);
    } while (__any(head_min(s) <= now_eff));
  }
}

template <int S, int M, int kMode, int kWaves>
__global__ void __launch_bounds__(64 * kWaves) seg_kernel(SimArgs a) {
  constexpr bool kTok = mode_ledger(kMode);     // the ledger is priced
  constexpr bool kKv = kMode != kModeBase;      // occupancy is priced
  constexpr bool kSamp = mode_sampled(kMode);   // two candidates per pool
  constexpr int kSegs = 64 / S;               // replicas per wave
  const int lane = threadIdx.x & 63;
  const int sl = lane & (S - 1);
  const int segw = (int)(threadIdx.x >> 6) * kSegs + lane / S;  // segment within the block
  // a workgroup has 1 .. kWaves waves (chosen at launch)
  const int64_t item = (int64_t)blockIdx.x * ((int64_t)(blockDim.x >> 6) * kSegs) + segw;
  const bool live = item < a.n_work;
  const int rep = live ? a.work[item] : 0;
  const int64_t base = live ? a.offsets[rep] : 0;
  const int32_t R = live ? (int32_t)(a.offsets[rep + 1] - base) : 0;
  const int pid = (live && a.param_point) ? a.param_point[rep] : 0;
  const DevPoint& pt = a.points[pid];
  const int32_t P = pt.P, D = pt.D, ncls = pt.n_classes, policy = pt.policy;
  const bool thr = policy == kPolicyLengthThreshold;
  const int32_t half_d = (D + 1) / 2;  // first instance of the decode pool's upper part
  const int32_t len_thr = pt.len_thr;
  const int32_t LP = (P + M - 1) / M;  // lanes holding prefill instances
  const bool isp = sl < LP;
  const int32_t j0 = (isp ? sl : sl - LP) * M;  // this lane's first instance in its pool
  const int32_t npool = isp ? P : D;
  const float w_b = pt.w_b, w_s = pt.w_s, w_q = pt.w_q, rho = pt.rho;
  const float inv = isp ? pt.inv_cap_pre : pt.inv_cap_dec;
  const float tau = isp ? pt.tau_pre : pt.tau_dec;
  const float basec = isp ? pt.pre_base : 0.0f;  // proxy ledger: base per in-flight prefill
  const double pre_base_ns = (double)pt.pre_base_ns, pre_tok_ns = (double)pt.pre_tok_ns;
  const double dec_tok_ns = (double)pt.dec_tok_ns, xfer_tok_ns = (double)pt.xfer_tok_ns;
  char* const recb = isp ? a.rec[0] : a.rec[1];
  // The wave's dummy record: a negative request index whose records lie in
  // the dummy areas just before the planes.  Record loads and stores with
  // nothing to do use it, so that only an index is selected.  (Stores stay
  // unconditional: each lane of a store sends its own L2 request, but
  // switching exec off and on around the store costs more issue time here.)
  const uint32_t wave_id = ((blockIdx.x * blockDim.x + threadIdx.x) >> 6) & (kDummyRecords - 1);
  // the lane's plane at its replica's request 0, and the dummy's index
  // relative to it
  char* const recr = recb + rec_off<kTok>(base);
  const int64_t dmy = -1 - (int64_t)wave_id - base;

  // sigma per class of each segment's point, read a step ahead of its use
  __shared__ float sig[kWaves * kSegs * kMaxClasses];
  for (int k = sl; k < kMaxClasses; k += S) sig[segw * kMaxClasses + k] = pt.sigma[k];
  __syncthreads();

  Slot s[M];
  bool ok[M];  // the slot holds an instance of the lane's pool
#pragma unroll
  for (int m = 0; m < M; ++m) {
    init_slot(s[m]);
    ok[m] = live && j0 + m < npool;
  }

  // steps of this wave (wave-uniform, so the loop test is scalar)
  const int32_t Rmax = __builtin_amdgcn_readfirstlane(wave_max_nonneg(R));

  // The features of request t+1 are loaded during step t-1 (index clamped
  // into the replica; request 0 of the trace for a segment without a
  // replica), its class a step earlier still.
  const int64_t rd_base = R > 0 ? base : 0;
  const int32_t rd_last = R > 0 ? R - 1 : 0;
  double last_now = 0.0;  // latest accepted arrival (arrivals must not decrease)

  // Raw features of one request as loaded.
  struct Feat {
    int64_t arr;
    int32_t p, o, oh;
    uint32_t c;
    uint32_t u, v;  // the lane's pool's candidate words (sampled modes)
  };
  auto load_feat = [&](Feat& f, int32_t tt) {
    const int64_t g = rd_base + min(tt, rd_last);
    f.arr = a.arrival[g];
    f.p = a.plen[g];
    f.o = a.olen[g];
    f.oh = a.ohat[g];
    f.c = a.cls[g];
    if constexpr (kSamp) {
      const uint2 w = *reinterpret_cast<const uint2*>(a.samp + 4 * g + (isp ? 0 : 2));
      f.u = w.x;
      f.v = w.y;
    } else {
      f.u = f.v = 0;
    }
  };

  // Outcomes of the current block of S steps: lane k of a segment keeps
  // step (block start + k)'s, and the block is written with one coalesced
  // store per output array (a per-step store would send one write request
  // per lane of the wave, mostly to a dummy slot).
  int32_t b_ip = -1, b_id = -1;
  int64_t b_tt = -1, b_sp = -1;
  auto flush = [&](int32_t t0) {
    const int32_t tl = t0 + sl;
    if (tl < R) {
      const int64_t gi = base + tl;
      a.i_pre[gi] = b_ip;
      a.i_dec[gi] = b_id;
      a.ttft[gi] = b_tt;
      a.span[gi] = b_sp;
    }
  };

  int32_t rr = 0;     // round robin: t mod (size of this lane's pool)
  double tmax = 0.0;  // latest decode end this lane recorded (time-range check)
  uint32_t rej = 0;   // a rejected request was recorded by this lane
  Req cur;            // request t, checked, its releases done
  float sg;           // sigma of request t's class
  uint32_t cu = 0, cv = 0;  // request t's candidate words (sampled modes)

  // Step t: score, argmin, serve and record request t; store; then merge the
  // successors loaded during the releases for request t (a step ago), check
  // request t+1 (features `nx`, loaded a step ago) and do its releases, and
  // load the features of request t+2 into `ld`.
  auto step = [&](int32_t t, Feat& nx, Feat& ld) {
    const int32_t p = cur.p, o = cur.o, oh = cur.oh, po = cur.po, poh = cur.poh;
    const double now = cur.now;
    const bool go = cur.go;

    // 1. score this lane's instances
    const int32_t cnt = isp ? p : oh;           // priced tokens of the pool
    const float work = w_s * (float)cnt * tau;  // w_s * p * tau_pre, or w_s * o^ * tau_dec
    const double need = (double)(isp ? p : poh);
    const bool long_req = oh >= len_thr;  // length threshold: the upper part
    uint32_t bkey = 0xffffffffu;
    int32_t bm = 0;
    double bbusy = s[0].busy;
    uint32_t c1 = 0, c2 = 0;  // the pool's sampled candidates
    if constexpr (kSamp) sample_pair(cu, cv, (uint32_t)npool, c1, c2);
#pragma unroll
    for (int m = 0; m < M; ++m) {
      const Slot& x = s[m];
      uint32_t key;
      if constexpr (kMode == kModeBase) {
        // round robin; least loaded; or least loaded within the decode
        // part the request's predicted length picks (length threshold)
        const int32_t j = (j0 + m);
        key = policy == kPolicyRoundRobin ? (j == rr ? 0u : 1u) : (uint32_t)x.q;
        const bool part = D == 1 || ((j >= half_d) == long_req);
        key = (thr && !isp && !part) ? 0xffffffffu : key;
      } else {
        float bl;
        if constexpr (!kTok)
          bl = (float)__builtin_fmax(x.busy - now, 0.0) * 1e-9f;
        else
          bl = tau * (float)x.pend + basec * (float)x.q;
        const float press = (float)(x.kv + need) * inv;
        const float load = w_b * bl * sg;
        const float size = work * (1.0f + rho * press) * sg;
        const float cost = load + size + w_q * (float)x.q;
        key = cost != cost ? 0x7fc00000u : __float_as_uint(cost);
      }
      if constexpr (kSamp) {
        const uint32_t j = (uint32_t)(j0 + m);
        key = (j == c1 || j == c2) ? key : 0xffffffffu;
      }
      key = ok[m] ? key : 0xffffffffu;
      if (m == 0) {
        bkey = key;
      } else {
        const bool b = key < bkey;
        bkey = b ? key : bkey;
        bm = b ? m : bm;
        bbusy = b ? x.busy : bbusy;
      }
    }

    // 2. argmin of each pool over the segment, lowest index on equal keys
    uint32_t kp = isp ? bkey : 0xffffffffu, kd = isp ? 0xffffffffu : bkey;
    const uint32_t kp0 = kp, kd0 = kd;
    seg_min2<S>(kp, kd);
    const int32_t wp = seg_first<S>(kp0 == kp, lane);  // winning lanes
    const int32_t wd = seg_first<S>(kd0 == kd, lane);
    // the winning slots and the winners' busy-until, read by every lane of
    // the segment (so that every lane forms both ends): from 8 lanes up
    // through lane permutes, below that through DPP reductions
    int32_t mp = 0, md = 0;
    double busy_p = bbusy, busy_d = bbusy;
    if constexpr (S >= 8) {
      seg_pick2_f64<S>(busy_p, wp, busy_d, wd, lane);
      if constexpr (M > 1) {
        mp = seg_pick<S>(bm, wp, lane);
        md = seg_pick<S>(bm, wd, lane);
      }
    } else {
      if constexpr (M > 1) {
        mp = (int32_t)seg_or<S>(sl == wp ? (uint32_t)bm : 0u);
        md = (int32_t)seg_or<S>(sl == wd ? (uint32_t)bm : 0u);
      }
      seg_bcast2_f64<S>(busy_p, sl == wp, busy_d, sl == wd);
    }
    const int32_t ip = wp * M + mp;
    const int32_t id = (wd - LP) * M + md;

    // 3. serve: prefill, KV transfer, decode (exact integers in doubles)
    const double s_pre = __builtin_fma((double)p, pre_tok_ns, pre_base_ns);
    const double pf_end = __builtin_fmax(now, busy_p) + s_pre;
    const double kv_at = pf_end + (double)p * xfer_tok_ns;
    const double de = __builtin_fmax(kv_at, busy_d) + (double)(o - 1) * dec_tok_ns;
    const double end = isp ? pf_end : de;
    const int32_t fp = isp ? p : po;  // cache tokens held until release
    const int32_t tk = isp ? p : oh;  // ledger tokens
    const Elem z{end, t, fp, tk};
    const int32_t wl = go ? (isp ? wp : wd) : -1;
    const bool own_lane = opaque(wl) == sl;
    const int32_t wm = own_lane ? (isp ? mp : md) : -1;
    int32_t st1 = -1, st2 = -1;  // requests whose first / second successor is z (z beyond the window)
#pragma unroll
    for (int m = 0; m < M; ++m) {
      Slot& x = s[m];
      const bool own = (M == 1) ? own_lane : (opaque(wm) == m);
      const int32_t w = opaque(own ? x.q : -1);  // z's FIFO position
      x.h = sel(w == 0, z, x.h);
      x.n = sel(w == 1, z, x.n);
      x.n2 = sel(w == 2, z, x.n2);
      st1 = w >= 3 ? x.tail : st1;
      st2 = w >= 3 ? x.tail2 : st2;
      x.tail2 = own ? x.tail : x.tail2;
      x.tail = own ? t : x.tail;
      x.q = own ? x.q + 1 : x.q;
      if constexpr (kKv) x.kv = x.kv + (own ? (double)fp : 0.0);
      if constexpr (kTok) x.pend = x.pend + (own ? (double)tk : 0.0);
      x.busy = own ? end : x.busy;
    }

    // 4. the outcome, kept by lane t mod S of the segment until the block's
    // flush; the records of z, stored by every lane (the ones with nothing to
    // store address the dummies)
    {
      const int32_t o_ip = go ? ip : -1, o_id = go ? id : -1;
      const int64_t o_ttft = go ? f64_to_i64(pf_end - now) : -1;
      const int64_t o_span = go ? f64_to_i64(de - pf_end) : -1;
      const bool keep = opaque(t & (S - 1)) == sl;
      b_ip = keep ? o_ip : b_ip;
      b_id = keep ? o_id : b_id;
      b_tt = keep ? o_ttft : b_tt;
      b_sp = keep ? o_span : b_sp;
      tmax = __builtin_fmax(tmax, opaque(opaque(go ? wd : -1) == sl ? de : 0.0));
      rej |= opaque(go ? 0u : 1u) & opaque((R - t) >= 1 && sl == 0 ? 1u : 0u);
      const Entry ze{end, t, fp};
      const bool s1 = opaque(st1) >= 0, s2 = opaque(st2) >= 0;
      char* const r1 = rec_at<kTok>(recr, sel_index(s1, st1, dmy));
      char* const r2 = rec_at<kTok>(recr, sel_index(s2, st2, dmy));
      *reinterpret_cast<Entry*>(r1) = ze;
      *reinterpret_cast<Entry*>(r2 + 16) = ze;
      if constexpr (kTok) {
        *reinterpret_cast<int32_t*>(r1 + kRecTok) = tk;
        *reinterpret_cast<int32_t*>(r2 + kRecTok + 4) = tk;
      }
    }
    if constexpr (kMode == kModeBase) rr = (rr + 1 == npool) ? 0 : rr + 1;

    // 5. the successors loaded during request t's releases (the step's one
    // wait: those loads and the features of request t+1 were issued a step
    // ago), kept apart from the surrounding code by the scheduling barriers
    // (with two or more slots per lane, only slots where some lane loaded)
    __builtin_amdgcn_sched_barrier(0);
    static_for<M>([&](auto mc) __attribute__((always_inline)) {
      constexpr int m = decltype(mc)::value;
      if constexpr (M >= 2) {
        if (__any(s[m].lq != 0)) {
          merge_pending(s[m]);
          pin_window<kTok>(s[m]);
        }
      } else {
        merge_pending(s[m]);
        pin_window<kTok>(s[m]);
      }
    });
    if constexpr (kSamp)
      asm volatile("" : "+v"(nx.arr), "+v"(nx.p), "+v"(nx.o), "+v"(nx.oh), "+v"(nx.c), "+v"(nx.u), "+v"(nx.v));
    else
      asm volatile("" : "+v"(nx.arr), "+v"(nx.p), "+v"(nx.o), "+v"(nx.oh), "+v"(nx.c));
    __builtin_amdgcn_sched_barrier(0);

    // 6. request t+1: check, sigma, releases (the test for a slow path is
    // made ahead of the fast releases, so that the scalar branch does not
    // wait for its vector compare); load request t+2
    cur = admit_check(R - (t + 1), ncls, nx.arr, nx.p, nx.o, nx.oh, nx.c, last_now);
    sg = sig[segw * kMaxClasses + (nx.c & (kMaxClasses - 1))];
    cu = nx.u;
    cv = nx.v;
    const bool more = __any(third_min(s) <= cur.now_eff);
    release_fast<M, kTok, kKv>(s, cur.now_eff, recr, R, dmy);
    release_more<M, kTok, kKv>(more, s, cur.now_eff, recr, R, dmy);
    load_feat(ld, t + 2);
  };

  // request 0 (nothing to release yet); requests 1 and 2 in flight
  Feat fa, fb;
  load_feat(fa, 0);
  __builtin_amdgcn_s_waitcnt(0);
  cur = admit_check(R, ncls, fa.arr, fa.p, fa.o, fa.oh, fa.c, last_now);
  sg = sig[segw * kMaxClasses + (fa.c & (kMaxClasses - 1))];
  cu = fa.u;
  cv = fa.v;
  load_feat(fa, 1);
  // enter the loop with nothing in flight, so that the loop header needs no
  // wait
  __builtin_amdgcn_s_waitcnt(0);

  // two steps per iteration, so that the features loaded in one step are
  // read in the next from the same registers
  // (the count of steps left is a scalar, so the loop tests read no vector
  // register)
  // (S is even, so a block ends on the second step of an iteration)
  int32_t t = 0;
  for (int32_t left = Rmax; left > 0; left -= 2, t += 2) {
    step(t, fa, fb);
    if (left > 1) {
      step(t + 1, fb, fa);
      if (((t + 1) & (S - 1)) == S - 1) flush((t + 1) & ~(S - 1));
    }
  }
  if (Rmax & (S - 1)) flush(Rmax & ~(S - 1));
  const uint32_t flag = (tmax >= kTimeLimit ? kFlagTimeRange : 0u) | (rej ? kFlagRejected : 0u);
  if (flag) atomicOr(a.flag, flag);
}

// Up to four waves per workgroup (one per SIMD of a compute unit).  A launch
// with few waves uses smaller workgroups, so that they spread over more
// compute units (each unit's memory pipeline is shared by its waves).
constexpr int kSegWaves = 4;
constexpr int kComputeUnits = 256;

template <int S, int M, int kMode>
hipError_t launch_seg(const SimArgs& a, hipStream_t stream) {
  if (a.n_work <= 0) return hipSuccess;
  constexpr int64_t kSegs = 64 / S;
  const int64_t waves = (a.n_work + kSegs - 1) / kSegs;
  const int64_t wpb = std::min<int64_t>(kSegWaves, std::max<int64_t>(1, (waves + kComputeUnits - 1) / kComputeUnits));
  const int64_t blocks = (waves + wpb - 1) / wpb;
  hipLaunchKernelGGL((seg_kernel<S, M, kMode, kSegWaves>), dim3((unsigned)blocks), dim3(64 * (unsigned)wpb), 0, stream,
                     a);
  return hipGetLastError();
}

// The segment widths and lane depths compiled for every mode.
#define RT_SEG_FOR_EACH(X)                                                    \
  X(2, 1) X(4, 1) X(8, 1) X(16, 1) X(32, 1) X(64, 1) X(2, 2) X(4, 2) X(8, 2)  \
  X(16, 2) X(32, 2) X(64, 2) X(2, 3) X(4, 3) X(8, 3) X(16, 3) X(32, 3)        \
  X(64, 3) X(2, 4) X(4, 4) X(8, 4) X(16, 4) X(32, 4) X(64, 4)

// Launch the (S, M) kernel of one mode (defined in one source file per mode).
template <int kMode>
hipError_t launch_mode(int S, int M, const SimArgs& a, hipStream_t stream);


}  // namespace seg
}  // namespace rt
