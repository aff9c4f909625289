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
// Argmin.  Each wave reduces both pools over its 64 lanes (DPP + readlane;
// within a wave the lowest lane and slot hold the lowest index), then lane 0
// of every wave folds its two winners into an LDS minimum of the packed key
// (cost key << 32 | instance index), so equal costs keep the lowest index,
// and writes their busy-until next to it.  After one barrier per step every
// wave reads both minima and the two winners' busy-until, so all waves form
// the same prefill and decode ends.  The LDS cells rotate over three step
// slots: slot t % 3 is filled at step t, read after its barrier, and reset by
// wave 0 after the barrier of step t + 1 (every wave has read it by then, and
// none writes it again before the barrier of step t + 2).
//
// Per-step work is kept to one vector compare and one uniform branch per
// phase where it is usually idle: the merge of refill loads runs only for
// slots that issued one (a scalar mask), the releases only when some head of
// the wave has finished, the slow path only when a head is still finished
// after them, and the appends, whose FIFO position is the winner's queue
// length read as a scalar, touch scratch only beyond the register window.
//
// Requests and outcomes move in blocks of 64: lane k of every wave holds the
// features of request (block start + k), loaded one block ahead with one
// coalesced load per field, and a step reads its request with readlane;
// wave 0's lane k keeps the outcome of step (block start + k) and the block
// is written with one coalesced store per output array.
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

__device__ __forceinline__ int64_t rl_i64(int64_t v, int lane) {
  return (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int32_t)(v >> 32), lane) << 32) |
                   (uint32_t)__builtin_amdgcn_readlane((int32_t)v, lane));
}

template <int W, int M, int kMode>
__global__ void __launch_bounds__(64 * W) wseg_kernel(SimArgs a) {
  static_assert(W == 2 || W == 4 || W == 8, "workgroups of 2, 4 or 8 waves");
  constexpr int kLogW = W == 2 ? 1 : (W == 4 ? 2 : 3);
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
  const float w_b = pt.w_b, w_s = pt.w_s, w_q = pt.w_q, rho = pt.rho;
  const float inv = isp ? pt.inv_cap_pre : pt.inv_cap_dec;
  const float tau = isp ? pt.tau_pre : pt.tau_dec;
  const float basec = isp ? pt.pre_base : 0.0f;  // proxy ledger: base per in-flight prefill
  const double pre_base_ns = (double)pt.pre_base_ns, pre_tok_ns = (double)pt.pre_tok_ns;
  const double dec_tok_ns = (double)pt.dec_tok_ns, xfer_tok_ns = (double)pt.xfer_tok_ns;
  const float sigv = pt.sigma[lane & (kMaxClasses - 1)];  // lane k: sigma of class k mod 8
  char* const recb = isp ? a.rec[0] : a.rec[1];
  const uint32_t wave_id = (blockIdx.x * W + wave) & (kDummyRecords - 1);
  // the lane's plane at its replica's request 0; the wave's dummy record,
  // indexed relative to it
  char* const recr = recb + rec_off<kTok>(base);
  const int64_t dmy = -1 - (int64_t)wave_id - base;

  __shared__ unsigned long long best[3][2];  // per step slot: packed minimum of each pool
  __shared__ double wbusy[3][W][2];          // per step slot: each wave's winners' busy-until
  if (threadIdx.x < 6) best[threadIdx.x >> 1][threadIdx.x & 1] = ~0ull;
  __syncthreads();

  Slot s[M];
  bool ok[M];  // the slot holds an instance of the lane's pool
#pragma unroll
  for (int m = 0; m < M; ++m) {
    init_slot(s[m]);
    ok[m] = inpool && wave + W * (lrel * M + m) < npool;
  }

  // Features of a block of 64 requests, lane k holding request (block + k)
  // (clamped into the replica).
  struct Block {
    int64_t arr;
    int32_t p, o, oh;
    uint32_t c;
    uint32_t w[4];  // candidate words (sampled modes)
  };
  auto load_block = [&](Block& f, int32_t blk) __attribute__((always_inline)) {
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
  Block fb0, fb1;  // the current block and the next
  load_block(fb0, 0);
  load_block(fb1, 64);

  double last_now = 0.0;  // latest accepted arrival (arrivals must not decrease)
  float sg;               // sigma of the current request's class
  uint32_t cu = 0, cv = 0;  // the lane's pool's candidate words of the current request
  // Request k of the current block, checked against the replica (its
  // features are uniform: read from lane k).
  auto take = [&](int k, int32_t t) __attribute__((always_inline)) {
    const uint32_t c = (uint32_t)__builtin_amdgcn_readlane((int32_t)fb0.c, k);
    sg = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int32_t, sigv), (int)(c & 7u)));
    if constexpr (kSamp) {
      const uint32_t w0 = (uint32_t)__builtin_amdgcn_readlane((int32_t)fb0.w[0], k);
      const uint32_t w1 = (uint32_t)__builtin_amdgcn_readlane((int32_t)fb0.w[1], k);
      const uint32_t w2 = (uint32_t)__builtin_amdgcn_readlane((int32_t)fb0.w[2], k);
      const uint32_t w3 = (uint32_t)__builtin_amdgcn_readlane((int32_t)fb0.w[3], k);
      cu = isp ? w0 : w2;
      cv = isp ? w1 : w3;
    }
    return admit_check(R - t, ncls, rl_i64(fb0.arr, k), __builtin_amdgcn_readlane(fb0.p, k),
                       __builtin_amdgcn_readlane(fb0.o, k), __builtin_amdgcn_readlane(fb0.oh, k), c, last_now);
  };
  Req cur = take(0, 0);

  // outcomes of the current block (wave 0, lane k: step block start + k)
  int32_t b_ip = -1, b_id = -1;
  int64_t b_tt = -1, b_sp = -1;
  int32_t rr = 0;      // round robin: t mod (size of this lane's pool)
  double tmax = 0.0;   // latest decode end (time-range check)
  bool rej = false;    // a request was rejected
  uint32_t pend = 0;   // slots whose refill load is in flight (bit m)
  int sl3 = 0;         // step slot t % 3 of the LDS cells

  for (int32_t t = 0; t < R; ++t) {
    const int32_t p = cur.p, o = cur.o, oh = cur.oh, po = cur.po, poh = cur.poh;
    const double now = cur.now;
    const bool go = cur.go;

    // 1. score this lane's instances
    const int32_t cnt = isp ? p : oh;
    const float work = w_s * (float)cnt * tau;
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
        const int32_t j = (wave + W * (lrel * M + m));
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
        bbusy = b ? x.busy : bbusy;
      }
    }

    // 2. per-wave argmin of both pools; lane 0 folds the wave's winners into
    // the LDS minima and publishes their busy-until
    {
      uint32_t kp = isp ? bkey : 0xffffffffu, kd = isp ? 0xffffffffu : bkey;
      const uint32_t kp0 = kp, kd0 = kd;
      seg_min2<64>(kp, kd, lane);
      const int32_t wp = seg_first<64>(kp0 == kp, lane) & 63;  // the wave's winning lanes
      const int32_t wd = seg_first<64>(kd0 == kd, lane) & 63;
      const int32_t mpw = __builtin_amdgcn_readlane(bm, wp);
      const int32_t mdw = __builtin_amdgcn_readlane(bm, wd);
      const double bpw = rl_f64(bbusy, wp), bdw = rl_f64(bbusy, wd);
      const uint32_t ipw = (uint32_t)(wave + W * (wp * M + mpw));
      const uint32_t idw = (uint32_t)(wave + W * ((wd - LPW) * M + mdw));
      if (lane == 0) {
        atomicMin(&best[sl3][0], ((unsigned long long)kp << 32) | ipw);
        atomicMin(&best[sl3][1], ((unsigned long long)kd << 32) | idw);
        wbusy[sl3][wave][0] = bpw;
        wbusy[sl3][wave][1] = bdw;
      }
    }
    __syncthreads();
    const int32_t ip = __builtin_amdgcn_readfirstlane((int32_t)(uint32_t)best[sl3][0]);
    const int32_t id = __builtin_amdgcn_readfirstlane((int32_t)(uint32_t)best[sl3][1]);
    double busy_ip = wbusy[sl3][0][0], busy_id = wbusy[sl3][0][1];
#pragma unroll
    for (int w = 1; w < W; ++w) {
      busy_ip = (ip & (W - 1)) == w ? wbusy[sl3][w][0] : busy_ip;
      busy_id = (id & (W - 1)) == w ? wbusy[sl3][w][1] : busy_id;
    }
    // the cells of step t - 1 are free again (every wave has read them)
    const int sl_prev = sl3 == 0 ? 2 : sl3 - 1;
    if (wave == 0 && lane < 2) best[sl_prev][lane] = ~0ull;

    // 3. serve (uniform): prefill, KV transfer, decode (exact integers in
    // doubles)
    const double s_pre = __builtin_fma((double)p, pre_tok_ns, pre_base_ns);
    const double pf_end = __builtin_fmax(now, busy_ip) + s_pre;
    const double kv_at = pf_end + (double)p * xfer_tok_ns;
    const double de = __builtin_fmax(kv_at, busy_id) + (double)(o - 1) * dec_tok_ns;

    // 4. refill loads of request t's releases, where any were issued
    if (pend) {
      static_for<M>([&](auto mc) __attribute__((always_inline)) {
        if (pend & (1u << decltype(mc)::value)) merge_pending(s[decltype(mc)::value]);
      });
      pend = 0;
    }

    // 5. append the request to the winning slot of each pool (uniform
    // branches: the winner's wave and slot, then its FIFO position)
    if (go) {
      auto append = [&](int32_t win, int32_t lane_off, double end, int32_t fp, int32_t tk) __attribute__((always_inline)) {
        const int32_t q = win >> kLogW;       // position within the wave
        const int32_t lw = lane_off + q / M;  // lane
        const int32_t mw = q - (q / M) * M;  // slot
        const bool own = lane == lw;
        const Elem z{end, t, fp, tk};
        static_for<M>([&](auto mc) __attribute__((always_inline)) {
          constexpr int m = decltype(mc)::value;
          if (m != mw) return;
          Slot& x = s[m];
          const int32_t w = __builtin_amdgcn_readlane(x.q, lw);  // z's FIFO position
          if (w == 0) {
            x.h = sel(own, z, x.h);
          } else if (w == 1) {
            x.n = sel(own, z, x.n);
          } else if (w == 2) {
            x.n2 = sel(own, z, x.n2);
          } else if (own) {
            // beyond the window: z is the first successor of the tail and
            // the second of the request before it
            char* const r1 = rec_at<kTok>(recr, x.tail);
            char* const r2 = rec_at<kTok>(recr, x.tail2);
            *reinterpret_cast<Entry*>(r1) = Entry{end, t, fp};
            *reinterpret_cast<Entry*>(r2 + 16) = Entry{end, t, fp};
            if constexpr (kTok) {
              *reinterpret_cast<int32_t*>(r1 + kRecTok) = tk;
              *reinterpret_cast<int32_t*>(r2 + kRecTok + 4) = tk;
            }
          }
          const int32_t tl_old = x.tail;
          x.tail2 = own ? tl_old : x.tail2;
          x.tail = own ? t : tl_old;
          x.q = own ? x.q + 1 : x.q;
          if constexpr (kKv) x.kv = x.kv + (own ? (double)fp : 0.0);
          if constexpr (kTok) x.pend = x.pend + (own ? (double)tk : 0.0);
          x.busy = own ? end : x.busy;
        });
      };
      if (wave == (ip & (W - 1))) append(ip, 0, pf_end, p, p);
      if (wave == (id & (W - 1))) append(id, LPW, de, po, oh);
    }

    // 6. the outcome, kept by wave 0's lane t mod 64 until its block is
    // written
    if (wave == 0) {
      const bool keep = lane == (t & 63);
      b_ip = keep ? (go ? ip : -1) : b_ip;
      b_id = keep ? (go ? id : -1) : b_id;
      b_tt = keep ? (go ? f64_to_i64(pf_end - now) : -1) : b_tt;
      b_sp = keep ? (go ? f64_to_i64(de - pf_end) : -1) : b_sp;
      tmax = go ? __builtin_fmax(tmax, de) : tmax;
      rej = rej || !go;
      if ((t & 63) == 63 || t == R - 1) {
        const int32_t tl = (t & ~63) + lane;
        if (tl <= t) {
          const int64_t gi = base + tl;
          a.i_pre[gi] = b_ip;
          a.i_dec[gi] = b_id;
          a.ttft[gi] = b_tt;
          a.span[gi] = b_sp;
        }
      }
    }
    if constexpr (kMode == kModeBase) rr = (rr + 1 == npool) ? 0 : rr + 1;
    sl3 = sl3 == 2 ? 0 : sl3 + 1;
    if (t + 1 == R) break;

    // 7. request t+1 (the next block moves in at a block boundary, and the
    // block after it is loaded), then its releases
    if (((t + 1) & 63) == 0) {
      fb0 = fb1;
      load_block(fb1, t + 1 + 64);
    }
    cur = take((t + 1) & 63, t + 1);
    {
      bool done = false;
#pragma unroll
      for (int m = 0; m < M; ++m) done = done || s[m].h.t <= cur.now_eff;
      if (__any(done)) {
        static_for<M>([&](auto mc) __attribute__((always_inline)) {
          constexpr int m = decltype(mc)::value;
          if (__any(s[m].h.t <= cur.now_eff)) {
            release_pop<kTok, kKv>(s[m], cur.now_eff);
            if (__any(s[m].lq != 0)) {
              load_refill<kTok>(s[m], recr, R, dmy);
              pend |= 1u << m;
            }
          }
        });
        // a head still finished: more releases than the window holds
        if (__builtin_expect(__any(head_min(s) <= cur.now_eff), 0)) {
          release_more<M, kTok, kKv>(true, s, cur.now_eff, recr, R, dmy);
          pend = (1u << M) - 1u;
        }
      }
    }
  }
  if (wave == 0) {
    const uint32_t flag = (tmax >= kTimeLimit ? kFlagTimeRange : 0u) | (rej ? kFlagRejected : 0u);
    if (flag && lane == 0) atomicOr(a.flag, flag);
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
#define RT_WSEG_FOR_EACH(X) X(2, 2) X(4, 2) X(2, 3) X(4, 3) X(4, 5) X(8, 2) X(8, 3) X(8, 5)

template <int kMode>
hipError_t launch_wide_mode(int W, int M, const SimArgs& a, hipStream_t stream);

}  // namespace seg
}  // namespace rt
