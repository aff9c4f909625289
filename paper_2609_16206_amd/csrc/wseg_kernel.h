// Replica-batched simulation of the learned prefill/decode router for pools
// wider than one wave, on gfx950.
//
// Method and per-instance machinery as in seg_kernel.h (Algorithm 1 per
// admission on the serial-service simulator of Section III-D / Section VI;
// Section III-A costs; the register FIFO window with two-successor records;
// the rotated step).  Differences for wide pools:
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
// of every wave publishes its two winners (and the prefill winner's
// busy-until) in LDS; after one barrier every wave combines them by (cost,
// index), so equal costs keep the lowest index.  The LDS slots are
// double-buffered by step parity, so one barrier per step suffices.
//
// Sparse work.  Per step only the two winning instances are appended to and
// only instances whose head has finished are released, so both run under
// uniform branches: the append in the winner's wave and only for the
// winner's slot, the release only for slots where some lane's head has
// finished.
#pragma once

#include "seg_kernel.h"

namespace rt {
namespace seg {

// Lanes per wave holding a pool of n instances, dealt round robin to W waves
// at M per lane.
__host__ __device__ inline int wide_pool_lanes(int n, int M, int W) { return ((n + W - 1) / W + M - 1) / M; }

template <int W, int M, int kMode>
__global__ void __launch_bounds__(64 * W) wseg_kernel(SimArgs a) {
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
  char* const recb = isp ? a.rec[0] : a.rec[1];
  const uint32_t wave_id = (blockIdx.x * W + wave) & (kDummyRecords - 1);
  // the lane's plane at its replica's request 0; the wave's dummy record,
  // indexed relative to it
  char* const recr = recb + rec_off<kTok>(base);
  const int64_t dmy = -1 - (int64_t)wave_id - base;

  struct Part {
    uint32_t kp, kd;  // the wave's best prefill / decode key
    int32_t ip, id;   // their instance indices
    double bp;        // busy-until of the wave's best prefill instance
  };
  __shared__ float sig[kMaxClasses];
  __shared__ Part part[2][W];
  if (threadIdx.x < kMaxClasses) sig[threadIdx.x] = pt.sigma[threadIdx.x];
  __syncthreads();

  Slot s[M];
  bool ok[M];  // the slot holds an instance of the lane's pool
#pragma unroll
  for (int m = 0; m < M; ++m) {
    init_slot(s[m]);
    ok[m] = inpool && wave + W * (lrel * M + m) < npool;
  }

  // request 0 (nothing to release yet); the features of request 1 in flight
  double last_now = 0.0;
  Req cur = admit_check(R, ncls, a.arrival[base], a.plen[base], a.olen[base], a.ohat[base], a.cls[base], last_now);
  float sg = sig[a.cls[base] & (kMaxClasses - 1)];
  // the candidate words of the lane's pool (sampled modes)
  auto load_words = [&](int64_t g, uint32_t& u, uint32_t& v) {
    if constexpr (kSamp) {
      const uint2 w = *reinterpret_cast<const uint2*>(a.samp + 4 * g + (isp ? 0 : 2));
      u = w.x;
      v = w.y;
    } else {
      u = v = 0;
    }
  };
  uint32_t cu, cv;
  load_words(base, cu, cv);
  const int32_t last = R - 1;
  int64_t nx_arr;
  int32_t nx_p, nx_o, nx_oh;
  uint32_t nx_c, nx_u, nx_v;
  {
    const int64_t g = base + min(1, last);
    nx_arr = a.arrival[g];
    nx_p = a.plen[g];
    nx_o = a.olen[g];
    nx_oh = a.ohat[g];
    nx_c = a.cls[g];
    load_words(g, nx_u, nx_v);
  }
  int32_t rr = 0;     // round robin: t mod (size of this lane's pool)
  double tmax = 0.0;  // latest decode end this lane recorded (time-range check)
  uint32_t rej = 0;   // a rejected request was recorded by this lane

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

    // 2. per-wave argmin of both pools, then across waves through LDS
    {
      uint32_t kp = isp ? bkey : 0xffffffffu, kd = isp ? 0xffffffffu : bkey;
      const uint32_t kp0 = kp, kd0 = kd;
      seg_min2<64>(kp, kd, lane);
      const int32_t wp = seg_first<64>(kp0 == kp, lane) & 63;  // the wave's winning lanes
      const int32_t wd = seg_first<64>(kd0 == kd, lane) & 63;
      const int32_t mpw = __builtin_amdgcn_readlane(bm, wp);
      const int32_t mdw = __builtin_amdgcn_readlane(bm, wd);
      const double bpw = __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(bbusy), wp),
                                          __builtin_amdgcn_readlane(__double2loint(bbusy), wp));
      if (lane == 0)
        part[t & 1][wave] = Part{kp, kd, wave + W * (wp * M + mpw), wave + W * ((wd - LPW) * M + mdw), bpw};
    }
    __syncthreads();
    uint32_t kp = part[t & 1][0].kp, kd = part[t & 1][0].kd;
    int32_t ip = part[t & 1][0].ip, id = part[t & 1][0].id;
    double busy_ip = part[t & 1][0].bp;
#pragma unroll
    for (int w = 1; w < W; ++w) {
      const Part x = part[t & 1][w];
      const bool bp = x.kp < kp || (x.kp == kp && x.ip < ip);
      const bool bd = x.kd < kd || (x.kd == kd && x.id < id);
      kp = bp ? x.kp : kp;
      ip = bp ? x.ip : ip;
      busy_ip = bp ? x.bp : busy_ip;
      kd = bd ? x.kd : kd;
      id = bd ? x.id : id;
    }
    ip = __builtin_amdgcn_readfirstlane(ip);
    id = __builtin_amdgcn_readfirstlane(id);

    // 3. serve (uniform up to the decode winner's own busy-until); the
    // winners' waves, lanes and slots
    const double s_pre = __builtin_fma((double)p, pre_tok_ns, pre_base_ns);
    const double pf_end = __builtin_fmax(now, busy_ip) + s_pre;
    const double kv_at = pf_end + (double)p * xfer_tok_ns;
    const int32_t wpo = ip % W, wdo = id % W;            // waves
    const int32_t qp = ip / W, qd = id / W;              // positions within the wave
    const int32_t lpo = qp / M, ldo = LPW + qd / M;      // lanes
    const int32_t mp = qp - (qp / M) * M, md = qd - (qd / M) * M;  // slots

    // 4. the successors loaded during request t's releases (slots where any
    // lane loaded some; every slot's test is made before the first branch,
    // so that the scalar branches wait for one vector compare, not one each)
    {
      uint64_t any_lq[M];
#pragma unroll
      for (int m = 0; m < M; ++m) any_lq[m] = __ballot(s[m].lq >= 2);
#pragma unroll
      for (int m = 0; m < M; ++m)
        if (any_lq[m]) merge_pending(s[m]);
    }

    // 5. request t+1: check and sigma (its features are waited for here,
    // ahead of the stores below, which the compiler's waits do not count)
    const Req nxt = [&] {
      // (uniform over the workgroup; reading the first lane tells the compiler)
      const int64_t u_arr = ((int64_t)__builtin_amdgcn_readfirstlane((int32_t)(nx_arr >> 32)) << 32) |
                            (uint32_t)__builtin_amdgcn_readfirstlane((int32_t)nx_arr);
      const uint32_t u_c = (uint32_t)__builtin_amdgcn_readfirstlane((int32_t)nx_c);
      sg = sig[u_c & (kMaxClasses - 1)];
      return admit_check(R - (t + 1), ncls, u_arr, __builtin_amdgcn_readfirstlane(nx_p),
                         __builtin_amdgcn_readfirstlane(nx_o), __builtin_amdgcn_readfirstlane(nx_oh), u_c, last_now);
    }();

    // 6. append the request to the winning slot of each pool (uniform
    // branches: the winner's wave, the winner's slot) and record the outcome;
    // only the lanes with something to store store it.  Addresses stay inside
    // the plane on every lane: a tail is >= -1, and index -1 is the record
    // before the replica's first (a dummy record for the trace's first).
    if (go && wave == wpo) {
      const Elem z{pf_end, t, p, p};
      const u32x4 zv = {(uint32_t)__double2loint(pf_end), (uint32_t)__double2hiint(pf_end), (uint32_t)t, (uint32_t)p};
#pragma unroll
      for (int m = 0; m < M; ++m)
        if (m == mp) {
          Slot& x = s[m];
          const bool own = lane == lpo;
          const int32_t w = opaque(own ? x.q : -1);  // z's FIFO position
          x.h = sel(w == 0, z, x.h);
          x.n = sel(w == 1, z, x.n);
          x.n2 = sel(w == 2, z, x.n2);
          const uint32_t s1 = opaque(w) >= 1 ? 1u : 0u, s2 = opaque(w) >= 2 ? 1u : 0u;
          const int64_t g1 = x.tail, g2 = x.tail2;
          x.tail2 = own ? x.tail : x.tail2;
          x.tail = own ? t : x.tail;
          x.q = own ? x.q + 1 : x.q;
          if constexpr (kKv) x.kv = x.kv + (own ? (double)p : 0.0);
          if constexpr (kTok) x.pend = x.pend + (own ? (double)p : 0.0);
          x.busy = own ? pf_end : x.busy;
          if constexpr (kTok) {
            store_x4_b32_if(s1, recr + rec_off<kTok>(g1), zv, recr + rec_off<kTok>(g1) + kRecTok, (uint32_t)p);
            store_x4_b32_if(s2, recr + rec_off<kTok>(g2) + 16, zv, recr + rec_off<kTok>(g2) + kRecTok + 4, (uint32_t)p);
          } else {
            store_x4_if(s1, recr + rec_off<kTok>(g1), zv);
            store_x4_if(s2, recr + rec_off<kTok>(g2) + 16, zv);
          }
        }
    }
    if (go && wave == wdo) {
#pragma unroll
      for (int m = 0; m < M; ++m)
        if (m == md) {
          Slot& x = s[m];
          const bool own = lane == ldo;
          const double de = __builtin_fmax(kv_at, x.busy) + (double)(o - 1) * dec_tok_ns;
          const Elem z{de, t, po, oh};
          const int32_t w = opaque(own ? x.q : -1);
          x.h = sel(w == 0, z, x.h);
          x.n = sel(w == 1, z, x.n);
          x.n2 = sel(w == 2, z, x.n2);
          const uint32_t s1 = opaque(w) >= 1 ? 1u : 0u, s2 = opaque(w) >= 2 ? 1u : 0u;
          const int64_t g1 = x.tail, g2 = x.tail2;
          x.tail2 = own ? x.tail : x.tail2;
          x.tail = own ? t : x.tail;
          x.q = own ? x.q + 1 : x.q;
          if constexpr (kKv) x.kv = x.kv + (own ? (double)po : 0.0);
          if constexpr (kTok) x.pend = x.pend + (own ? (double)oh : 0.0);
          x.busy = own ? de : x.busy;
          const u32x4 zv = {(uint32_t)__double2loint(de), (uint32_t)__double2hiint(de), (uint32_t)t, (uint32_t)po};
          if constexpr (kTok) {
            store_x4_b32_if(s1, recr + rec_off<kTok>(g1), zv, recr + rec_off<kTok>(g1) + kRecTok, (uint32_t)oh);
            store_x4_b32_if(s2, recr + rec_off<kTok>(g2) + 16, zv, recr + rec_off<kTok>(g2) + kRecTok + 4, (uint32_t)oh);
          } else {
            store_x4_if(s1, recr + rec_off<kTok>(g1), zv);
            store_x4_if(s2, recr + rec_off<kTok>(g2) + 16, zv);
          }
          // the outcome, by the decode winner
          tmax = __builtin_fmax(tmax, own ? de : 0.0);
          const int64_t go_i = base + t;
          store_out_if(own ? 1u : 0u, a.i_pre + go_i, ip, a.i_dec + go_i, id, a.ttft + go_i, f64_to_i64(pf_end - now),
                       a.span + go_i, f64_to_i64(de - pf_end));
        }
    }
    if (!go && wave == 0) {
      // a rejected request: -1 outputs, by lane 0
      rej |= lane == 0 ? 1u : 0u;
      const int64_t go_i = base + t;
      store_out_if(lane == 0 ? 1u : 0u, a.i_pre + go_i, -1, a.i_dec + go_i, -1, a.ttft + go_i, (int64_t)-1,
                   a.span + go_i, (int64_t)-1);
    }
    if constexpr (kMode == kModeBase) rr = (rr + 1 == npool) ? 0 : rr + 1;

    // 7. the releases for request t+1 (slot by slot, where some lane's head
    // has finished); load request t+2
    cur = nxt;
    cu = nx_u;
    cv = nx_v;
    {
      // (slots release independently, so all tests come first)
      uint64_t any_done[M];
#pragma unroll
      for (int m = 0; m < M; ++m) any_done[m] = __ballot(s[m].h.t <= cur.now_eff);
#pragma unroll
      for (int m = 0; m < M; ++m)
        if (any_done[m]) release_slot<kTok, kKv>(s[m], cur.now_eff, recr, R, dmy);
    }
    release_more<M, kTok, kKv>(__any(head_min(s) <= cur.now_eff), s, cur.now_eff, recr, R, dmy);
    {
      const int64_t g = base + min(t + 2, last);
      nx_arr = a.arrival[g];
      nx_p = a.plen[g];
      nx_o = a.olen[g];
      nx_oh = a.ohat[g];
      nx_c = a.cls[g];
      load_words(g, nx_u, nx_v);
    }
  }
  const uint32_t flag = (tmax >= kTimeLimit ? kFlagTimeRange : 0u) | (rej ? kFlagRejected : 0u);
  if (flag) atomicOr(a.flag, flag);
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
