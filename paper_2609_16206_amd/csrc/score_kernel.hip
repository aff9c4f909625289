// Standalone batched scorer (Section III-A cost equation + per-pool argmin)
// and the per-replica goodput reduction (Section IV-B SLO targets, Table II
// goodput), for gfx950.
//
// Shared snapshot (inst_stride 0): the instance terms that do not depend on
// the request, w_b * backlog and w_q * queue, are formed once per block into
// LDS (the same float32 operations the equation performs first), then each
// thread scores kReq requests against every instance, reading each LDS entry
// once for all of its requests.  VALU-bound.
//
// Per-request snapshot (inst_stride >= n_inst): rows of at most 64 instances
// laid out for 16-byte loads take 16 lanes per request, four instances per
// lane; any other shape takes a segment of S lanes per request that walks the
// request's row with unit stride across lanes (coalesced), keeps a
// lane-local best, and reduces (key, index) over the segment.  HBM-bound.
#include "rt_internal.h"

namespace rt {
namespace {

constexpr int kReq = 2;       // requests per thread (shared snapshot; measured: 1, 2, 4, 8 give 30.0, 29.5, 31.4, 37.1 us on 2^20 x 64)
constexpr int kBlock = 256;

struct SnapEntry {
  float lb;    // w_b * backlog
  float qq;    // w_q * (float)queue
  int32_t kv;  // occupancy
  int32_t pad;
};

__device__ __forceinline__ bool req_ok(int32_t pool, int32_t p, int32_t oh, uint32_t c) {
  if (p < 1 || c >= (uint32_t)kMaxClasses) return false;
  if (pool == 1 && (oh < 1 || (int64_t)p + oh > INT32_MAX)) return false;
  return true;
}

// One thread's kReq requests against every snapshot entry.  kNonNeg: every
// occupancy is >= 0, so occupancy + need < 2^32 and the sum converts exactly
// through the unsigned 32-bit path (same value and rounding as int64).
template <bool kNonNeg>
__device__ __forceinline__ void score_loop(const SnapEntry* snap, int n, const ScoreArgs& a, const float* sg,
                                           const float* work, const int64_t* need, uint32_t* bkey,
                                           int32_t* bi) {
  for (int j = 0; j < n; ++j) {
    const SnapEntry e = snap[j];
#pragma unroll
    for (int r = 0; r < kReq; ++r) {
      float press;
      if constexpr (kNonNeg)
        press = (float)((uint32_t)e.kv + (uint32_t)need[r]) * a.inv_cap;
      else
        press = (float)((int64_t)e.kv + need[r]) * a.inv_cap;
      const float load = e.lb * sg[r];
      const float size = work[r] * (1.0f + a.rho * press) * sg[r];
      const float cost = load + size + e.qq;
      const uint32_t k = cost_key(cost);
      if (k < bkey[r]) {
        bkey[r] = k;
        bi[r] = j;
      }
    }
  }
}

__global__ void __launch_bounds__(kBlock) score_shared_kernel(ScoreArgs a) {
  extern __shared__ SnapEntry snap[];
  const int n = a.n_inst;
  int nonneg = 1;
  for (int j = threadIdx.x; j < n; j += kBlock) {
    SnapEntry e;
    e.lb = a.w_b * a.backlog[j];
    e.qq = a.w_q * (float)a.queue[j];
    e.kv = a.kv[j];
    e.pad = 0;
    nonneg &= e.kv >= 0;
    snap[j] = e;
  }
  nonneg = __syncthreads_and(nonneg);

  const int64_t first = ((int64_t)blockIdx.x * kBlock + threadIdx.x) * kReq;
  float sg[kReq], work[kReq];
  int64_t need[kReq];
  int32_t bi[kReq];
  uint32_t bkey[kReq];
  bool ok[kReq];
#pragma unroll
  for (int r = 0; r < kReq; ++r) {
    const int64_t i = first + r;
    ok[r] = false;
    sg[r] = 0.0f;
    work[r] = 0.0f;
    need[r] = 0;
    bi[r] = -1;
    bkey[r] = 0xffffffffu;
    if (i < a.n_req) {
      const int32_t p = a.plen[i];
      const int32_t oh = a.pool == 1 ? a.ohat[i] : 0;
      const uint32_t c = a.cls[i];
      ok[r] = req_ok(a.pool, p, oh, c);
      if (ok[r]) {
        sg[r] = a.sigma[c];
        work[r] = a.pool == 1 ? a.w_s * (float)oh * a.tau : a.w_s * (float)p * a.tau;
        need[r] = a.pool == 1 ? (int64_t)p + oh : (int64_t)p;
      }
    }
  }
  if (nonneg)
    score_loop<true>(snap, n, a, sg, work, need, bkey, bi);
  else
    score_loop<false>(snap, n, a, sg, work, need, bkey, bi);
#pragma unroll
  for (int r = 0; r < kReq; ++r) {
    const int64_t i = first + r;
    if (i < a.n_req) {
      a.out_idx[i] = ok[r] ? bi[r] : -1;
      a.out_score[i] = __uint_as_float(ok[r] ? bkey[r] : 0x7fc00000u);
    }
  }
}

template <int S>
__global__ void __launch_bounds__(kBlock) score_rows_kernel(ScoreArgs a) {
  constexpr int kSegs = 64 / S;
  const int lane = threadIdx.x & 63;
  const int sl = lane % S;
  const int64_t i = ((int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6)) * kSegs + lane / S;
  const bool live = i < a.n_req;
  int32_t p = 0, oh = 0;
  uint32_t c = 0;
  if (live) {
    p = a.plen[i];
    oh = a.pool == 1 ? a.ohat[i] : 0;
    c = a.cls[i];
  }
  const bool ok = live && req_ok(a.pool, p, oh, c);
  uint64_t best = ~0ull;  // (key << 32) | index
  if (ok) {
    const float sg = a.sigma[c];
    const float work = a.pool == 1 ? a.w_s * (float)oh * a.tau : a.w_s * (float)p * a.tau;
    const int64_t need = a.pool == 1 ? (int64_t)p + oh : (int64_t)p;
    const int64_t row = i * a.stride;
    for (int j = sl; j < a.n_inst; j += S) {
      const float press = (float)((int64_t)a.kv[row + j] + need) * a.inv_cap;
      const float load = a.w_b * a.backlog[row + j] * sg;
      const float size = work * (1.0f + a.rho * press) * sg;
      const float cost = load + size + a.w_q * (float)a.queue[row + j];
      const uint64_t k = ((uint64_t)cost_key(cost) << 32) | (uint32_t)j;
      best = k < best ? k : best;
    }
  }
#pragma unroll
  for (int m = 1; m < S; m <<= 1) {
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)best, m, 64);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(best >> 32), m, 64);
    const uint64_t o = ((uint64_t)hi << 32) | lo;
    best = o < best ? o : best;
  }
  if (live && sl == 0) {
    a.out_idx[i] = ok ? (int32_t)(uint32_t)best : -1;
    a.out_score[i] = __uint_as_float(ok ? (uint32_t)(best >> 32) : 0x7fc00000u);
  }
}

// Per-request rows of at most 64 instances, n_inst and the stride multiples
// of 4 and the snapshot arrays 16-byte aligned: 16 lanes per request, four
// consecutive instances per lane (one 16-byte load per array), four
// requests per wave and kRowGroups groups of four per wave, every load of a
// wave issued before its first cost.  Within a lane the four costs are taken
// in index order (the first of equal keys stays); the 16 lanes of a request
// reduce the key, then the lowest index holding it, with DPP within their
// row.
constexpr int kRowGroups = 4;

__device__ __forceinline__ uint32_t row_min(uint32_t v) {
  v = min(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, true));   // quad_perm xor 1
  v = min(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, true));   // quad_perm xor 2
  v = min(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x141, 0xF, 0xF, true));  // row_half_mirror
  v = min(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x140, 0xF, 0xF, true));  // row_mirror
  return v;
}

__global__ void __launch_bounds__(kBlock) score_rows16_kernel(ScoreArgs a) {
  constexpr int G = kRowGroups;
  const int lane = threadIdx.x & 63;
  const int rq = lane >> 4, ql = lane & 15;
  const int64_t wave = (int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  const int64_t first = wave * 4 * G;
  const int j0 = 4 * ql;  // this lane's first instance
  const bool lane_in = j0 < a.n_inst;
  float4 b4[G];
  int4 q4[G], k4[G];
  int32_t p[G], oh[G];
  uint32_t c[G];
  bool live[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int64_t i = first + 4 * g + rq;
    live[g] = i < a.n_req;
    const int64_t ii = live[g] ? i : 0;
    p[g] = a.plen[ii];
    oh[g] = a.pool == 1 ? a.ohat[ii] : 0;
    c[g] = a.cls[ii];
    const int64_t e = ii * a.stride + (lane_in ? j0 : 0);
    b4[g] = *reinterpret_cast<const float4*>(a.backlog + e);
    q4[g] = *reinterpret_cast<const int4*>(a.queue + e);
    k4[g] = *reinterpret_cast<const int4*>(a.kv + e);
  }
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const bool ok = live[g] && req_ok(a.pool, p[g], oh[g], c[g]);
    const float sg = a.sigma[c[g] & (kMaxClasses - 1)];
    const float work = a.pool == 1 ? a.w_s * (float)oh[g] * a.tau : a.w_s * (float)p[g] * a.tau;
    const uint32_t need = a.pool == 1 ? (uint32_t)p[g] + (uint32_t)oh[g] : (uint32_t)p[g];  // < 2^31 when ok
    const float bb[4] = {b4[g].x, b4[g].y, b4[g].z, b4[g].w};
    const int32_t qq[4] = {q4[g].x, q4[g].y, q4[g].z, q4[g].w};
    const int32_t kk[4] = {k4[g].x, k4[g].y, k4[g].z, k4[g].w};
    uint32_t bkey = 0xffffffffu;
    int32_t bj = j0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      // occupancy + need, exact in 32 bits: unsigned when the occupancy is
      // >= 0 (the sum is < 2^32), signed otherwise (the sum is < 2^31)
      const uint32_t sum = (uint32_t)kk[u] + need;
      const float kvn = kk[u] >= 0 ? (float)sum : (float)(int32_t)sum;
      const float press = kvn * a.inv_cap;
      const float load = a.w_b * bb[u] * sg;
      const float size = work * (1.0f + a.rho * press) * sg;
      const float cost = load + size + a.w_q * (float)qq[u];
      uint32_t k = cost_key(cost);
      k = lane_in ? k : 0xffffffffu;
      const bool b = k < bkey;
      bkey = b ? k : bkey;
      bj = b ? j0 + u : bj;
    }
    const uint32_t m = row_min(bkey);
    const uint32_t idx = row_min(bkey == m ? (uint32_t)bj : 0xffffffffu);
    const int64_t i = first + 4 * g + rq;
    if (live[g] && ql == 0) {
      a.out_idx[i] = ok ? (int32_t)idx : -1;
      a.out_score[i] = __uint_as_float(ok ? m : 0x7fc00000u);
    }
  }
}

__global__ void __launch_bounds__(kBlock) goodput_kernel(GoodputArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t rep = (int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  if (rep >= a.n_replicas) return;  // whole wave leaves together
  const int64_t lo = a.offsets[rep], hi = a.offsets[rep + 1];
  const int pid = a.param_point ? a.param_point[rep] : 0;
  if (lo < 0 || hi < lo || hi > a.n_requests || pid < 0 || pid >= a.n_points) {
    // a replica this trace does not describe consistently: no read outside it
    if (lane == 0) {
      a.goodput[rep] = 0.0;
      if (a.met) a.met[rep] = -1;
      atomicOr(a.flag, kFlagBadTrace);
    }
    return;
  }
  // the point's targets, lane k < 8 holding class k's (read per request
  // with a cross-lane shuffle instead of a dependent load)
  const DevPoint& pp = a.points[pid];
  const int k8 = lane & (kMaxClasses - 1);
  const int64_t my_ttft = pp.slo_ttft[k8], my_tpot = pp.slo_tpot[k8];
  int64_t met = 0;
  // four 64-request chunks per iteration, their loads issued together
  constexpr int kU = 4;
  for (int64_t i0 = lo; i0 < hi; i0 += 64 * kU) {
    int64_t tt[kU], sp[kU];
    int32_t o[kU];
    uint32_t c[kU];
    bool in[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int64_t i = i0 + u * 64 + lane;
      in[u] = i < hi;
      const int64_t j = in[u] ? i : lo;
      tt[u] = a.ttft[j];
      sp[u] = a.span[j];
      o[u] = a.olen[j];
      c[u] = a.cls[j];
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const bool valid = in[u] && tt[u] >= 0 && c[u] < (uint32_t)kMaxClasses;
      const int cc = valid ? (int)c[u] : 0;
      const int64_t lim_ttft = __shfl(my_ttft, cc, 64), lim_tpot = __shfl(my_tpot, cc, 64);
      const bool ok_ttft = tt[u] <= lim_ttft;
      const bool ok_tpot = o[u] <= 1 || sp[u] <= lim_tpot * (int64_t)(o[u] - 1);
      met += (valid && ok_ttft && ok_tpot) ? 1 : 0;
    }
  }
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) {
    const uint32_t l = (uint32_t)__shfl_xor((int)(uint32_t)met, m, 64);
    const uint32_t h = (uint32_t)__shfl_xor((int)(uint32_t)((uint64_t)met >> 32), m, 64);
    met += (int64_t)(((uint64_t)h << 32) | l);
  }
  if (lane == 0) {
    const int64_t n = hi - lo;
    a.goodput[rep] = n > 0 ? (double)met / (double)n : 0.0;
    if (a.met) a.met[rep] = met;
  }
}

}  // namespace

hipError_t launch_score(const ScoreArgs& a, hipStream_t stream) {
  if (a.n_req <= 0) return hipSuccess;
  if (a.stride == 0) {
    const int64_t per_block = (int64_t)kBlock * kReq;
    const int64_t blocks = (a.n_req + per_block - 1) / per_block;
    const size_t lds = sizeof(SnapEntry) * (size_t)a.n_inst;
    hipLaunchKernelGGL(score_shared_kernel, dim3((unsigned)blocks), dim3(kBlock), lds, stream, a);
    return hipGetLastError();
  }
  const bool aligned = ((uintptr_t)a.backlog | (uintptr_t)a.queue | (uintptr_t)a.kv) % 16 == 0;
  if (a.n_inst <= 64 && a.n_inst % 4 == 0 && a.stride % 4 == 0 && aligned) {
    const int64_t per_block = (kBlock / 64) * 4 * kRowGroups;
    const unsigned blocks = (unsigned)((a.n_req + per_block - 1) / per_block);
    hipLaunchKernelGGL(score_rows16_kernel, dim3(blocks), dim3(kBlock), 0, stream, a);
    return hipGetLastError();
  }
  int S = 1;
  while (S < a.n_inst && S < 64) S <<= 1;
  const int64_t per_block = (kBlock / 64) * (64 / S);
  const unsigned blocks = (unsigned)((a.n_req + per_block - 1) / per_block);
  switch (S) {
    case 1: hipLaunchKernelGGL(score_rows_kernel<1>, dim3(blocks), dim3(kBlock), 0, stream, a); break;
    case 2: hipLaunchKernelGGL(score_rows_kernel<2>, dim3(blocks), dim3(kBlock), 0, stream, a); break;
    case 4: hipLaunchKernelGGL(score_rows_kernel<4>, dim3(blocks), dim3(kBlock), 0, stream, a); break;
    case 8: hipLaunchKernelGGL(score_rows_kernel<8>, dim3(blocks), dim3(kBlock), 0, stream, a); break;
    case 16: hipLaunchKernelGGL(score_rows_kernel<16>, dim3(blocks), dim3(kBlock), 0, stream, a); break;
    case 32: hipLaunchKernelGGL(score_rows_kernel<32>, dim3(blocks), dim3(kBlock), 0, stream, a); break;
    default: hipLaunchKernelGGL(score_rows_kernel<64>, dim3(blocks), dim3(kBlock), 0, stream, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_goodput(const GoodputArgs& a, hipStream_t stream) {
  if (a.n_replicas <= 0) return hipSuccess;
  const unsigned blocks = (unsigned)((a.n_replicas + 3) / 4);
  hipLaunchKernelGGL(goodput_kernel, dim3(blocks), dim3(kBlock), 0, stream, a);
  return hipGetLastError();
}

}  // namespace rt
