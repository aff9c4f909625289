// Internal declarations shared by the HIP kernels and the C-ABI host code of
// librt_router.  Not installed; the public interface is include/rt_router.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rt {

constexpr int kMaxClasses = 8;

// One parameter point as the kernels read it: the public rt_point plus
// host-computed constants (reciprocal cache capacities).
struct DevPoint {
  int32_t P, D, n_classes, policy, mode, pad0[3];
  float w_b, w_s, w_q, rho;
  float tau_pre, tau_dec, pre_base;
  float inv_cap_pre, inv_cap_dec;  // 1.0f / (float)capacity, rounded once
  float pad1[3];
  float sigma[kMaxClasses];
  int64_t pre_base_ns, pre_tok_ns, dec_tok_ns, xfer_tok_ns;
  int64_t slo_ttft[kMaxClasses], slo_tpot[kMaxClasses];
};

enum : uint32_t { kFlagRejected = 1u, kFlagBadTrace = 2u, kFlagTimeRange = 4u };

// Arguments of the replica-simulation kernels.
struct SimArgs {
  const DevPoint* points;
  const int32_t* work;  // replica ids of this launch, in processing order
  int64_t n_work;
  const int64_t* offsets;
  const int32_t* param_point;  // may be null: every replica uses point 0
  const int64_t* arrival;
  const int32_t* plen;
  const int32_t* olen;
  const int32_t* ohat;
  const uint8_t* cls;
  int32_t* i_pre;
  int32_t* i_dec;
  int64_t* ttft;
  int64_t* span;
  // Successor records of the per-instance FIFOs (one slot per request and
  // pool, indexed by the global request index of the predecessor).
  int4* sp;       // prefill: {release (double bits lo, hi), successor index, prompt tokens}
  double* sd_t;   // decode release time
  int4* sd_m;     // decode: {successor index, cache tokens p+o, ledger tokens o^, 0}
  char* dummy;    // kDummyLanes private 64-byte slots (writes with nothing to write)
  uint32_t* flag;
};

constexpr int kDummyLanes = 1 << 16;

// Kernel classes: lanes per replica S (a power of two; S > 64 spans S/64
// waves of one workgroup) and instances per lane for each pool.
struct SimClass {
  int S, MP, MD;
};

hipError_t launch_sim(const SimClass& c, const SimArgs& a, hipStream_t stream);
int sim_class_count();
SimClass sim_class(int i);

struct ScoreArgs {
  float w_b, w_s, w_q, rho, tau, inv_cap;
  float sigma[kMaxClasses];
  int32_t pool, n_inst;
  int64_t stride, n_req;
  const float* backlog;
  const int32_t* queue;
  const int32_t* kv;
  const int32_t* plen;
  const int32_t* ohat;
  const uint8_t* cls;
  int32_t* out_idx;
  float* out_score;
};

hipError_t launch_score(const ScoreArgs& a, hipStream_t stream);

struct GoodputArgs {
  const DevPoint* points;
  int32_t n_points;
  int64_t n_requests;
  int64_t n_replicas;
  const int64_t* offsets;
  const int32_t* param_point;
  const int32_t* olen;
  const uint8_t* cls;
  const int64_t* ttft;
  const int64_t* span;
  double* goodput;
  int64_t* met;
  uint32_t* flag;
};

hipError_t launch_goodput(const GoodputArgs& a, hipStream_t stream);

// Ordering key of a non-negative cost for the argmin: both zeros equal, NaN
// after +inf, otherwise the IEEE bit pattern (monotone for x >= 0).
__device__ __forceinline__ uint32_t cost_key(float c) {
  uint32_t u = __float_as_uint(c);
  u = (c == 0.0f) ? 0u : u;
  u = (c != c) ? 0x7fc00000u : u;
  return u;
}

}  // namespace rt
