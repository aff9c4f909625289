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
  int32_t P, D, n_classes, policy, mode, len_thr;
  int32_t service, batch_cap;  // rt_service; ring capacity (power of two)
  float w_b, w_s, w_q, rho;
  float tau_pre, tau_dec, pre_base;
  float inv_cap_pre, inv_cap_dec;  // 1.0f / (float)capacity, rounded once
  float pad1[3];
  float sigma[kMaxClasses];
  int64_t pre_base_ns, pre_tok_ns, dec_tok_ns, xfer_tok_ns;
  int64_t slo_ttft[kMaxClasses], slo_tpot[kMaxClasses];
  double beta_pre, beta_dec;  // batched service: slowdown per extra member
};

enum : uint32_t { kFlagRejected = 1u, kFlagBadTrace = 2u, kFlagTimeRange = 4u, kFlagBatchCap = 8u };

// rt_policy values as the kernels read them from DevPoint::policy.
enum : int32_t {
  kPolicyLearned = 0,
  kPolicyRoundRobin = 1,
  kPolicyLeastLoaded = 2,
  kPolicyLearnedSampled = 3,
  kPolicyLengthThreshold = 4
};

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
  const uint32_t* samp;  // [n][4] candidate words (sampled modes only)
  int32_t* i_pre;
  int32_t* i_dec;
  int64_t* ttft;
  int64_t* span;
  // Successor records of the per-instance FIFOs, one plane per pool
  // (0 prefill, 1 decode), indexed by the global request index of the
  // predecessor.  Record x holds x's first and second successor in the same
  // instance's FIFO, each {release time (double), index, cache tokens}: one
  // aligned 32-byte sector.  The modes that price the ledger use 64-byte
  // records that hold the same successors' ledger tokens after the pair, so
  // that a release reads one line (rec_shift).  Every plane has
  // kDummyRecords more records right before its index 0, at indices
  // -1 .. -kDummyRecords: wave-private targets of record loads and stores
  // with nothing to do.
  char* rec[2];
  uint32_t* flag;
};

// Record x of a plane lies at byte x << rec_shift(ledger) from its index 0;
// in the ledger modes the two ledger tokens follow the pair at kRecTok.
constexpr int rec_shift(bool ledger) { return ledger ? 6 : 5; }
constexpr int kRecTok = 32;

constexpr int kDummyRecords = 1024;  // a power of two

// Kernel classes.  kSeg: one replica per aligned segment of S <= 64 lanes of
// one wave, prefill instances on the first lanes and decode instances on the
// next, MP = MD instances per lane; `mode` fixes the scoring path (clock
// backlog, ledger backlog, or a baseline policy; the two learned ones also
// over two sampled candidates per pool).  kWseg: the same for one replica
// per workgroup of S / 64 waves, instances dealt round-robin over the waves.
// kBat: the continuous-batching service model, one replica per lane.
enum SimKind { kSeg = 0, kWseg = 1, kBat = 2 };
enum SimMode { kModeTrue = 0, kModeProxy = 1, kModeBase = 2, kModeTrueSampled = 3, kModeProxySampled = 4 };
constexpr bool mode_ledger(int m) { return m == kModeProxy || m == kModeProxySampled; }  // proxy backlog
constexpr bool mode_sampled(int m) { return m == kModeTrueSampled || m == kModeProxySampled; }

struct SimClass {
  int kind, S, MP, MD, mode;
};

// Every kernel class, one-wave classes first (in order of preference), and
// the launch of one class over a work list.
hipError_t launch_sim(const SimClass& c, const SimArgs& a, hipStream_t stream);
int sim_class_count();
SimClass sim_class(int i);

// Scratch of the continuous-batching kernel for S lanes, NI instance slots
// per lane (the largest P + D of the launch) and ring capacity C (a power of
// two).  Per-instance state is structure-of-arrays, element [j * S + lane]
// (a wave reads 64 consecutive elements); the rings are per lane, contiguous,
// 16 bytes an entry, entry [((lane * NI + j) * C + pos].
struct BatScratch {
  double *v, *tl, *kv, *pend, *owed, *left;  // [NI][S]; left: the batch's remaining work
  int32_t *q, *nact, *head, *nw, *whead;   // [NI][S]
  char* ring;   // batch members {f, request}, sorted by (f, request) from head
  char* wring;  // KV transfers in flight {landing time, request}, sorted likewise
  int64_t S;
  int32_t NI, C;
};

// Bytes of BatScratch for S lanes, NI instance slots and capacity C, and the
// carving of one allocation into it.
size_t bat_scratch_bytes(int64_t S, int32_t NI, int32_t C);
BatScratch bat_scratch_carve(char* base, int64_t S, int32_t NI, int32_t C);
// Batched classes {S, M}: one replica per aligned segment of S lanes, M
// instances per lane (ceil(P / M) + ceil(D / M) <= S; MP = MD = M), then the
// general one, one replica per lane (S = 1, MP = MD = 0).  bat_lanes: the
// lanes a launch spans, each the owner of NI state slots and NI ring pairs in
// the class's scratch (NI = M for a segment class).
#define RT_BSEG_FOR_EACH(X) X(4, 1) X(8, 1) X(16, 1) X(32, 1) X(64, 1) X(64, 2)
hipError_t launch_bat(const SimClass& c, const SimArgs& a, const BatScratch& b, hipStream_t stream);
int64_t bat_lanes(const SimClass& c, int64_t n_work);

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
