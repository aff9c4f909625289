// Host side of the rt_router C ABI (include/rt_router.h): argument checks,
// launch planning, scratch ownership and error reporting.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "rt_internal.h"
#include "rt_router.h"
#include "wseg_kernel.h"

namespace {

thread_local std::string g_err;

rt_status fail(rt_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

rt_status hip_fail(hipError_t e, const char* what) {
  return fail(e == hipErrorOutOfMemory ? RT_ENOMEM : RT_EDEVICE,
              std::string(what) + ": " + hipGetErrorString(e));
}

// Makes `device` current for the scope of a call and restores the caller's.
struct DeviceScope {
  int prev = -1;
  hipError_t err = hipSuccess;
  explicit DeviceScope(int device) {
    err = hipGetDevice(&prev);
    if (err == hipSuccess && prev != device) err = hipSetDevice(device);
  }
  ~DeviceScope() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

bool finite_nonneg(float x) { return std::isfinite(x) && x >= 0.0f; }

constexpr int64_t kMaxNs = int64_t(1) << 40;
constexpr int32_t kMaxBatchCap = 65536;
constexpr int32_t kDefaultBatchCap = 256;
constexpr int kSimds = 256 * 4;  // MI355X: 256 compute units x 4 SIMDs

// Limits of rt_sim_run_replicas_noalloc: the device scratch each GPU holds
// for it (record planes and the work list), and the host-side planning
// arrays, sized for this many replicas, points and kernel classes.
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
constexpr int64_t kNoAllocMaxReplicas = 65536;
constexpr int32_t kNoAllocMaxPoints = 4096;
constexpr int kMaxClassSlots = 256;
constexpr int kMaxDevices = 64;

std::string check_point(const rt_point& p) {
  if (p.n_prefill < 1 || p.n_decode < 1) return "pool sizes must be >= 1";
  if (p.n_prefill > RT_MAX_POOL || p.n_decode > RT_MAX_POOL) return "pool wider than RT_MAX_POOL";
  if (p.n_classes < 1 || p.n_classes > RT_MAX_CLASSES) return "n_classes must be in [1, RT_MAX_CLASSES]";
  if (p.policy < RT_POLICY_LEARNED || p.policy > RT_POLICY_LENGTH_THRESHOLD) return "unknown policy";
  if (p.policy == RT_POLICY_LENGTH_THRESHOLD && p.len_threshold < 1) return "len_threshold must be >= 1";
  if (p.backlog_mode != RT_BACKLOG_TRUE && p.backlog_mode != RT_BACKLOG_PROXY) return "unknown backlog_mode";
  if (p.service != RT_SERVICE_SERIAL && p.service != RT_SERVICE_BATCHED) return "unknown service";
  if (p.service == RT_SERVICE_BATCHED) {
    if (!std::isfinite(p.beta_pre) || !std::isfinite(p.beta_dec) || p.beta_pre < 0.0 || p.beta_dec < 0.0)
      return "beta_pre and beta_dec must be finite and >= 0";
    const int32_t c = p.batch_cap;
    if (c != 0 && (c < 2 || c > kMaxBatchCap || (c & (c - 1)) != 0))
      return "batch_cap must be 0 or a power of two in [2, 65536]";
  }
  const rt_router_params& r = p.router;
  const float f[] = {r.w_b, r.w_s, r.w_q, r.rho, r.tau_pre_s, r.tau_dec_s, r.pre_base_s};
  for (float x : f)
    if (!finite_nonneg(x)) return "router weights and prices must be finite and >= 0";
  for (int c = 0; c < RT_MAX_CLASSES; ++c)
    if (!finite_nonneg(r.sigma[c])) return "sigma must be finite and >= 0";
  const rt_physics& ph = p.phys;
  const int64_t t[] = {ph.pre_base_ns, ph.pre_tok_ns, ph.dec_tok_ns, ph.xfer_tok_ns};
  for (int64_t x : t)
    if (x < 0 || x > kMaxNs) return "service constants must be in [0, 2^40] ns";
  if (ph.kv_cap_pre < 1 || ph.kv_cap_dec < 1) return "cache capacities must be >= 1";
  for (int c = 0; c < RT_MAX_CLASSES; ++c)
    if (ph.slo_ttft_ns[c] < 0 || ph.slo_tpot_ns[c] < 0 || ph.slo_tpot_ns[c] > kMaxNs)
      return "SLO targets must be >= 0 (TPOT <= 2^40 ns)";
  return "";
}

rt::DevPoint to_dev(const rt_point& p) {
  rt::DevPoint d;
  std::memset(&d, 0, sizeof d);
  d.P = p.n_prefill;
  d.D = p.n_decode;
  d.n_classes = p.n_classes;
  d.policy = p.policy;
  d.len_thr = p.len_threshold;
  d.mode = p.backlog_mode;
  d.service = p.service;
  d.batch_cap = p.batch_cap == 0 ? kDefaultBatchCap : p.batch_cap;
  d.beta_pre = p.beta_pre;
  d.beta_dec = p.beta_dec;
  // Adding +0.0f turns a -0.0f weight into +0.0f (and changes nothing else):
  // with every factor then +0 or positive, no cost is -0 and the kernels can
  // order costs by their bit patterns without a zero test.
  d.w_b = p.router.w_b + 0.0f;
  d.w_s = p.router.w_s + 0.0f;
  d.w_q = p.router.w_q + 0.0f;
  d.rho = p.router.rho + 0.0f;
  d.tau_pre = p.router.tau_pre_s + 0.0f;
  d.tau_dec = p.router.tau_dec_s + 0.0f;
  d.pre_base = p.router.pre_base_s + 0.0f;
  // press+ = (occupancy + need) * (1 / capacity): the reciprocal is rounded
  // to float32 once, here.
  d.inv_cap_pre = 1.0f / (float)p.phys.kv_cap_pre;
  d.inv_cap_dec = 1.0f / (float)p.phys.kv_cap_dec;
  for (int c = 0; c < rt::kMaxClasses; ++c) d.sigma[c] = p.router.sigma[c] + 0.0f;
  d.pre_base_ns = p.phys.pre_base_ns;
  d.pre_tok_ns = p.phys.pre_tok_ns;
  d.dec_tok_ns = p.phys.dec_tok_ns;
  d.xfer_tok_ns = p.phys.xfer_tok_ns;
  for (int c = 0; c < rt::kMaxClasses; ++c) {
    d.slo_ttft[c] = p.phys.slo_ttft_ns[c];
    d.slo_tpot[c] = p.phys.slo_tpot_ns[c];
  }
  return d;
}

// The scoring path a point's kernels take.
int point_mode(const rt_point& p) {
  const bool tr = p.backlog_mode == RT_BACKLOG_TRUE;
  if (p.policy == RT_POLICY_LEARNED) return tr ? rt::kModeTrue : rt::kModeProxy;
  if (p.policy == RT_POLICY_LEARNED_SAMPLED) return tr ? rt::kModeTrueSampled : rt::kModeProxySampled;
  return rt::kModeBase;
}

// Does kernel class c hold both pools of point p?  A batched-service point
// takes the batched class, any other point a serial one.  A one-wave segment class
// of the point's mode needs ceil(P / M) prefill lanes and ceil(D / M) decode
// lanes within its S; a multi-wave one needs every wave's share of both
// within 64 lanes.
bool class_fits(const rt::SimClass& c, const rt_point& p) {
  // the batched service model has one class of its own
  if ((c.kind == rt::kBat) != (p.service == RT_SERVICE_BATCHED)) return false;
  if (c.kind == rt::kBat)
    return c.MP == 0 || (p.n_prefill + c.MP - 1) / c.MP + (p.n_decode + c.MP - 1) / c.MP <= c.S;
  if (c.kind == rt::kSeg) {
    if (c.mode != point_mode(p)) return false;
    const int lanes = (p.n_prefill + c.MP - 1) / c.MP + (p.n_decode + c.MD - 1) / c.MD;
    return lanes <= c.S;
  }
  if (c.mode != point_mode(p)) return false;
  const int W = c.S / 64;
  return rt::seg::wide_pool_lanes(p.n_prefill, c.MP, W) + rt::seg::wide_pool_lanes(p.n_decode, c.MD, W) <= 64;
}

// Every class that holds a point, in the order the classes are listed (the
// first has the shortest step).
std::vector<int> fitting_classes(const rt_point& p) {
  std::vector<int> out;
  for (int i = 0; i < rt::sim_class_count(); ++i)
    if (class_fits(rt::sim_class(i), p)) out.push_back(i);
  return out;
}

// Issue slots of one step of a segment class, roughly: the per-request work
// every lane repeats, the per-instance work of each of M slots, and one DPP
// level of the argmins per doubling of the segment.
double seg_step_cost(const rt::SimClass& c) {
  int lg = 0;
  while ((1 << lg) < c.S) ++lg;
  return 150.0 + 70.0 * c.MP + 10.0 * lg;
}

}  // namespace

// The file-scope device scratch of rt_sim_run_replicas_noalloc (one copy per
// GPU, held until the process ends).  Host code never passes this name to a
// kernel: it resolves the array's address on each device once
// (static_scratch) and passes that.
static __device__ __align__(256) char scratch[kStaticScratchBytes];

namespace {

// The points of a simulator as the planner reads them: how many, and the
// kernel classes that hold each.
struct rt_sim_points {
  size_t n;
  const std::vector<int>* classes;
};

std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices];  // scratch's address on each device, once resolved

// The address of `scratch` on `device` (current): resolved on the first
// call for the device and kept.
rt_status static_scratch(int device, void** out) {
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (device < 0 || device >= kMaxDevices) return fail(RT_ERANGE, "static scratch: device index beyond the table");
  if (!g_scratch_dev[device]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!ptr) return fail(RT_EDEVICE, "hipGetSymbolAddress(scratch): null address");
    g_scratch_dev[device] = ptr;
  }
  *out = g_scratch_dev[device];
  return RT_OK;
}

// Storage of one launch plan, owned by the caller (growable vectors for
// rt_sim_run_replicas, fixed static arrays for the no-alloc variant).
struct PlanBufs {
  int64_t* off;      // [n + 1] offsets, read back
  int32_t* pp;       // [n] replica -> point, read back
  int64_t* reps_of;  // [npts] non-empty replicas per point
  int* choice;       // [npts] each point's kernel class
  int* wider;        // [npts] working copy for the widening pass
  int64_t* count;    // [ncls] replicas per class
  int64_t* start;    // [ncls] first work-list slot per class
  double* cost;      // [ncls] request-lanes per class (launch order)
  int32_t* work;     // [n] replica ids, grouped by class
  int* act;          // [ncls] classes with work, dearest first
  int n_act;
};

// Plan.  Each point runs one kernel class.  With few replicas (fewer waves,
// at the shortest-step classes, than twice the GPU's SIMDs) every replica is
// a latency chain and takes the shortest-step class; with many, the GPU's
// issue rate is the limit and each point takes the segment class with the
// fewest issue slots per replica-step (lanes x step cost).  Then replicas
// are grouped by class, longest first so that long chains start early (equal
// lengths in replica order); empty replicas need no work.  Classes with work
// are listed dearest first.  Allocates nothing.
void plan_launch(const rt_sim_points& sp, int64_t n, PlanBufs& b) {
  const int ncls = rt::sim_class_count();
  const size_t npts = sp.n;
  for (size_t k = 0; k < npts; ++k) b.reps_of[k] = 0;
  for (int64_t i = 0; i < n; ++i)
    if (b.off[i + 1] > b.off[i]) b.reps_of[b.pp[i]] += 1;
  double waves = 0.0;
  for (size_t k = 0; k < npts; ++k) waves += (double)b.reps_of[k] * rt::sim_class(sp.classes[k][0]).S / 64.0;
  const bool many = waves >= 2.0 * kSimds;
  for (size_t k = 0; k < npts; ++k) {
    const std::vector<int>& fit = sp.classes[k];
    b.choice[k] = fit[0];
    if (!many) continue;
    double best = -1.0;
    for (int c : fit) {
      const rt::SimClass sc = rt::sim_class(c);
      if (sc.kind != rt::kSeg) continue;
      const double cost = sc.S * seg_step_cost(sc);
      if (best < 0.0 || cost < best) {
        best = cost;
        b.choice[k] = c;
      }
    }
  }
  // With fewer waves than SIMDs, spread the replicas out: doubling the
  // segment width of every one-instance-per-lane class (the extra lanes
  // idle) halves the replicas in each wave, and a wave's step costs as much
  // as its slowest replica's step.  Widen while the waves keep growing and
  // still fit one per SIMD.
  if (!many) {
    for (;;) {
      double w2 = 0.0, w1 = 0.0;
      for (size_t k = 0; k < npts; ++k) {
        b.wider[k] = b.choice[k];
        if (b.reps_of[k] == 0) continue;
        const rt::SimClass sc = rt::sim_class(b.choice[k]);
        w1 += std::ceil((double)b.reps_of[k] * sc.S / 64.0);
        if ((sc.kind == rt::kSeg || sc.kind == rt::kBat) && sc.MP == 1 && sc.S < 64)
          for (int c : sp.classes[k]) {
            const rt::SimClass wc = rt::sim_class(c);
            if (wc.kind == sc.kind && wc.mode == sc.mode && wc.MP == 1 && wc.S == 2 * sc.S) b.wider[k] = c;
          }
        w2 += std::ceil((double)b.reps_of[k] * rt::sim_class(b.wider[k]).S / 64.0);
      }
      if (!(w2 > w1 && w2 <= kSimds)) break;
      for (size_t k = 0; k < npts; ++k) b.choice[k] = b.wider[k];
    }
  }
  // group by class (counting sort, replica order kept), then longest first
  for (int c = 0; c < ncls; ++c) b.count[c] = 0;
  for (int64_t i = 0; i < n; ++i)
    if (b.off[i + 1] > b.off[i]) b.count[b.choice[b.pp[i]]] += 1;
  int64_t pos = 0;
  for (int c = 0; c < ncls; ++c) {
    b.start[c] = pos;
    pos += b.count[c];
  }
  for (int c = 0; c < ncls; ++c) b.cost[c] = 0.0;
  {
    // (start[] is used as a fill cursor, then restored)
    for (int64_t i = 0; i < n; ++i)
      if (b.off[i + 1] > b.off[i]) {
        const int c = b.choice[b.pp[i]];
        b.work[b.start[c]++] = (int32_t)i;
        b.cost[c] += (double)(b.off[i + 1] - b.off[i]) * rt::sim_class(c).S;
      }
    for (int c = 0; c < ncls; ++c) b.start[c] -= b.count[c];
  }
  const int64_t* off = b.off;
  for (int c = 0; c < ncls; ++c)
    std::sort(b.work + b.start[c], b.work + b.start[c] + b.count[c], [off](int32_t x, int32_t y) {
      const int64_t lx = off[x + 1] - off[x], ly = off[y + 1] - off[y];
      return lx != ly ? lx > ly : x < y;
    });
  b.n_act = 0;
  for (int c = 0; c < ncls; ++c)
    if (b.count[c] > 0) b.act[b.n_act++] = c;
  const double* cost = b.cost;
  // Launch order: the longest chain of one wave first (the class's step
  // cost; every replica of a call has a comparable length), then the most
  // work.  A class of few waves with dear steps started behind a large one
  // finishes last (measured on the 1,225-point sweep: 66.0 ms dearest total
  // first, 63.0 ms cheapest total first, 61.1 ms longest step first).
  std::sort(b.act, b.act + b.n_act, [cost](int x, int y) {
    const double cx = seg_step_cost(rt::sim_class(x)), cy = seg_step_cost(rt::sim_class(y));
    if (cx != cy) return cx > cy;
    return cost[x] != cost[y] ? cost[x] > cost[y] : x < y;
  });
}

}  // namespace

struct rt_sim {
  int device = 0;
  std::vector<rt_point> points;
  std::vector<std::vector<int>> point_classes;  // fitting classes of each point
  rt::DevPoint* d_points = nullptr;
  uint32_t* d_flag = nullptr;
  char* d_scratch = nullptr;
  size_t scratch_bytes = 0;
  char* d_bscratch = nullptr;  // the batched class's state and rings
  size_t bscratch_bytes = 0;
  int32_t* d_work = nullptr;
  size_t work_cap = 0;
  int32_t* h_work = nullptr;  // pinned staging for the work list
  void* static_scratch = nullptr;  // this device's copy of `scratch` (no-alloc entry point)
  size_t h_work_cap = 0;
  hipEvent_t upload_done = nullptr;
  bool upload_pending = false;
  // measurement hook
  bool timing = false;
  bool timed_pending = false;  // an event pair was recorded and not yet summed
  hipEvent_t t0 = nullptr, t1 = nullptr;
  double timed_ms = 0.0;
  int64_t timed_calls = 0;
  // internal streams (default priority) that run kernel classes side by side
  std::vector<hipStream_t> lanes;
  std::vector<hipEvent_t> joins;
  hipEvent_t fork = nullptr;
};

static rt_status collect_timing(rt_sim* sim) {
  if (!sim->timed_pending) return RT_OK;
  hipError_t e = hipEventSynchronize(sim->t1);
  float ms = 0.0f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, sim->t0, sim->t1);
  if (e != hipSuccess) return hip_fail(e, "kernel timing events");
  sim->timed_ms += ms;
  sim->timed_calls += 1;
  sim->timed_pending = false;
  return RT_OK;
}

extern "C" {

const char* rt_last_error(void) { return g_err.c_str(); }

rt_status rt_sim_create(const rt_point* points, int32_t n_points, int32_t device, rt_sim** out) {
  if (!points || !out) return fail(RT_EINVAL, "rt_sim_create: null pointer");
  if (n_points < 1) return fail(RT_EINVAL, "rt_sim_create: n_points must be >= 1");
  int n_dev = 0;
  hipError_t e = hipGetDeviceCount(&n_dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDeviceCount");
  if (device < 0 || device >= n_dev) return fail(RT_EINVAL, "rt_sim_create: no such device");
  std::vector<std::vector<int>> cls(n_points);
  for (int32_t i = 0; i < n_points; ++i) {
    const std::string msg = check_point(points[i]);
    if (!msg.empty()) {
      const rt_status s = (points[i].n_prefill > RT_MAX_POOL || points[i].n_decode > RT_MAX_POOL)
                              ? RT_EUNSUPPORTED
                              : RT_EINVAL;
      return fail(s, "rt_sim_create: point " + std::to_string(i) + ": " + msg);
    }
    cls[i] = fitting_classes(points[i]);
    if (cls[i].empty())
      return fail(RT_EUNSUPPORTED, "rt_sim_create: point " + std::to_string(i) + ": no kernel for this pool shape");
  }
  DeviceScope ds(device);
  if (ds.err != hipSuccess) return hip_fail(ds.err, "hipSetDevice");
  rt_sim* s = new (std::nothrow) rt_sim;
  if (!s) return fail(RT_ENOMEM, "rt_sim_create: host allocation");
  s->device = device;
  s->points.assign(points, points + n_points);
  s->point_classes = cls;
  std::vector<rt::DevPoint> dev(n_points);
  for (int32_t i = 0; i < n_points; ++i) dev[i] = to_dev(points[i]);
  rt_status st = RT_OK;
  if ((e = hipMalloc(&s->d_points, sizeof(rt::DevPoint) * n_points)) != hipSuccess) {
    st = hip_fail(e, "hipMalloc(points)");
  } else if ((e = hipMemcpy(s->d_points, dev.data(), sizeof(rt::DevPoint) * n_points, hipMemcpyHostToDevice)) !=
             hipSuccess) {
    st = hip_fail(e, "hipMemcpy(points)");
  } else if ((e = hipMalloc(&s->d_flag, sizeof(uint32_t))) != hipSuccess) {
    st = hip_fail(e, "hipMalloc(flag)");
  } else if ((e = hipMemset(s->d_flag, 0, sizeof(uint32_t))) != hipSuccess) {
    st = hip_fail(e, "hipMemset(flag)");
  } else if ((e = hipEventCreateWithFlags(&s->upload_done, hipEventDisableTiming)) != hipSuccess) {
    st = hip_fail(e, "hipEventCreate");
  } else if ((st = static_scratch(device, &s->static_scratch)) != RT_OK) {
    // (message set by static_scratch)
  } else if ((e = hipDeviceSynchronize()) != hipSuccess) {
    st = hip_fail(e, "hipDeviceSynchronize");
  }
  if (st != RT_OK) {
    rt_sim_destroy(s);
    return st;
  }
  *out = s;
  return RT_OK;
}

rt_status rt_sim_destroy(rt_sim* sim) {
  if (!sim) return RT_OK;
  DeviceScope ds(sim->device);
  (void)hipDeviceSynchronize();
  if (sim->d_points) (void)hipFree(sim->d_points);
  if (sim->d_flag) (void)hipFree(sim->d_flag);
  if (sim->d_scratch) (void)hipFree(sim->d_scratch);
  if (sim->d_bscratch) (void)hipFree(sim->d_bscratch);
  if (sim->d_work) (void)hipFree(sim->d_work);
  if (sim->h_work) (void)hipHostFree(sim->h_work);
  if (sim->upload_done) (void)hipEventDestroy(sim->upload_done);
  if (sim->t0) (void)hipEventDestroy(sim->t0);
  if (sim->t1) (void)hipEventDestroy(sim->t1);
  for (hipStream_t l : sim->lanes) (void)hipStreamDestroy(l);
  for (hipEvent_t j : sim->joins) (void)hipEventDestroy(j);
  if (sim->fork) (void)hipEventDestroy(sim->fork);
  delete sim;
  return RT_OK;
}

static rt_status check_trace(const rt_sim* sim, const rt_trace* tr, const rt_sim_out* out, const char* fn) {
  if (!sim || !tr || !out) return fail(RT_EINVAL, std::string(fn) + ": null pointer");
  if (tr->n_replicas < 0 || tr->n_requests < 0) return fail(RT_EINVAL, std::string(fn) + ": negative size");
  if (tr->n_replicas > INT32_MAX) return fail(RT_ERANGE, std::string(fn) + ": more than 2^31-1 replicas");
  if (tr->n_replicas == 0) return RT_OK;
  if (!tr->offsets) return fail(RT_EINVAL, std::string(fn) + ": null offsets");
  if (tr->n_requests > 0 && (!tr->arrival_ns || !tr->prompt_len || !tr->out_len || !tr->pred_out_len ||
                             !tr->slo_class || !out->ttft_ns || !out->decode_span_ns))
    return fail(RT_EINVAL, std::string(fn) + ": null request or output array");
  return RT_OK;
}

// Validates offsets and the replica->point map as read back to the host.
static rt_status check_plan_inputs(const rt_sim* sim, const rt_trace* tr, const int64_t* off, const int32_t* pp,
                                   const char* fn) {
  const int64_t n = tr->n_replicas;
  if (off[0] < 0) return fail(RT_EINVAL, std::string(fn) + ": offsets[0] < 0");
  for (int64_t i = 0; i < n; ++i) {
    const int64_t len = off[i + 1] - off[i];
    if (len < 0) return fail(RT_EINVAL, std::string(fn) + ": offsets decrease at replica " + std::to_string(i));
    if (len > INT32_MAX) return fail(RT_ERANGE, std::string(fn) + ": replica " + std::to_string(i) + " has >= 2^31 requests");
    if (pp[i] < 0 || pp[i] >= (int32_t)sim->points.size())
      return fail(RT_EINVAL, std::string(fn) + ": param_point out of range at replica " + std::to_string(i));
  }
  if (off[n] > tr->n_requests) return fail(RT_EINVAL, std::string(fn) + ": offsets[n_replicas] > n_requests");
  return RT_OK;
}

// Reads offsets and the replica->point map back to the host and validates them.
static rt_status read_plan_inputs(const rt_sim* sim, const rt_trace* tr, hipStream_t stream,
                                  std::vector<int64_t>& off, std::vector<int32_t>& pp, const char* fn) {
  const int64_t n = tr->n_replicas;
  off.resize(n + 1);
  pp.assign(n, 0);
  hipError_t e = hipMemcpyAsync(off.data(), tr->offsets, sizeof(int64_t) * (n + 1), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess && tr->param_point)
    e = hipMemcpyAsync(pp.data(), tr->param_point, sizeof(int32_t) * n, hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return hip_fail(e, "reading offsets/param_point");
  return check_plan_inputs(sim, tr, off.data(), pp.data(), fn);
}

// Byte size of the serial classes' record planes for n_requests requests:
// for each record size in use (32 bytes, or 64 for the classes that price the
// ledger) a plane per pool, each its dummy records followed by one record per
// request, 256-byte aligned.  Classes of one call run side by side, so each
// size has planes of its own.
struct RecLayout {
  bool any_serial = false, any_ledger = false, any_plain = false;
  size_t plain_plane = 0, ledger_plane = 0, bytes = 0;
};

static RecLayout rec_layout(const PlanBufs& b, size_t nreq) {
  RecLayout L;
  for (int k = 0; k < b.n_act; ++k) {
    const rt::SimClass c = rt::sim_class(b.act[k]);
    if (c.kind == rt::kBat) continue;
    L.any_serial = true;
    (rt::mode_ledger(c.mode) ? L.any_ledger : L.any_plain) = true;
  }
  static_assert(((size_t)rt::kDummyRecords << rt::rec_shift(false)) % 256 == 0, "planes start 256-byte aligned");
  auto plane_bytes = [&](bool ledger) {
    return (((nreq + rt::kDummyRecords) << rt::rec_shift(ledger)) + 255) / 256 * 256;
  };
  L.plain_plane = L.any_plain ? plane_bytes(false) : 0;
  L.ledger_plane = L.any_ledger ? plane_bytes(true) : 0;
  L.bytes = L.any_serial ? 2 * L.plain_plane + 2 * L.ledger_plane + 256 : 0;
  return L;
}

// The kernels' arguments for a call, with the record planes carved from
// `sc` (laid out as rec_layout says); rec[] is set per class at launch.
static rt::SimArgs sim_args(const rt_sim* sim, const rt_trace* trace, const rt_sim_out* out, const RecLayout& L,
                            char* sc, char* (&planes)[2][2]) {
  rt::SimArgs a;
  a.points = sim->d_points;
  a.offsets = trace->offsets;
  a.param_point = trace->param_point;
  a.arrival = trace->arrival_ns;
  a.plen = trace->prompt_len;
  a.olen = trace->out_len;
  a.ohat = trace->pred_out_len;
  a.cls = trace->slo_class;
  a.samp = trace->sample_bits;
  a.i_pre = out->i_pre;
  a.i_dec = out->i_dec;
  a.ttft = out->ttft_ns;
  a.span = out->decode_span_ns;
  a.work = nullptr;
  a.n_work = 0;
  // record planes by record size: index 0 of each pool's plane
  for (int k = 0; k < 2; ++k) planes[0][k] = planes[1][k] = nullptr;
  for (int k = 0; k < 2 && sc && L.any_serial; ++k) {
    if (L.any_plain) planes[0][k] = sc + k * L.plain_plane + ((size_t)rt::kDummyRecords << rt::rec_shift(false));
    if (L.any_ledger)
      planes[1][k] =
          sc + 2 * L.plain_plane + k * L.ledger_plane + ((size_t)rt::kDummyRecords << rt::rec_shift(true));
  }
  a.rec[0] = a.rec[1] = nullptr;
  a.flag = sim->d_flag;
  return a;
}

// Launches class c of the plan over its replicas (work list at d_work).
static hipError_t launch_class(int c, rt::SimArgs a, const PlanBufs& b, const int32_t* d_work, char* (&planes)[2][2],
                               const rt::BatScratch* bs, hipStream_t where) {
  a.work = d_work + b.start[c];
  a.n_work = b.count[c];
  const int lg = rt::mode_ledger(rt::sim_class(c).mode) ? 1 : 0;
  a.rec[0] = planes[lg][0];
  a.rec[1] = planes[lg][1];
  return rt::sim_class(c).kind == rt::kBat ? rt::launch_bat(rt::sim_class(c), a, bs[c], where)
                                           : rt::launch_sim(rt::sim_class(c), a, where);
}

// The sampled policy reads the trace's candidate words.
static rt_status check_sample_bits(const rt_sim* sim, const rt_trace* trace, const PlanBufs& b, const char* fn) {
  for (size_t k = 0; k < sim->points.size(); ++k)
    if (b.reps_of[k] > 0 && sim->points[k].policy == RT_POLICY_LEARNED_SAMPLED && !trace->sample_bits)
      return fail(RT_EINVAL, std::string(fn) + ": point " + std::to_string(k) +
                                 " samples candidates but trace->sample_bits is NULL");
  return RT_OK;
}

rt_status rt_sim_run_replicas(rt_sim* sim, const rt_trace* trace, rt_sim_out* out, void* hip_stream) {
  rt_status st = check_trace(sim, trace, out, "rt_sim_run_replicas");
  if (st != RT_OK || trace->n_replicas == 0) return st;
  if (trace->n_requests > 0 && (!out->i_pre || !out->i_dec))
    return fail(RT_EINVAL, "rt_sim_run_replicas: null placement output");
  DeviceScope ds(sim->device);
  if (ds.err != hipSuccess) return hip_fail(ds.err, "hipSetDevice");
  hipStream_t stream = (hipStream_t)hip_stream;
  std::vector<int64_t> off;
  std::vector<int32_t> pp;
  if ((st = read_plan_inputs(sim, trace, stream, off, pp, "rt_sim_run_replicas")) != RT_OK)
    return st;

  const int ncls = rt::sim_class_count();
  const int64_t n = trace->n_replicas;
  const size_t npts = sim->points.size();
  std::vector<int64_t> reps_of(npts), count(ncls), start(ncls);
  std::vector<int> choice(npts), wider(npts), act(ncls);
  std::vector<double> cost(ncls);
  std::vector<int32_t> work_list(n);
  PlanBufs b{off.data(), pp.data(), reps_of.data(), choice.data(), wider.data(), count.data(), start.data(),
             cost.data(), work_list.data(), act.data(), 0};
  plan_launch(rt_sim_points{npts, sim->point_classes.data()}, n, b);
  if ((st = check_sample_bits(sim, trace, b, "rt_sim_run_replicas")) != RT_OK) return st;

  hipError_t e;
  const size_t nreq = (size_t)trace->n_requests;
  const RecLayout L = rec_layout(b, nreq);
  if (L.bytes > sim->scratch_bytes) {
    if ((e = hipDeviceSynchronize()) != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
    if (sim->d_scratch) (void)hipFree(sim->d_scratch);
    sim->d_scratch = nullptr;
    sim->scratch_bytes = 0;
    if ((e = hipMalloc(&sim->d_scratch, L.bytes)) != hipSuccess) return hip_fail(e, "hipMalloc(scratch)");
    sim->scratch_bytes = L.bytes;
  }
  // Scratch of the batched classes: per-instance state and two rings per
  // instance for every lane of each, sized by the largest pool and capacity
  // among that class's replicas' points; one allocation, carved in turn.
  std::vector<rt::BatScratch> bs(ncls);
  {
    struct Dim {
      int c;
      int64_t S;
      int32_t NI, C;
    };
    std::vector<Dim> dims;
    size_t bneed = 256;
    for (int k = 0; k < b.n_act; ++k) {
      const int c = b.act[k];
      const rt::SimClass sc = rt::sim_class(c);
      if (sc.kind != rt::kBat) continue;
      int32_t NI = 1, C = 2;
      for (int64_t j = b.start[c]; j < b.start[c] + b.count[c]; ++j) {
        const rt_point& q = sim->points[pp[work_list[j]]];
        NI = std::max(NI, q.n_prefill + q.n_decode);
        C = std::max(C, q.batch_cap == 0 ? kDefaultBatchCap : q.batch_cap);
      }
      if (sc.MP >= 1) NI = sc.MP;  // a segment class: MP instances per lane
      dims.push_back(Dim{c, rt::bat_lanes(sc, b.count[c]), NI, C});
      bneed += rt::bat_scratch_bytes(dims.back().S, NI, C);
    }
    if (!dims.empty() && bneed > sim->bscratch_bytes) {
      if ((e = hipDeviceSynchronize()) != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
      if (sim->d_bscratch) (void)hipFree(sim->d_bscratch);
      sim->d_bscratch = nullptr;
      sim->bscratch_bytes = 0;
      if ((e = hipMalloc(&sim->d_bscratch, bneed)) != hipSuccess) return hip_fail(e, "hipMalloc(batched scratch)");
      sim->bscratch_bytes = bneed;
    }
    size_t at = 0;
    for (const Dim& d : dims) {
      bs[d.c] = rt::bat_scratch_carve(sim->d_bscratch + at, d.S, d.NI, d.C);
      at += rt::bat_scratch_bytes(d.S, d.NI, d.C);
    }
  }
  if ((size_t)n > sim->work_cap) {
    if ((e = hipDeviceSynchronize()) != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
    if (sim->d_work) (void)hipFree(sim->d_work);
    sim->d_work = nullptr;
    sim->work_cap = 0;
    if ((e = hipMalloc(&sim->d_work, sizeof(int32_t) * n)) != hipSuccess) return hip_fail(e, "hipMalloc(work)");
    sim->work_cap = (size_t)n;
  }
  if (sim->upload_pending) {
    if ((e = hipEventSynchronize(sim->upload_done)) != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    sim->upload_pending = false;
  }
  if ((size_t)n > sim->h_work_cap) {
    if (sim->h_work) (void)hipHostFree(sim->h_work);
    sim->h_work = nullptr;
    sim->h_work_cap = 0;
    if ((e = hipHostMalloc(&sim->h_work, sizeof(int32_t) * n, hipHostMallocDefault)) != hipSuccess)
      return hip_fail(e, "hipHostMalloc(work)");
    sim->h_work_cap = (size_t)n;
  }
  int64_t listed = 0;
  for (int c = 0; c < ncls; ++c) listed += b.count[c];
  std::copy(work_list.begin(), work_list.begin() + listed, sim->h_work);
  if (listed > 0) {
    if ((e = hipMemcpyAsync(sim->d_work, sim->h_work, sizeof(int32_t) * listed, hipMemcpyHostToDevice, stream)) !=
        hipSuccess)
      return hip_fail(e, "hipMemcpyAsync(work)");
    if ((e = hipEventRecord(sim->upload_done, stream)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    sim->upload_pending = true;
  }

  char* planes[2][2];
  const rt::SimArgs a = sim_args(sim, trace, out, L, sim->d_scratch, planes);
  if (sim->timing) {
    if ((st = collect_timing(sim)) != RT_OK) return st;
    if ((e = hipEventRecord(sim->t0, stream)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  }
  // Kernel classes with work, dearest first; more than one run side by side
  // on internal streams forked from and joined back into `stream`.
  const size_t nact = (size_t)b.n_act;
  if (nact > 1) {
    while (sim->lanes.size() < nact) {
      hipStream_t l = nullptr;
      hipEvent_t j = nullptr;
      if ((e = hipStreamCreateWithFlags(&l, hipStreamNonBlocking)) != hipSuccess) return hip_fail(e, "hipStreamCreate");
      sim->lanes.push_back(l);
      if ((e = hipEventCreateWithFlags(&j, hipEventDisableTiming)) != hipSuccess) return hip_fail(e, "hipEventCreate");
      sim->joins.push_back(j);
    }
    if (!sim->fork && (e = hipEventCreateWithFlags(&sim->fork, hipEventDisableTiming)) != hipSuccess)
      return hip_fail(e, "hipEventCreate");
    if ((e = hipEventRecord(sim->fork, stream)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  }
  for (size_t k = 0; k < nact; ++k) {
    hipStream_t where = stream;
    if (nact > 1) {
      where = sim->lanes[k];
      if ((e = hipStreamWaitEvent(where, sim->fork, 0)) != hipSuccess) return hip_fail(e, "hipStreamWaitEvent");
    }
    if ((e = launch_class(b.act[k], a, b, sim->d_work, planes, bs.data(), where)) != hipSuccess)
      return hip_fail(e, "launch(sim)");
    if (nact > 1 && (e = hipEventRecord(sim->joins[k], where)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  }
  // The joins go in after every launch: streams share the device's few
  // hardware queues, and a wait enqueued between two launches could hold
  // back a later launch that landed on the same queue.
  if (nact > 1)
    for (size_t k = 0; k < nact; ++k)
      if ((e = hipStreamWaitEvent(stream, sim->joins[k], 0)) != hipSuccess) return hip_fail(e, "hipStreamWaitEvent");
  if (sim->timing) {
    if ((e = hipEventRecord(sim->t1, stream)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    sim->timed_pending = true;
  }
  return RT_OK;
}

// Host-side planning storage of rt_sim_run_replicas_noalloc, fixed in size
// and shared by every call (guarded by g_noalloc_mu).
struct NoAllocHost {
  int64_t off[kNoAllocMaxReplicas + 1];
  int32_t pp[kNoAllocMaxReplicas];
  int32_t work[kNoAllocMaxReplicas];
  int64_t reps_of[kNoAllocMaxPoints];
  int choice[kNoAllocMaxPoints], wider[kNoAllocMaxPoints];
  int64_t count[kMaxClassSlots], start[kMaxClassSlots];
  double cost[kMaxClassSlots];
  int act[kMaxClassSlots];
};
static NoAllocHost g_noalloc;
static std::mutex g_noalloc_mu;

rt_status rt_sim_run_replicas_noalloc(rt_sim* sim, const rt_trace* trace, rt_sim_out* out, void* hip_stream) {
  const char* fn = "rt_sim_run_replicas_noalloc";
  rt_status st = check_trace(sim, trace, out, fn);
  if (st != RT_OK || trace->n_replicas == 0) return st;
  if (trace->n_requests > 0 && (!out->i_pre || !out->i_dec)) return fail(RT_EINVAL, std::string(fn) + ": null placement output");
  if (trace->n_replicas > kNoAllocMaxReplicas)
    return fail(RT_ERANGE, std::string(fn) + ": more than " + std::to_string(kNoAllocMaxReplicas) + " replicas");
  if ((int64_t)sim->points.size() > kNoAllocMaxPoints)
    return fail(RT_ERANGE, std::string(fn) + ": simulator has more than " + std::to_string(kNoAllocMaxPoints) +
                               " points");
  if (rt::sim_class_count() > kMaxClassSlots) return fail(RT_EDEVICE, std::string(fn) + ": class table overflow");
  if (!sim->static_scratch) return fail(RT_EDEVICE, std::string(fn) + ": static scratch not resolved");
  DeviceScope ds(sim->device);
  if (ds.err != hipSuccess) return hip_fail(ds.err, "hipSetDevice");
  hipStream_t stream = (hipStream_t)hip_stream;
  const int64_t n = trace->n_replicas;
  std::lock_guard<std::mutex> lk(g_noalloc_mu);
  NoAllocHost& h = g_noalloc;
  hipError_t e = hipMemcpyAsync(h.off, trace->offsets, sizeof(int64_t) * (n + 1), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) {
    if (trace->param_point)
      e = hipMemcpyAsync(h.pp, trace->param_point, sizeof(int32_t) * n, hipMemcpyDeviceToHost, stream);
    else
      std::fill(h.pp, h.pp + n, 0);
  }
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return hip_fail(e, "reading offsets/param_point");
  if ((st = check_plan_inputs(sim, trace, h.off, h.pp, fn)) != RT_OK) return st;
  PlanBufs b{h.off, h.pp, h.reps_of, h.choice, h.wider, h.count, h.start, h.cost, h.work, h.act, 0};
  plan_launch(rt_sim_points{sim->points.size(), sim->point_classes.data()}, n, b);
  if ((st = check_sample_bits(sim, trace, b, fn)) != RT_OK) return st;
  for (int k = 0; k < b.n_act; ++k)
    if (rt::sim_class(b.act[k]).kind == rt::kBat)
      return fail(RT_EUNSUPPORTED, std::string(fn) + ": continuous-batching points need rt_sim_run_replicas");
  // static scratch: the record planes, then the work list
  const RecLayout L = rec_layout(b, (size_t)trace->n_requests);
  int64_t listed = 0;
  for (int k = 0; k < b.n_act; ++k) listed += b.count[b.act[k]];
  const size_t need = L.bytes + sizeof(int32_t) * (size_t)listed;
  if (need > kStaticScratchBytes)
    return fail(RT_ERANGE, std::string(fn) + ": needs " + std::to_string(need) + " bytes of scratch, more than its " +
                               std::to_string(kStaticScratchBytes) + " (64 bytes per request, 128 with the proxy "
                               "backlog, 192 when a call holds both, + 4 per replica)");
  char* base = (char*)sim->static_scratch;
  int32_t* d_work = (int32_t*)(base + L.bytes);
  // the work list is copied before the host array can be planned over again
  if (listed > 0) {
    if ((e = hipMemcpyAsync(d_work, h.work, sizeof(int32_t) * listed, hipMemcpyHostToDevice, stream)) != hipSuccess)
      return hip_fail(e, "hipMemcpyAsync(work)");
    if ((e = hipEventRecord(sim->upload_done, stream)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    if ((e = hipEventSynchronize(sim->upload_done)) != hipSuccess) return hip_fail(e, "hipEventSynchronize");
  }
  char* planes[2][2];
  const rt::SimArgs a = sim_args(sim, trace, out, L, base, planes);
  if (sim->timing) {
    if ((st = collect_timing(sim)) != RT_OK) return st;
    if ((e = hipEventRecord(sim->t0, stream)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  }
  // every class on the caller's stream, dearest first (no internal streams)
  for (int k = 0; k < b.n_act; ++k)
    if ((e = launch_class(b.act[k], a, b, d_work, planes, nullptr, stream)) != hipSuccess)
      return hip_fail(e, "launch(sim)");
  if (sim->timing) {
    if ((e = hipEventRecord(sim->t1, stream)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    sim->timed_pending = true;
  }
  return RT_OK;
}

rt_status rt_goodput(const rt_sim* sim, const rt_trace* trace, const rt_sim_out* out, double* goodput,
                     int64_t* met, void* hip_stream) {
  rt_status st = check_trace(sim, trace, out, "rt_goodput");
  if (st != RT_OK || trace->n_replicas == 0) return st;
  if (!goodput) return fail(RT_EINVAL, "rt_goodput: null goodput");
  DeviceScope ds(sim->device);
  if (ds.err != hipSuccess) return hip_fail(ds.err, "hipSetDevice");
  rt::GoodputArgs a;
  a.points = sim->d_points;
  a.n_points = (int32_t)sim->points.size();
  a.n_requests = trace->n_requests;
  a.n_replicas = trace->n_replicas;
  a.offsets = trace->offsets;
  a.param_point = trace->param_point;
  a.olen = trace->out_len;
  a.cls = trace->slo_class;
  a.ttft = out->ttft_ns;
  a.span = out->decode_span_ns;
  a.goodput = goodput;
  a.met = met;
  a.flag = sim->d_flag;
  hipError_t e = rt::launch_goodput(a, (hipStream_t)hip_stream);
  if (e != hipSuccess) return hip_fail(e, "launch(goodput)");
  return RT_OK;
}

rt_status rt_sim_data_status(rt_sim* sim, void* hip_stream, uint32_t* flags) {
  if (!sim) return fail(RT_EINVAL, "rt_sim_data_status: null sim");
  DeviceScope ds(sim->device);
  if (ds.err != hipSuccess) return hip_fail(ds.err, "hipSetDevice");
  hipStream_t stream = (hipStream_t)hip_stream;
  uint32_t f = 0;
  hipError_t e = hipStreamSynchronize(stream);
  if (e == hipSuccess) e = hipMemcpy(&f, sim->d_flag, sizeof f, hipMemcpyDeviceToHost);
  if (e == hipSuccess && f) e = hipMemset(sim->d_flag, 0, sizeof f);
  if (e != hipSuccess) return hip_fail(e, "rt_sim_data_status");
  if (flags) *flags = f;
  if (f) return fail(RT_EDATA, "rt_sim_data_status: rejected requests (flag word " + std::to_string(f) + ")");
  return RT_OK;
}

rt_status rt_sim_timing(rt_sim* sim, int32_t enable) {
  if (!sim) return fail(RT_EINVAL, "rt_sim_timing: null sim");
  DeviceScope ds(sim->device);
  if (ds.err != hipSuccess) return hip_fail(ds.err, "hipSetDevice");
  hipError_t e;
  if (enable && !sim->t0) {
    if ((e = hipEventCreate(&sim->t0)) != hipSuccess) return hip_fail(e, "hipEventCreate");
    if ((e = hipEventCreate(&sim->t1)) != hipSuccess) return hip_fail(e, "hipEventCreate");
  }
  if (sim->timed_pending) {
    if ((e = hipEventSynchronize(sim->t1)) != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    sim->timed_pending = false;
  }
  sim->timing = enable != 0;
  sim->timed_ms = 0.0;
  sim->timed_calls = 0;
  return RT_OK;
}

rt_status rt_sim_kernel_time(rt_sim* sim, double* total_ms, int64_t* calls) {
  if (!sim) return fail(RT_EINVAL, "rt_sim_kernel_time: null sim");
  DeviceScope ds(sim->device);
  if (ds.err != hipSuccess) return hip_fail(ds.err, "hipSetDevice");
  rt_status st = collect_timing(sim);
  if (st != RT_OK) return st;
  if (total_ms) *total_ms = sim->timed_ms;
  if (calls) *calls = sim->timed_calls;
  return RT_OK;
}

rt_status rt_score_argmin(const rt_router_params* prm, int32_t pool, int32_t n_inst, const float* backlog_s,
                          const int32_t* queue, const int32_t* kv_occ, int32_t kv_cap, int64_t inst_stride,
                          int64_t n_req, const int32_t* prompt_len, const int32_t* pred_out_len,
                          const uint8_t* slo_class, int32_t* out_idx, float* out_score, void* hip_stream) {
  if (!prm) return fail(RT_EINVAL, "rt_score_argmin: null params");
  if (pool != RT_POOL_PREFILL && pool != RT_POOL_DECODE) return fail(RT_EINVAL, "rt_score_argmin: unknown pool");
  if (n_inst < 1) return fail(RT_EINVAL, "rt_score_argmin: n_inst must be >= 1");
  if (n_inst > RT_MAX_POOL) return fail(RT_ERANGE, "rt_score_argmin: n_inst > RT_MAX_POOL");
  if (kv_cap < 1) return fail(RT_EINVAL, "rt_score_argmin: kv_cap must be >= 1");
  if (inst_stride != 0 && inst_stride < n_inst)
    return fail(RT_EINVAL, "rt_score_argmin: inst_stride must be 0 or >= n_inst");
  if (n_req < 0) return fail(RT_EINVAL, "rt_score_argmin: negative n_req");
  const float f[] = {prm->w_b, prm->w_s, prm->w_q, prm->rho, prm->tau_pre_s, prm->tau_dec_s, prm->pre_base_s};
  for (float x : f)
    if (!finite_nonneg(x)) return fail(RT_EINVAL, "rt_score_argmin: weights and prices must be finite and >= 0");
  for (int c = 0; c < RT_MAX_CLASSES; ++c)
    if (!finite_nonneg(prm->sigma[c])) return fail(RT_EINVAL, "rt_score_argmin: sigma must be finite and >= 0");
  if (n_req == 0) return RT_OK;
  if (!backlog_s || !queue || !kv_occ || !prompt_len || !slo_class || !out_idx || !out_score ||
      (pool == RT_POOL_DECODE && !pred_out_len))
    return fail(RT_EINVAL, "rt_score_argmin: null array");
  if (inst_stride != 0 && n_req > INT64_MAX / inst_stride) return fail(RT_ERANGE, "rt_score_argmin: size overflow");
  rt::ScoreArgs a;
  a.w_b = prm->w_b;
  a.w_s = prm->w_s;
  a.w_q = prm->w_q;
  a.rho = prm->rho;
  a.tau = pool == RT_POOL_DECODE ? prm->tau_dec_s : prm->tau_pre_s;
  a.inv_cap = 1.0f / (float)kv_cap;
  for (int c = 0; c < RT_MAX_CLASSES; ++c) a.sigma[c] = prm->sigma[c];
  a.pool = pool;
  a.n_inst = n_inst;
  a.stride = inst_stride;
  a.n_req = n_req;
  a.backlog = backlog_s;
  a.queue = queue;
  a.kv = kv_occ;
  a.plen = prompt_len;
  a.ohat = pred_out_len;
  a.cls = slo_class;
  a.out_idx = out_idx;
  a.out_score = out_score;
  hipError_t e = rt::launch_score(a, (hipStream_t)hip_stream);
  if (e != hipSuccess) return hip_fail(e, "launch(score)");
  return RT_OK;
}

}  // extern "C"
