// Host side of the rt_router C ABI (include/rt_router.h): argument checks,
// launch planning, scratch ownership and error reporting.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
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
  if (c.kind == rt::kBat) return c.MP == 0 || p.n_prefill + p.n_decode <= c.S;
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
  if ((st = read_plan_inputs(sim, trace, stream, off, pp, "rt_sim_run_replicas")) != RT_OK) return st;

  // Plan.  Each point runs one kernel class.  With few replicas (fewer
  // waves, at the shortest-step classes, than twice the GPU's SIMDs) every
  // replica is a latency chain and takes the shortest-step class; with many,
  // the GPU's issue rate is the limit and each point takes the segment class
  // with the fewest issue slots per replica-step (lanes x step cost).  Then
  // replicas are bucketed by class, longest first so that long chains start
  // early; empty replicas need no work.
  const int ncls = rt::sim_class_count();
  const int64_t n = trace->n_replicas;
  const size_t npts = sim->points.size();
  std::vector<int64_t> reps_of(npts, 0);
  for (int64_t i = 0; i < n; ++i)
    if (off[i + 1] > off[i]) reps_of[pp[i]] += 1;
  for (size_t k = 0; k < npts; ++k)
    if (reps_of[k] > 0 && sim->points[k].policy == RT_POLICY_LEARNED_SAMPLED && !trace->sample_bits)
      return fail(RT_EINVAL, "rt_sim_run_replicas: point " + std::to_string(k) +
                                 " samples candidates but trace->sample_bits is NULL");
  double waves = 0.0;
  for (size_t k = 0; k < npts; ++k) waves += (double)reps_of[k] * rt::sim_class(sim->point_classes[k][0]).S / 64.0;
  const bool many = waves >= 2.0 * kSimds;
  std::vector<int> choice(npts);
  for (size_t k = 0; k < npts; ++k) {
    const std::vector<int>& fit = sim->point_classes[k];
    choice[k] = fit[0];
    if (!many) continue;
    double best = -1.0;
    for (int c : fit) {
      const rt::SimClass sc = rt::sim_class(c);
      if (sc.kind != rt::kSeg) continue;
      const double cost = sc.S * seg_step_cost(sc);
      if (best < 0.0 || cost < best) {
        best = cost;
        choice[k] = c;
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
      std::vector<int> wider(choice);
      double w2 = 0.0, w1 = 0.0;
      for (size_t k = 0; k < npts; ++k) {
        if (reps_of[k] == 0) continue;
        const rt::SimClass sc = rt::sim_class(choice[k]);
        w1 += std::ceil((double)reps_of[k] * sc.S / 64.0);
        if ((sc.kind == rt::kSeg || sc.kind == rt::kBat) && sc.MP == 1 && sc.S < 64)
          for (int c : sim->point_classes[k]) {
            const rt::SimClass wc = rt::sim_class(c);
            if (wc.kind == sc.kind && wc.mode == sc.mode && wc.MP == 1 && wc.S == 2 * sc.S) wider[k] = c;
          }
        w2 += std::ceil((double)reps_of[k] * rt::sim_class(wider[k]).S / 64.0);
      }
      if (!(w2 > w1 && w2 <= kSimds)) break;
      choice.swap(wider);
    }
  }
  std::vector<std::vector<int32_t>> buckets(ncls);
  for (int64_t i = 0; i < n; ++i)
    if (off[i + 1] > off[i]) buckets[choice[pp[i]]].push_back((int32_t)i);
  for (auto& b : buckets)
    std::stable_sort(b.begin(), b.end(), [&](int32_t x, int32_t y) {
      return off[x + 1] - off[x] > off[y + 1] - off[y];
    });

  hipError_t e;
  // Scratch of the serial classes: for each record size in use (32 bytes,
  // or 64 for the classes that price the ledger) a plane per pool, each its
  // dummy records followed by one record per request, 256-byte aligned.
  // Classes of one call run side by side, so each size has planes of its own.
  bool any_serial = false, any_ledger = false, any_plain = false;
  std::vector<int> bat_classes;
  for (int c = 0; c < ncls; ++c) {
    if (buckets[c].empty()) continue;
    if (rt::sim_class(c).kind == rt::kBat) {
      bat_classes.push_back(c);
    } else {
      any_serial = true;
      (rt::mode_ledger(rt::sim_class(c).mode) ? any_ledger : any_plain) = true;
    }
  }
  const size_t nreq = (size_t)trace->n_requests;
  static_assert(((size_t)rt::kDummyRecords << rt::rec_shift(false)) % 256 == 0, "planes start 256-byte aligned");
  auto plane_bytes = [&](bool ledger) {
    return (((nreq + rt::kDummyRecords) << rt::rec_shift(ledger)) + 255) / 256 * 256;
  };
  const size_t plain_plane = any_plain ? plane_bytes(false) : 0, ledger_plane = any_ledger ? plane_bytes(true) : 0;
  const size_t need = any_serial ? 2 * plain_plane + 2 * ledger_plane + 256 : 0;
  if (need > sim->scratch_bytes) {
    if ((e = hipDeviceSynchronize()) != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
    if (sim->d_scratch) (void)hipFree(sim->d_scratch);
    sim->d_scratch = nullptr;
    sim->scratch_bytes = 0;
    if ((e = hipMalloc(&sim->d_scratch, need)) != hipSuccess) return hip_fail(e, "hipMalloc(scratch)");
    sim->scratch_bytes = need;
  }
  // Scratch of the batched classes: per-instance state and two rings per
  // instance for every lane of each, sized by the largest pool and capacity
  // among that class's replicas' points; one allocation, carved in turn.
  std::vector<rt::BatScratch> bs(ncls);
  if (!bat_classes.empty()) {
    struct Dim {
      int64_t S;
      int32_t NI, C;
    };
    std::vector<Dim> dims;
    size_t bneed = 256;
    for (int c : bat_classes) {
      int32_t NI = 1, C = 2;
      for (int32_t r : buckets[c]) {
        const rt_point& q = sim->points[pp[r]];
        NI = std::max(NI, q.n_prefill + q.n_decode);
        C = std::max(C, q.batch_cap == 0 ? kDefaultBatchCap : q.batch_cap);
      }
      const rt::SimClass sc = rt::sim_class(c);
      if (sc.MP == 1) NI = 1;  // a segment class: one instance per lane
      dims.push_back(Dim{rt::bat_lanes(sc, (int64_t)buckets[c].size()), NI, C});
      bneed += rt::bat_scratch_bytes(dims.back().S, NI, C);
    }
    if (bneed > sim->bscratch_bytes) {
      if ((e = hipDeviceSynchronize()) != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
      if (sim->d_bscratch) (void)hipFree(sim->d_bscratch);
      sim->d_bscratch = nullptr;
      sim->bscratch_bytes = 0;
      if ((e = hipMalloc(&sim->d_bscratch, bneed)) != hipSuccess) return hip_fail(e, "hipMalloc(batched scratch)");
      sim->bscratch_bytes = bneed;
    }
    size_t at = 0;
    for (size_t k = 0; k < bat_classes.size(); ++k) {
      bs[bat_classes[k]] = rt::bat_scratch_carve(sim->d_bscratch + at, dims[k].S, dims[k].NI, dims[k].C);
      at += rt::bat_scratch_bytes(dims[k].S, dims[k].NI, dims[k].C);
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
  size_t pos = 0;
  std::vector<size_t> start(ncls);
  for (int c = 0; c < ncls; ++c) {
    start[c] = pos;
    std::copy(buckets[c].begin(), buckets[c].end(), sim->h_work + pos);
    pos += buckets[c].size();
  }
  if (pos > 0) {
    if ((e = hipMemcpyAsync(sim->d_work, sim->h_work, sizeof(int32_t) * pos, hipMemcpyHostToDevice, stream)) !=
        hipSuccess)
      return hip_fail(e, "hipMemcpyAsync(work)");
    if ((e = hipEventRecord(sim->upload_done, stream)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    sim->upload_pending = true;
  }

  char* sc = sim->d_scratch;
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
  // record planes by record size: index 0 of each pool's plane
  char* rec_planes[2][2] = {{nullptr, nullptr}, {nullptr, nullptr}};
  for (int k = 0; k < 2 && sc; ++k) {
    if (any_plain) rec_planes[0][k] = sc + k * plain_plane + ((size_t)rt::kDummyRecords << rt::rec_shift(false));
    if (any_ledger)
      rec_planes[1][k] = sc + 2 * plain_plane + k * ledger_plane + ((size_t)rt::kDummyRecords << rt::rec_shift(true));
  }
  a.rec[0] = a.rec[1] = nullptr;
  a.flag = sim->d_flag;
  if (sim->timing) {
    if ((st = collect_timing(sim)) != RT_OK) return st;
    if ((e = hipEventRecord(sim->t0, stream)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  }
  // Kernel classes with work, largest first; more than one run side by side
  // on internal streams forked from and joined back into `stream`.
  std::vector<int> act;
  std::vector<double> cost(ncls, 0.0);
  for (int c = 0; c < ncls; ++c) {
    if (buckets[c].empty()) continue;
    act.push_back(c);
    for (int32_t r : buckets[c]) cost[c] += (double)(off[r + 1] - off[r]) * rt::sim_class(c).S;
  }
  std::stable_sort(act.begin(), act.end(), [&](int x, int y) { return cost[x] > cost[y]; });
  if (act.size() > 1) {
    while (sim->lanes.size() < act.size()) {
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
  for (size_t k = 0; k < act.size(); ++k) {
    const int c = act[k];
    a.work = sim->d_work + start[c];
    a.n_work = (int64_t)buckets[c].size();
    const int lg = rt::mode_ledger(rt::sim_class(c).mode) ? 1 : 0;
    a.rec[0] = rec_planes[lg][0];
    a.rec[1] = rec_planes[lg][1];
    hipStream_t where = stream;
    if (act.size() > 1) {
      where = sim->lanes[k];
      if ((e = hipStreamWaitEvent(where, sim->fork, 0)) != hipSuccess) return hip_fail(e, "hipStreamWaitEvent");
    }
    e = rt::sim_class(c).kind == rt::kBat ? rt::launch_bat(rt::sim_class(c), a, bs[c], where)
                                          : rt::launch_sim(rt::sim_class(c), a, where);
    if (e != hipSuccess) return hip_fail(e, "launch(sim)");
    if (act.size() > 1 && (e = hipEventRecord(sim->joins[k], where)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  }
  // The joins go in after every launch: streams share the device's few
  // hardware queues, and a wait enqueued between two launches could hold
  // back a later launch that landed on the same queue.
  if (act.size() > 1)
    for (size_t k = 0; k < act.size(); ++k)
      if ((e = hipStreamWaitEvent(stream, sim->joins[k], 0)) != hipSuccess) return hip_fail(e, "hipStreamWaitEvent");
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
