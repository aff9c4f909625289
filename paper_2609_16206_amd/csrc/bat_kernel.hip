// Replica-batched simulation of the learned prefill/decode router under
// continuous batching in both stages, on gfx950.
//
// Model (the service model Section VI adds to the serial one; routing is
// Algorithm 1 with the Section III-A cost equation, unchanged): every
// instance serves all its admitted requests at once; while b requests share
// an instance each receives stand-alone service at 1 / (1 + beta (b - 1)) of
// full speed, and leaves once it has received its stand-alone work (its
// serial service time).  A request joins its prefill instance's batch at its
// arrival and its decode instance's batch when its KV lands there.  Each
// instance keeps a virtual clock v, valid at time t_last, counting the
// stand-alone service every member has received; a member leaves when v
// reaches its finish virtual time f (v at joining + its work), so the
// members kept sorted by (f, request) leave from the front, and the next
// completion lies at t_last + max(f_front - v, 0) (1 + beta (b - 1)).
//
// Mapping.  A replica is a chain of events with a data-dependent number of
// events per arrival (completions, KV landings), and replicas are
// independent: one replica per lane.  Between two arrivals the prefill
// instances evolve alone (nothing but arrivals feeds them) and each decode
// instance evolves from its own completions and the KV landings that the
// prefill completions up to that arrival scheduled, so a lane processes each
// prefill instance's events up to the arrival, then each decode instance's;
// every instance sees the same sequence of events, in the same order and
// with the same arithmetic, as a global time-ordered loop.  Per-instance
// scalars are structure-of-arrays (the lanes of a wave read one contiguous
// line per field); batch members and KV transfers in flight are sorted rings
// of 16-byte entries, contiguous per lane, so the walk over a batch (the
// backlog sum, an insertion) stays within a few cache lines.
//
// Arithmetic.  Times are float64 ns; every operation matches the written
// model one for one (built with -ffp-contract=off): s = 1 + beta * (b - 1),
// v += (t - t_last) / s, tc = t_last + max(f - v, 0) * s.  Token totals and
// the owed decode work of requests not yet joined are exact integers in
// doubles.  The cost equation is the serial kernels' (float32, written
// order).  Outputs round to whole ns, nearest with ties to even.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "lane_ops.h"
#include "rt_internal.h"

namespace rt {
namespace bat {

constexpr double kInf = __builtin_huge_val();
constexpr int kBlock = 256;

struct alignas(16) Entry {
  double t;   // finish virtual time (batch) or landing time (transfer)
  int32_t r;  // request index within the replica
  int32_t pad;
};

__device__ __forceinline__ double slowdown(double beta, int32_t b) { return 1.0 + beta * (double)(b - 1); }

// Nearest integer of a double in [0, 2^52), ties to even, as an int64.
__device__ __forceinline__ int64_t round_ns(double x) { return f64_to_i64(__builtin_rint(x)); }

// One lane's replica: its point, its request arrays and its scratch.
struct Lane {
  const SimArgs& a;
  const BatScratch& b;
  const DevPoint& pt;
  int64_t lane;
  int64_t lo;        // global index of the replica's request 0
  Entry* ring;       // this lane's batch rings, instance j at ring + j * C
  Entry* wring;      // this lane's transfer rings
  int32_t P, D, C;
  double tmax;       // largest time reached
  bool full;         // a ring would overflow: the replica stops

  __device__ int64_t at(int32_t j) const { return (int64_t)j * b.S + lane; }
  __device__ Entry& member(int32_t j, int32_t pos) { return ring[(int64_t)j * C + (pos & (C - 1))]; }
  __device__ Entry& transfer(int32_t j, int32_t pos) { return wring[(int64_t)j * C + (pos & (C - 1))]; }

  __device__ double work_pre(int32_t p) const { return (double)pt.pre_base_ns + (double)p * (double)pt.pre_tok_ns; }
  __device__ double work_dec(int32_t o) const { return (double)(o - 1) * (double)pt.dec_tok_ns; }

  // Insert (key, r) into a ring of n entries starting at head, keeping
  // (key, r) order: entries after it move one place back.
  template <bool kBatch>
  __device__ bool insert(int32_t j, int32_t head, int32_t n, double key, int32_t r) {
    if (n >= C) {
      full = true;
      return false;
    }
    int32_t i = head + n;
    while (i > head) {
      Entry e = kBatch ? member(j, i - 1) : transfer(j, i - 1);
      if (!(e.t > key || (e.t == key && e.r > r))) break;
      (kBatch ? member(j, i) : transfer(j, i)) = e;
      --i;
    }
    Entry& d = kBatch ? member(j, i) : transfer(j, i);
    d.t = key;
    d.r = r;
    return true;
  }

  // A prefill completion of request r at time tc: the instance lets go of
  // its tokens, TTFT is recorded, the prefill end is kept in the span slot
  // until decode ends, and the KV leaves for the decode instance.
  __device__ void prefill_done(int32_t j, int32_t r, double tc, int32_t& q, double& kv, double& pend) {
    const int64_t g = lo + r;
    const int32_t p = a.plen[g];
    q -= 1;
    kv = kv - (double)p;
    pend = pend - (double)p;
    a.ttft[g] = round_ns(tc - i64_to_f64(a.arrival[g]));
    a.span[g] = __double_as_longlong(tc);
    const int32_t d = P + a.i_dec[g];
    const double land = tc + (double)p * (double)pt.xfer_tok_ns;
    tmax = fmax(tmax, land);
    const int64_t k = at(d);
    const int32_t n = b.nw[k];
    if (insert<false>(d, b.whead[k], n, land, r)) b.nw[k] = n + 1;
  }

  __device__ void decode_done(int32_t r, double tc, int32_t& q, double& kv, double& pend) {
    const int64_t g = lo + r;
    const int32_t p = a.plen[g], o = a.olen[g], oh = a.ohat[g];
    q -= 1;
    kv = kv - ((double)p + (double)o);
    pend = pend - (double)oh;
    a.span[g] = round_ns(tc - __longlong_as_double(a.span[g]));
  }

  // Every event of prefill instance j at or before `now` in time order; then
  // its clock is brought to `now` (unless now is +inf: the final drain).
  __device__ void run_prefill(int32_t j, double now) {
    const int64_t k = at(j);
    int32_t nact = b.nact[k];
    if (nact == 0) {
      if (now < kInf) b.tl[k] = now;
      return;
    }
    double v = b.v[k], tl = b.tl[k], kv = b.kv[k], pend = b.pend[k];
    int32_t head = b.head[k], q = b.q[k];
    const double beta = pt.beta_pre;
    while (nact > 0 && !full) {
      Entry e = member(j, head);
      double rem = e.t - v;
      rem = rem < 0.0 ? 0.0 : rem;
      const double tc = tl + rem * slowdown(beta, nact);
      if (tc > now) break;
      v = e.t;
      tl = tc;
      tmax = fmax(tmax, tc);
      for (;;) {
        prefill_done(j, e.r, tc, q, kv, pend);
        ++head;
        --nact;
        if (nact == 0) break;
        e = member(j, head);
        if (e.t != v) break;
      }
    }
    if (now < kInf) {
      if (nact > 0) v += (now - tl) / slowdown(beta, nact);
      tl = now;
    }
    b.v[k] = v;
    b.tl[k] = tl;
    b.kv[k] = kv;
    b.pend[k] = pend;
    b.head[k] = head;
    b.q[k] = q;
    b.nact[k] = nact;
  }

  // The same for decode instance d: its completions and the KV landings
  // queued for it (a completion first at equal times).
  __device__ void run_decode(int32_t d, double now) {
    const int32_t j = P + d;
    const int64_t k = at(j);
    int32_t nact = b.nact[k], nw = b.nw[k];
    if (nact == 0 && nw == 0) {
      if (now < kInf) b.tl[k] = now;
      return;
    }
    double v = b.v[k], tl = b.tl[k], kv = b.kv[k], pend = b.pend[k], owed = b.owed[k];
    int32_t head = b.head[k], q = b.q[k], wh = b.whead[k];
    const double beta = pt.beta_dec;
    while (!full) {
      double tc = kInf;
      Entry e{};
      if (nact > 0) {
        e = member(j, head);
        double rem = e.t - v;
        rem = rem < 0.0 ? 0.0 : rem;
        tc = tl + rem * slowdown(beta, nact);
      }
      const double tj = nw > 0 ? transfer(j, wh).t : kInf;
      if (nact == 0 && nw == 0) break;
      if (tc <= tj) {
        if (tc > now) break;
        v = e.t;
        tl = tc;
        tmax = fmax(tmax, tc);
        for (;;) {
          decode_done(e.r, tc, q, kv, pend);
          ++head;
          --nact;
          if (nact == 0) break;
          e = member(j, head);
          if (e.t != v) break;
        }
      } else {
        if (tj > now) break;
        const int32_t r = transfer(j, wh).r;
        ++wh;
        --nw;
        if (nact > 0) v += (tj - tl) / slowdown(beta, nact);
        tl = tj;
        const double w = work_dec(a.olen[lo + r]);
        owed = owed - w;
        if (insert<true>(j, head, nact, v + w, r)) ++nact;
      }
    }
    if (now < kInf) {
      if (nact > 0) v += (now - tl) / slowdown(beta, nact);
      tl = now;
    }
    b.v[k] = v;
    b.tl[k] = tl;
    b.kv[k] = kv;
    b.pend[k] = pend;
    b.owed[k] = owed;
    b.head[k] = head;
    b.q[k] = q;
    b.nact[k] = nact;
    b.whead[k] = wh;
    b.nw[k] = nw;
  }

  __device__ void run_to(double now) {
    for (int32_t j = 0; j < P && !full; ++j) run_prefill(j, now);
    for (int32_t d = 0; d < D && !full; ++d) run_decode(d, now);
  }

  // Clock backlog of instance j in seconds: the batch's remaining virtual
  // work in member order, then the owed work of requests not yet joined.
  __device__ float owed_s(int32_t j) {
    const int64_t k = at(j);
    const int32_t nact = b.nact[k], head = b.head[k];
    const double v = b.v[k];
    double w = 0.0;
    for (int32_t i = 0; i < nact; ++i) {
      const double rem = member(j, head + i).t - v;
      w += rem < 0.0 ? 0.0 : rem;
    }
    w += b.owed[k];
    return (float)w * 1e-9f;
  }

  // The cost equation for instance j (pool-relative index jj) of one pool.
  __device__ uint32_t cost_key_of(bool isp, int32_t j, float work, double need, float sg, float inv) {
    const int64_t k = at(j);
    const int32_t q = b.q[k];
    float bl;
    if (pt.mode == 0)
      bl = owed_s(j);
    else if (isp)
      bl = pt.tau_pre * (float)b.pend[k] + pt.pre_base * (float)q;
    else
      bl = pt.tau_dec * (float)b.pend[k];
    const float press = (float)(b.kv[k] + need) * inv;
    const float load = pt.w_b * bl * sg;
    const float size = work * (1.0f + pt.rho * press) * sg;
    return cost_key(load + size + pt.w_q * (float)q);
  }

  // Each pool's choice for request r (local index rl), as in the serial
  // kernels: round robin, least loaded (within the length part), the
  // learned argmin, or the learned argmin over two sampled candidates.
  __device__ int32_t choose(bool isp, int32_t rl, int32_t p, int32_t oh, uint32_t c, uint32_t u, uint32_t w) {
    const int32_t n = isp ? P : D;
    const int32_t base = isp ? 0 : P;
    const int32_t pol = pt.policy;
    if (pol == kPolicyRoundRobin) return rl % n;
    if (pol == kPolicyLeastLoaded || pol == kPolicyLengthThreshold) {
      int32_t lo_j = 0, hi_j = n;
      if (pol == kPolicyLengthThreshold && !isp && n > 1) {
        const int32_t half = (n + 1) / 2;
        if (oh >= pt.len_thr)
          lo_j = half;
        else
          hi_j = half;
      }
      int32_t best = lo_j, bq = b.q[at(base + lo_j)];
      for (int32_t j = lo_j + 1; j < hi_j; ++j) {
        const int32_t qj = b.q[at(base + j)];
        if (qj < bq) {
          bq = qj;
          best = j;
        }
      }
      return best;
    }
    const float sg = pt.sigma[c];
    const float work = isp ? pt.w_s * (float)p * pt.tau_pre : pt.w_s * (float)oh * pt.tau_dec;
    const double need = isp ? (double)p : (double)p + (double)oh;
    const float inv = isp ? pt.inv_cap_pre : pt.inv_cap_dec;
    if (pol == kPolicyLearnedSampled) {
      const uint32_t c1 = __umulhi(u, (uint32_t)n);
      const uint32_t x = __umulhi(w, (uint32_t)(n - 1));
      const uint32_t c2 = n > 1 ? x + (x >= c1 ? 1u : 0u) : c1;
      const int32_t j0 = (int32_t)min(c1, c2), j1 = (int32_t)max(c1, c2);
      const uint32_t k0 = cost_key_of(isp, base + j0, work, need, sg, inv);
      if (j1 == j0) return j0;
      const uint32_t k1 = cost_key_of(isp, base + j1, work, need, sg, inv);
      return k1 < k0 ? j1 : j0;
    }
    int32_t best = 0;
    uint32_t bk = cost_key_of(isp, base, work, need, sg, inv);
    for (int32_t j = 1; j < n; ++j) {
      const uint32_t kj = cost_key_of(isp, base + j, work, need, sg, inv);
      if (kj < bk) {
        bk = kj;
        best = j;
      }
    }
    return best;
  }
};

__global__ __launch_bounds__(kBlock) void bat_kernel(SimArgs a, BatScratch b) {
  const int64_t lane = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (lane >= a.n_work) return;
  const int32_t rep = a.work[lane];
  const int64_t lo = a.offsets[rep], hi = a.offsets[rep + 1];
  const DevPoint& pt = a.points[a.param_point ? a.param_point[rep] : 0];
  Lane L{a, b, pt, lane, lo, nullptr, nullptr, pt.P, pt.D, b.C, 0.0, false};
  L.ring = reinterpret_cast<Entry*>(b.ring) + lane * b.NI * (int64_t)b.C;
  L.wring = reinterpret_cast<Entry*>(b.wring) + lane * b.NI * (int64_t)b.C;
  for (int32_t j = 0; j < L.P + L.D; ++j) {
    const int64_t k = L.at(j);
    b.v[k] = b.tl[k] = b.kv[k] = b.pend[k] = b.owed[k] = 0.0;
    b.q[k] = b.nact[k] = b.head[k] = b.nw[k] = b.whead[k] = 0;
  }
  bool rej = false;
  int64_t last = -1;
  const int32_t ncls = pt.n_classes;
  for (int64_t g = lo; g < hi && !L.full; ++g) {
    const int64_t arr = a.arrival[g];
    const int32_t p = a.plen[g], o = a.olen[g], oh = a.ohat[g];
    const uint32_t c = a.cls[g];
    const bool ok = p >= 1 && o >= 1 && oh >= 1 && (int64_t)p + o <= INT32_MAX && (int64_t)p + oh <= INT32_MAX &&
                    (int32_t)c < ncls && arr >= 0 && arr >= last;
    if (!ok) {
      a.i_pre[g] = a.i_dec[g] = -1;
      a.ttft[g] = a.span[g] = -1;
      rej = true;
      continue;
    }
    last = arr;
    const double now = i64_to_f64(arr);
    L.tmax = fmax(L.tmax, now);
    L.run_to(now);
    if (L.full) break;
    const int32_t rl = (int32_t)(g - lo);
    uint32_t w0 = 0, w1 = 0, w2 = 0, w3 = 0;
    if (pt.policy == kPolicyLearnedSampled) {
      const uint4 ws = *reinterpret_cast<const uint4*>(a.samp + 4 * g);
      w0 = ws.x;
      w1 = ws.y;
      w2 = ws.z;
      w3 = ws.w;
    }
    const int32_t ip = L.choose(true, rl, p, oh, c, w0, w1);
    const int32_t id = L.choose(false, rl, p, oh, c, w2, w3);
    a.i_pre[g] = ip;
    a.i_dec[g] = id;
    // admission: the prefill batch takes the request now; the decode
    // instance holds its tokens from now and takes it into its batch when
    // its KV lands
    {
      const int64_t k = L.at(ip);
      const int32_t n = b.nact[k];
      if (!L.insert<true>(ip, b.head[k], n, b.v[k] + L.work_pre(p), rl)) break;
      b.nact[k] = n + 1;
      b.q[k] += 1;
      b.kv[k] = b.kv[k] + (double)p;
      b.pend[k] = b.pend[k] + (double)p;
    }
    {
      const int64_t k = L.at(L.P + id);
      b.owed[k] = b.owed[k] + L.work_dec(o);
      b.q[k] += 1;
      b.kv[k] = b.kv[k] + ((double)p + (double)o);
      b.pend[k] = b.pend[k] + (double)oh;
    }
  }
  if (!L.full) L.run_to(kInf);
  const uint32_t flag = (L.tmax >= kTimeLimit ? kFlagTimeRange : 0u) | (rej ? kFlagRejected : 0u) |
                        (L.full ? kFlagBatchCap : 0u);
  if (flag) atomicOr(a.flag, flag);
}

}  // namespace bat

// One allocation, 256-byte aligned arrays: the ten state arrays, then the
// two ring blocks.  With base == nullptr only the size is computed.
static size_t carve(char* base, int64_t S, int32_t NI, int32_t C, BatScratch* out) {
  const size_t state = (size_t)S * NI;
  auto align = [](size_t x) { return (x + 255) & ~(size_t)255; };
  size_t off = 0;
  BatScratch b{};
  double** d[] = {&b.v, &b.tl, &b.kv, &b.pend, &b.owed};
  for (double** x : d) {
    *x = reinterpret_cast<double*>(base + off);
    off = align(off + state * sizeof(double));
  }
  int32_t** i[] = {&b.q, &b.nact, &b.head, &b.nw, &b.whead};
  for (int32_t** x : i) {
    *x = reinterpret_cast<int32_t*>(base + off);
    off = align(off + state * sizeof(int32_t));
  }
  b.ring = base + off;
  off = align(off + state * (size_t)C * sizeof(bat::Entry));
  b.wring = base + off;
  off = align(off + state * (size_t)C * sizeof(bat::Entry));
  b.S = S;
  b.NI = NI;
  b.C = C;
  if (out) *out = b;
  return off;
}

size_t bat_scratch_bytes(int64_t S, int32_t NI, int32_t C) { return carve(nullptr, S, NI, C, nullptr); }

BatScratch bat_scratch_carve(char* base, int64_t S, int32_t NI, int32_t C) {
  BatScratch b{};
  carve(base, S, NI, C, &b);
  return b;
}

hipError_t launch_bat(const SimArgs& a, const BatScratch& b, hipStream_t stream) {
  if (a.n_work <= 0) return hipSuccess;
  const int64_t blocks = (a.n_work + bat::kBlock - 1) / bat::kBlock;
  hipLaunchKernelGGL(bat::bat_kernel, dim3((unsigned)blocks), dim3(bat::kBlock), 0, stream, a, b);
  return hipGetLastError();
}

}  // namespace rt
