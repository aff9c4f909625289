// Replica-batched simulation of the learned prefill/decode router under
// continuous batching at the prefill and the decode stage alike, on gfx950.
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
// events per arrival (completions, KV landings); replicas are independent.
// Between two arrivals the prefill instances evolve alone (nothing but
// arrivals feeds them), and each decode instance evolves from its own
// completions and the KV landings that the prefill completions up to that
// arrival scheduled.  So every instance's events up to an arrival can be
// taken prefill pool first, then decode pool, each instance in time order:
// every instance sees the same sequence of events, in the same order and
// with the same arithmetic, as a global time-ordered loop.  Two kernels do
// this: bseg_kernel (below), one replica per segment of S <= 64 lanes and M
// instances per lane in registers (M = 1 for points with P + D <= 64, M = 2
// for pools of up to 128 instances); and bat_kernel, one replica per lane
// walking its instances in turn, for any point.  Batch members and KV
// transfers in flight are sorted rings in scratch, contiguous per instance.
//
// Arithmetic.  Times are float64 ns; every operation matches the written
// model one for one (built with -ffp-contract=off): s = 1 + beta * (b - 1),
// dv = (t - t_last) / s, v += dv, tc = t_last + max(f - v, 0) * s.  The
// batch's remaining stand-alone work is a running total (+ the work of each
// joining member, - b * dv at each clock step, - b * (f - v) when a member
// leaves, 0 once the batch empties), read clamped at 0 as the clock backlog.
// Token totals and the owed decode work of requests not yet joined are exact
// integers in doubles.  The cost equation is the serial kernels' (float32,
// written order).  Outputs round to whole ns, nearest with ties to even.
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

// bat_kernel's lane: its replica's point, request arrays and scratch.  The
// per-instance scalars are structure-of-arrays, element [j * S + lane] (the
// lanes of a wave read one contiguous line per field); entries are 16 bytes.
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
  // (key, r) order: entries after it move one place back.  Returns the
  // position taken, or -1 (and `full`) when the ring has no room.
  template <bool kBatch>
  __device__ int32_t insert(int32_t j, int32_t head, int32_t n, double key, int32_t r) {
    if (n >= C) {
      full = true;
      return -1;
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
    return i;
  }

  // A prefill completion of request r at time tc: the instance lets go of
  // its tokens, TTFT is recorded, the prefill end is kept in the span slot
  // until decode ends, and the KV leaves for the decode instance.
  __device__ void prefill_done(int32_t r, double tc, int32_t& q, double& kv, double& pend) {
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
    if (insert<false>(d, b.whead[k], n, land, r) >= 0) b.nw[k] = n + 1;
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
    double v = b.v[k], tl = b.tl[k], kv = b.kv[k], pend = b.pend[k], left = b.left[k];
    int32_t head = b.head[k], q = b.q[k];
    const double beta = pt.beta_pre;
    while (nact > 0 && !full) {
      Entry e = member(j, head);
      double rem = e.t - v;
      rem = rem < 0.0 ? 0.0 : rem;
      const double tc = tl + rem * slowdown(beta, nact);
      if (tc > now) break;
      left = left - (double)nact * (e.t - v);
      v = e.t;
      tl = tc;
      tmax = fmax(tmax, tc);
      for (;;) {
        prefill_done(e.r, tc, q, kv, pend);
        ++head;
        --nact;
        if (nact == 0) break;
        e = member(j, head);
        if (e.t != v) break;
      }
      if (nact == 0) left = 0.0;
    }
    if (now < kInf) {
      if (nact > 0) {
        const double dv = (now - tl) / slowdown(beta, nact);
        v = v + dv;
        left = left - (double)nact * dv;
      }
      tl = now;
    }
    b.v[k] = v;
    b.left[k] = left;
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
    double v = b.v[k], tl = b.tl[k], kv = b.kv[k], pend = b.pend[k], owed = b.owed[k], left = b.left[k];
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
        left = left - (double)nact * (e.t - v);
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
        if (nact == 0) left = 0.0;
      } else {
        if (tj > now) break;
        const int32_t r = transfer(j, wh).r;
        ++wh;
        --nw;
        if (nact > 0) {
          const double dv = (tj - tl) / slowdown(beta, nact);
          v = v + dv;
          left = left - (double)nact * dv;
        }
        tl = tj;
        const double w = work_dec(a.olen[lo + r]);
        owed = owed - w;
        if (insert<true>(j, head, nact, v + w, r) >= 0) {
          ++nact;
          left = left + w;
        }
      }
    }
    if (now < kInf) {
      if (nact > 0) {
        const double dv = (now - tl) / slowdown(beta, nact);
        v = v + dv;
        left = left - (double)nact * dv;
      }
      tl = now;
    }
    b.v[k] = v;
    b.left[k] = left;
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

  // Clock backlog of instance j in seconds: the batch's running remaining
  // work (clamped at 0), then the owed work of requests not yet joined.
  __device__ float owed_s(int32_t j) {
    const int64_t k = at(j);
    const double left = b.left[k];
    double w = left < 0.0 ? 0.0 : left;
    w = w + b.owed[k];
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

// lpw: replicas per wave (lanes 0 .. lpw - 1 of every wave hold one each,
// the others return at once).  The kernel waits on memory, so a launch of
// few replicas spreads them over more waves rather than filling each wave.
__global__ __launch_bounds__(kBlock) void bat_kernel(SimArgs a, BatScratch b, int32_t lpw) {
  const int32_t wl = (int32_t)(threadIdx.x & 63);
  if (wl >= lpw) return;
  const int64_t lane = ((int64_t)blockIdx.x * kBlock + threadIdx.x) / 64 * lpw + wl;
  if (lane >= a.n_work) return;
  const int32_t rep = a.work[lane];
  const int64_t lo = a.offsets[rep], hi = a.offsets[rep + 1];
  const DevPoint& pt = a.points[a.param_point ? a.param_point[rep] : 0];
  Lane L{a, b, pt, lane, lo, nullptr, nullptr, pt.P, pt.D, b.C, 0.0, false};
  L.ring = reinterpret_cast<Entry*>(b.ring) + lane * b.NI * (int64_t)b.C;
  L.wring = reinterpret_cast<Entry*>(b.wring) + lane * b.NI * (int64_t)b.C;
  for (int32_t j = 0; j < L.P + L.D; ++j) {
    const int64_t k = L.at(j);
    b.v[k] = b.tl[k] = b.kv[k] = b.pend[k] = b.owed[k] = b.left[k] = 0.0;
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
      const double w = L.work_pre(p);
      if (L.insert<true>(ip, b.head[k], n, b.v[k] + w, rl) < 0) break;
      b.nact[k] = n + 1;
      b.left[k] = b.left[k] + w;
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


// ---------------------------------------------------------------------------
// Segment variant: one replica per aligned segment of S lanes of a wave, one
// instance per lane (prefill instances on lanes [0, P), decode instances on
// [P, P + D)), as in the serial segment kernels.  A lane's instance state and
// the front entries of its rings (with the front request's data) live in its
// registers; the rings behind the fronts are the lane's own scratch.  Every
// step (one request of every segment's replica) runs wave-uniform rounds:
// prefill rounds, in each of which every prefill lane whose front completes
// by the arrival lets it go and the decode lanes of the segment take the
// departing KV transfers from it (read with cross-lane shuffles); decode
// rounds, in each of which every decode lane takes its next event (a
// completion, or a KV landing joining its batch); then every instance's clock
// is brought to the arrival, every lane scores its instance, the two argmins
// are DPP reductions over the segment, and the chosen lanes admit.  A round
// pops one member per lane: members with equal finish virtual times leave in
// consecutive rounds at the same time, with the same arithmetic as leaving
// together (the remaining work they see is 0).
struct RingTail {
  double t;
  int32_t r;
};

// Insert (key, r) into a ring of n entries from head: appended when it
// follows the cached tail, else entries after it move back one place.
// Returns the position taken, or -1 (and `full`) when the ring has no room.
__device__ __forceinline__ int32_t ring_put(Entry* rg, int32_t C, int32_t head, int32_t n, double key, int32_t r,
                                            RingTail& tail, bool& full) {
  if (n >= C) {
    full = true;
    return -1;
  }
  int32_t i = head + n;
  if (n == 0 || tail.t < key || (tail.t == key && tail.r < r)) {
    Entry& d = rg[i & (C - 1)];
    d.t = key;
    d.r = r;
    tail.t = key;
    tail.r = r;
    return i;
  }
  while (i > head) {
    const Entry e = rg[(i - 1) & (C - 1)];
    if (!(e.t > key || (e.t == key && e.r > r))) break;
    rg[i & (C - 1)] = e;
    --i;
  }
  Entry& d = rg[i & (C - 1)];
  d.t = key;
  d.r = r;
  return i;
}

// The first two entries of a ring, kept in registers: the front (valid when
// the ring holds one entry or more) and the one behind it (two or more), so
// that a departure needs no load before the next event time is known.
struct Window {
  double k0, k1;
  int32_t r0, r1;
};

// After inserting (key, r) at position `at` of a ring whose head is `head`.
__device__ __forceinline__ void window_put(Window& w, int32_t at, int32_t head, double key, int32_t r) {
  const bool front = at == head, second = at == head + 1;
  w.k1 = front ? w.k0 : (second ? key : w.k1);
  w.r1 = front ? w.r0 : (second ? r : w.r1);
  w.k0 = front ? key : w.k0;
  w.r0 = front ? r : w.r0;
}

// After the front left a ring (head already advanced, n entries left): the
// second becomes the front and the new second is loaded.
__device__ __forceinline__ void window_pop(Window& w, const Entry* rg, int32_t C, int32_t head, int32_t n) {
  w.k0 = w.k1;
  w.r0 = w.r1;
  if (n > 1) {
    const Entry e = rg[(head + 1) & (C - 1)];
    w.k1 = e.t;
    w.r1 = e.r;
  }
}

// One request's data, loaded a step ahead.
struct Req {
  int64_t arr;
  int32_t p, o, oh;
  uint32_t c;
  uint4 ws;
};

// One instance of the segment kernel, in registers (a lane holds M): the
// batch's state, the first two entries of its rings with the front
// requests' data, and the rings' cached tails.
struct BInst {
  double v, tl, left, kv, pend, owed;
  int32_t q, nact, head, nw, wh;
  // the batch's window and its front request's data (prefill: arrival, p,
  // o, o^, decode instance; decode: prefill end, p, o, o^)
  Window bw;
  double x0;
  int32_t p0, o0, oh0, dst0;
  // the transfers' window (decode) and the front transfer's data
  Window tw;
  double pf1;
  int32_t p1, o1, oh1;
  RingTail btail, wtail;
};

__device__ __forceinline__ void init_binst(BInst& x) {
  x.v = x.tl = x.left = x.kv = x.pend = x.owed = 0.0;
  x.q = x.nact = x.head = x.nw = x.wh = 0;
  x.bw = Window{0.0, 0.0, 0, 0};
  x.x0 = 0.0;
  x.p0 = x.o0 = x.oh0 = x.dst0 = 0;
  x.tw = Window{0.0, 0.0, 0, 0};
  x.pf1 = 0.0;
  x.p1 = x.o1 = x.oh1 = 0;
  x.btail = RingTail{0.0, 0};
  x.wtail = RingTail{0.0, 0};
}

// kMinBlocks: workgroups per compute unit the register budget must allow
// (1: as many registers as the kernel wants, for launches whose waves do not
// fill the GPU; 3 (M = 1) or 2 (M = 2): three or two waves per SIMD, for
// launches with many waves).  M: instances per lane (prefill instance j on
// lane j / M, slot j % M; decode instance d on lane ceil(P / M) + d / M,
// slot d % M).  A round takes at most one event of every instance, slot
// after slot; the state of every slot stays in registers (about 46 each).
template <int S, int kMinBlocks, int M>
__global__ __launch_bounds__(kBlock, kMinBlocks) void bseg_kernel(SimArgs a, BatScratch b) {
  const int lane = (int)(threadIdx.x & 63);
  const int64_t gl = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  const int sl = lane & (S - 1);
  const int base = lane & ~(S - 1);
  const int64_t seg = gl / S;
  const bool has = seg < a.n_work;
  const int32_t rep = has ? a.work[seg] : 0;
  const int64_t lo = has ? a.offsets[rep] : 0;
  const int64_t len = has ? a.offsets[rep + 1] - lo : 0;
  const DevPoint& pt = a.points[(has && a.param_point) ? a.param_point[rep] : 0];
  const int32_t P = pt.P, D = pt.D;
  const int32_t LP = (P + M - 1) / M, LD = (D + M - 1) / M;  // lanes holding each pool
  const bool isP = has && sl < LP;
  const bool isD = has && sl >= LP && sl < LP + LD;
  const int32_t j0 = (isP ? sl : sl - LP) * M;  // the lane's first instance in its pool
  bool ok[M];                                    // slot m holds an instance
#pragma unroll
  for (int m = 0; m < M; ++m) ok[m] = (isP && j0 + m < P) || (isD && j0 + m < D);
  const double beta = isP ? pt.beta_pre : pt.beta_dec;
  const double xfer = (double)pt.xfer_tok_ns;
  const bool samp = pt.policy == kPolicyLearnedSampled;
  // The point's parameters, read once: the loop's stores could alias them,
  // so reads inside it would be repeated, each with a wait for every memory
  // access still outstanding.
  const int32_t ncls = pt.n_classes, pol = pt.policy, len_thr = pt.len_thr, bmode = pt.mode;
  const float w_b = pt.w_b, w_s = pt.w_s, w_q = pt.w_q, rho = pt.rho;
  const float tau_pre = pt.tau_pre, tau_dec = pt.tau_dec, pre_base = pt.pre_base;
  const float inv = isP ? pt.inv_cap_pre : pt.inv_cap_dec;
  const double pre_base_ns = (double)pt.pre_base_ns, pre_tok_ns = (double)pt.pre_tok_ns;
  const double dec_tok_ns = (double)pt.dec_tok_ns;
  // sigma per class of each segment's point (LDS)
  __shared__ float sig[(kBlock / S) * kMaxClasses];
  const int sblk = (int)(threadIdx.x / S);
  for (int k = sl; k < kMaxClasses; k += S) sig[sblk * kMaxClasses + k] = pt.sigma[k];
  __syncthreads();
  const int32_t C = b.C;
  // the rings of slot m: batch members and KV transfers in flight
  Entry* rings[M];
  Entry* wrings[M];
#pragma unroll
  for (int m = 0; m < M; ++m) {
    rings[m] = reinterpret_cast<Entry*>(b.ring) + (gl * M + m) * (int64_t)C;
    wrings[m] = reinterpret_cast<Entry*>(b.wring) + (gl * M + m) * (int64_t)C;
  }

  BInst in[M];
#pragma unroll
  for (int m = 0; m < M; ++m) init_binst(in[m]);
  double tmax = 0.0;
  bool rej = false, full = false, dead = false;
  int64_t last = -1;

  // The data of a batch's new front (needed only when it leaves).
  auto front_data = [&](BInst& x) __attribute__((always_inline)) {
    const int64_t g = lo + x.bw.r0;
    x.p0 = a.plen[g];
    x.o0 = a.olen[g];
    x.oh0 = a.ohat[g];
    if (isP) {
      x.x0 = i64_to_f64(a.arrival[g]);
      x.dst0 = a.i_dec[g];
    } else {
      x.x0 = __longlong_as_double(a.span[g]);
    }
  };
  auto transfer_data = [&](BInst& x) __attribute__((always_inline)) {
    const int64_t g = lo + x.tw.r0;
    x.p1 = a.plen[g];
    x.o1 = a.olen[g];
    x.oh1 = a.ohat[g];
    x.pf1 = __longlong_as_double(a.span[g]);
  };

  // Every event at or before `now` (prefill rounds, then decode rounds).
  auto run_to = [&](double now) {
    // one prefill round; false when no lane had an event
    auto pre_round = [&]() -> bool {
      bool fire[M];
      uint64_t fm[M];
      uint64_t any = 0;
      double land[M], ftl[M], tcs[M];
      int32_t fr[M], fd[M], fp[M], fo[M], foh[M];
      static_for<M>([&](auto mc) __attribute__((always_inline)) {
        constexpr int m = decltype(mc)::value;
        const BInst& x = in[m];
        double tc = kInf;
        if (x.nact > 0) {
          double rem = x.bw.k0 - x.v;
          rem = rem < 0.0 ? 0.0 : rem;
          tc = x.tl + rem * slowdown(beta, x.nact);
        }
        tcs[m] = tc;
        fire[m] = isP && !dead && x.nact > 0 && tc <= now;
        fm[m] = __ballot(fire[m]);
        any |= fm[m];
      });
      if (any == 0) return false;
      static_for<M>([&](auto mc) __attribute__((always_inline)) {
        constexpr int m = decltype(mc)::value;
        BInst& x = in[m];
        const double tc = tcs[m];
        land[m] = 0.0;
        fr[m] = fd[m] = fp[m] = fo[m] = foh[m] = 0;
        if (fire[m]) {
          x.left = x.left - (double)x.nact * (x.bw.k0 - x.v);
          x.v = x.bw.k0;
          x.tl = tc;
          tmax = fmax(tmax, tc);
          const int64_t g = lo + x.bw.r0;
          x.q -= 1;
          x.kv = x.kv - (double)x.p0;
          x.pend = x.pend - (double)x.p0;
          a.ttft[g] = round_ns(tc - x.x0);
          a.span[g] = __double_as_longlong(tc);
          land[m] = tc + (double)x.p0 * xfer;
          tmax = fmax(tmax, land[m]);
          fr[m] = x.bw.r0;
          fd[m] = x.dst0;
          fp[m] = x.p0;
          fo[m] = x.o0;
          foh[m] = x.oh0;
          x.head += 1;
          x.nact -= 1;
          if (x.nact == 0) {
            x.left = 0.0;
          } else {
            window_pop(x.bw, rings[m], C, x.head, x.nact);
            front_data(x);
          }
        }
        ftl[m] = x.tl;
      });
      // the departing transfers go to their decode instances: every position
      // (within the segments) that fired somewhere in the wave is read by
      // every lane from its own segment, slot by slot
      static_for<M>([&](auto mc) __attribute__((always_inline)) {
        constexpr int m = decltype(mc)::value;
        uint64_t rel = 0;
#pragma unroll
        for (int s0 = 0; s0 < 64; s0 += S) rel |= (S == 64) ? fm[m] : ((fm[m] >> s0) & ((1ull << (S & 63)) - 1ull));
        while (rel) {
          const int i = __ffsll((unsigned long long)rel) - 1;
          rel &= rel - 1;
          const int src = base + i;
          const bool fi = __shfl((int)fire[m], src) != 0;
          const int32_t di = __shfl(fd[m], src);
          const double li = __shfl(land[m], src);
          const double ti = __shfl(ftl[m], src);
          const int32_t ri = __shfl(fr[m], src), pi = __shfl(fp[m], src), oi = __shfl(fo[m], src),
                        ohi = __shfl(foh[m], src);
          static_for<M>([&](auto nc) __attribute__((always_inline)) {
            constexpr int mm = decltype(nc)::value;
            BInst& y = in[mm];
            if (isD && fi && di == j0 + mm) {
              const int32_t at = ring_put(wrings[mm], C, y.wh, y.nw, li, ri, y.wtail, full);
              if (at >= 0) {
                window_put(y.tw, at, y.wh, li, ri);
                if (at == y.wh) {
                  y.pf1 = ti;
                  y.p1 = pi;
                  y.o1 = oi;
                  y.oh1 = ohi;
                }
                y.nw += 1;
              }
            }
          });
        }
      });
      return true;
    };
    // two rounds per loop trip (measured: 8 % faster on a 4,096-replica cluster,
    // 15 % on 65,536 replicas, than one)
    while (pre_round() && pre_round()) {
    }
    // one decode round; false when no lane had an event
    auto dec_round = [&]() -> bool {
      bool anyf = false;
      static_for<M>([&](auto mc) __attribute__((always_inline)) {
        constexpr int m = decltype(mc)::value;
        BInst& x = in[m];
        double tc = kInf, tj = kInf;
        if (x.nact > 0) {
          double rem = x.bw.k0 - x.v;
          rem = rem < 0.0 ? 0.0 : rem;
          tc = x.tl + rem * slowdown(beta, x.nact);
        }
        if (x.nw > 0) tj = x.tw.k0;
        const bool fire = isD && !dead && (x.nact > 0 || x.nw > 0) && (tc <= tj ? tc : tj) <= now;
        anyf = anyf || fire;
        if (!fire) return;
        if (tc <= tj) {
          x.left = x.left - (double)x.nact * (x.bw.k0 - x.v);
          x.v = x.bw.k0;
          x.tl = tc;
          tmax = fmax(tmax, tc);
          const int64_t g = lo + x.bw.r0;
          x.q -= 1;
          x.kv = x.kv - ((double)x.p0 + (double)x.o0);
          x.pend = x.pend - (double)x.oh0;
          a.span[g] = round_ns(tc - x.x0);
          x.head += 1;
          x.nact -= 1;
          if (x.nact == 0) {
            x.left = 0.0;
          } else {
            window_pop(x.bw, rings[m], C, x.head, x.nact);
            front_data(x);
          }
        } else {
          const int32_t r = x.tw.r0, pr = x.p1, orr = x.o1, ohr = x.oh1;
          const double pfr = x.pf1;
          x.wh += 1;
          x.nw -= 1;
          if (x.nw > 0) {
            window_pop(x.tw, wrings[m], C, x.wh, x.nw);
            transfer_data(x);
          }
          if (x.nact > 0) {
            const double dv = (tj - x.tl) / slowdown(beta, x.nact);
            x.v = x.v + dv;
            x.left = x.left - (double)x.nact * dv;
          }
          x.tl = tj;
          const double w = (double)(orr - 1) * dec_tok_ns;
          x.owed = x.owed - w;
          const double f = x.v + w;
          const int32_t at = ring_put(rings[m], C, x.head, x.nact, f, r, x.btail, full);
          if (at >= 0) {
            window_put(x.bw, at, x.head, f, r);
            if (at == x.head) {
              x.x0 = pfr;
              x.p0 = pr;
              x.o0 = orr;
              x.oh0 = ohr;
            }
            x.nact += 1;
            x.left = x.left + w;
          }
        }
      });
      return __any(anyf);
    };
    while (dec_round()) {
    }
  };

  auto fetch = [&](int32_t t) {
    Req q0{0, 1, 1, 1, 0u, make_uint4(0u, 0u, 0u, 0u)};
    if (t < len) {
      const int64_t g = lo + t;
      q0.arr = a.arrival[g];
      q0.p = a.plen[g];
      q0.o = a.olen[g];
      q0.oh = a.ohat[g];
      q0.c = a.cls[g];
      if (samp) q0.ws = *reinterpret_cast<const uint4*>(a.samp + 4 * g);
    }
    return q0;
  };

  const int32_t Rmax = wave_max_nonneg((int32_t)len);
  Req nx = fetch(0);
  for (int32_t t = 0; t < Rmax; ++t) {
    // request t, loaded a step ahead; request t + 1 is loaded now
    const Req cur = nx;
    nx = fetch(t + 1);
    const int64_t arr = cur.arr;
    const int32_t p = cur.p, o = cur.o, oh = cur.oh;
    const uint32_t c = cur.c;
    const uint4 ws = cur.ws;
    const bool mine = t < len && !dead;
    const int64_t g = lo + t;
    const bool valid = mine && p >= 1 && o >= 1 && oh >= 1 && (int64_t)p + o <= INT32_MAX &&
                       (int64_t)p + oh <= INT32_MAX && (int32_t)c < ncls && arr >= 0 && arr >= last;
    if (mine && !valid) {
      rej = true;
      if (sl == 0) {
        a.i_pre[g] = a.i_dec[g] = -1;
        a.ttft[g] = a.span[g] = -1;
      }
    }
    const double now = valid ? i64_to_f64(arr) : -1.0;
    if (valid) {
      last = arr;
      tmax = fmax(tmax, now);
    }
    run_to(now);
    // The rounds end on every lane at once, but the compiler may represent
    // their loops with per-lane exits and reuse a lane-mask compare made
    // inside them (where it has no bits for lanes it considers gone) after
    // them; passing the counts through opaque() makes every later test of
    // them a fresh compare.
#pragma unroll
    for (int m = 0; m < M; ++m) {
      in[m].nact = opaque(in[m].nact);
      in[m].nw = opaque(in[m].nw);
    }
    // every instance's clock to the arrival
    if (valid && (isP || isD)) {
      static_for<M>([&](auto mc) __attribute__((always_inline)) {
        constexpr int m = decltype(mc)::value;
        BInst& x = in[m];
        if (x.nact > 0) {
          const double dv = (now - x.tl) / slowdown(beta, x.nact);
          x.v = x.v + dv;
          x.left = x.left - (double)x.nact * dv;
        }
        x.tl = now;
      });
    }
    // each lane's key: the lowest of its instances' (lowest slot on equal
    // keys; 0xffffffff: not offered)
    uint32_t bkey = 0xffffffffu;
    int32_t bm = 0;
    if (valid && (isP || isD)) {
      const int32_t n = isP ? P : D;
      uint32_t c1 = 0, c2 = 0;
      if (pol == kPolicyLearnedSampled) {
        const uint32_t u = isP ? ws.x : ws.z, w2 = isP ? ws.y : ws.w;
        c1 = __umulhi(u, (uint32_t)n);
        const uint32_t x = __umulhi(w2, (uint32_t)(n - 1));
        c2 = n > 1 ? x + (x >= c1 ? 1u : 0u) : c1;
      }
      static_for<M>([&](auto mc) __attribute__((always_inline)) {
        constexpr int m = decltype(mc)::value;
        const BInst& x = in[m];
        const int32_t jj = j0 + m;
        uint32_t key;
        if (pol == kPolicyRoundRobin) {
          key = jj == t % n ? 0u : 1u;
        } else if (pol == kPolicyLeastLoaded) {
          key = (uint32_t)x.q;
        } else if (pol == kPolicyLengthThreshold) {
          const bool part = isP || n == 1 || ((jj >= (n + 1) / 2) == (oh >= len_thr));
          key = part ? (uint32_t)x.q : 0xffffffffu;
        } else {
          const float sg = sig[sblk * kMaxClasses + (int)(c & (kMaxClasses - 1))];
          const float work = isP ? w_s * (float)p * tau_pre : w_s * (float)oh * tau_dec;
          const double need = isP ? (double)p : (double)p + (double)oh;
          float bl;
          if (bmode == 0) {
            double w = x.left < 0.0 ? 0.0 : x.left;
            w = w + x.owed;
            bl = (float)w * 1e-9f;
          } else if (isP) {
            bl = tau_pre * (float)x.pend + pre_base * (float)x.q;
          } else {
            bl = tau_dec * (float)x.pend;
          }
          const float press = (float)(x.kv + need) * inv;
          const float load = w_b * bl * sg;
          const float size = work * (1.0f + rho * press) * sg;
          key = cost_key(load + size + w_q * (float)x.q);
          if (pol == kPolicyLearnedSampled) key = ((uint32_t)jj == c1 || (uint32_t)jj == c2) ? key : 0xffffffffu;
        }
        key = ok[m] ? key : 0xffffffffu;
        if (m == 0) {
          bkey = key;
        } else {
          const bool lower = key < bkey;
          bkey = lower ? key : bkey;
          bm = lower ? m : bm;
        }
      });
    }
    uint32_t kp = isP ? bkey : 0xffffffffu, kd = isD ? bkey : 0xffffffffu;
    const uint32_t kp0 = kp, kd0 = kd;
    seg_min2<S>(kp, kd);
    const int32_t wp = seg_first<S>(isP && kp0 == kp, lane);  // winning lanes
    const int32_t wd = seg_first<S>(isD && kd0 == kd, lane);
    int32_t mp = 0, md = 0;  // winning slots
    if constexpr (M > 1) {
      mp = (int32_t)seg_or<S>(sl == wp ? (uint32_t)bm : 0u);
      md = (int32_t)seg_or<S>(sl == wd ? (uint32_t)bm : 0u);
    }
    const int32_t ip = wp * M + mp;
    const int32_t id = (wd - LP) * M + md;
    if (valid) {
      if (sl == 0) {
        a.i_pre[g] = ip;
        a.i_dec[g] = id;
      }
      static_for<M>([&](auto mc) __attribute__((always_inline)) {
        constexpr int m = decltype(mc)::value;
        BInst& x = in[m];
        if (isP && sl == wp && m == mp) {
          const double w = pre_base_ns + (double)p * pre_tok_ns;
          const double f = x.v + w;
          const int32_t at = ring_put(rings[m], C, x.head, x.nact, f, t, x.btail, full);
          if (at >= 0) {
            window_put(x.bw, at, x.head, f, t);
            if (at == x.head) {
              x.x0 = now;
              x.p0 = p;
              x.o0 = o;
              x.oh0 = oh;
              x.dst0 = id;
            }
            x.nact += 1;
            x.q += 1;
            x.kv = x.kv + (double)p;
            x.pend = x.pend + (double)p;
            x.left = x.left + w;
          }
        }
        if (isD && sl == wd && m == md) {
          x.owed = x.owed + (double)(o - 1) * dec_tok_ns;
          x.q += 1;
          x.kv = x.kv + ((double)p + (double)o);
          x.pend = x.pend + (double)oh;
        }
      });
    }
    // a replica whose ring overflowed stops (its outputs are not valid)
    dead = seg_or<S>(full ? 1u : 0u) != 0;
  }
  run_to(kInf);
  const uint32_t flag = (tmax >= kTimeLimit ? kFlagTimeRange : 0u) | (rej ? kFlagRejected : 0u) |
                        (full ? kFlagBatchCap : 0u);
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
  double** d[] = {&b.v, &b.tl, &b.kv, &b.pend, &b.owed, &b.left};
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

// Replicas per wave of the one-replica-per-lane kernel.
static int32_t bat_lanes_per_wave(int64_t n_work) {
  int32_t lpw = 1;
  while (lpw < 64 && (int64_t)lpw * 1024 < n_work) lpw *= 2;
  return lpw;
}

hipError_t launch_bat(const SimClass& c, const SimArgs& a, const BatScratch& b, hipStream_t stream) {
  if (a.n_work <= 0) return hipSuccess;
  const int64_t lanes = a.n_work * (int64_t)c.S;
  const dim3 grid((unsigned)((lanes + bat::kBlock - 1) / bat::kBlock)), block(bat::kBlock);
  // with at least two waves per SIMD to place, occupancy pays more than
  // registers do; two instances per lane fit two waves per SIMD without
  // spilling, three spill (measured on 16,384 replicas of 8 + 64 instances:
  // two waves 27.5 ms, three 51.3 ms)
  const bool many = lanes >= 2 * 64 * 1024;
#define RT_BSEG_CASE(S_, M_)                                                              \
  if (c.MP == M_ && c.S == S_) {                                                          \
    if (many)                                                                             \
      hipLaunchKernelGGL((bat::bseg_kernel<S_, M_ == 1 ? 3 : 2, M_>), grid, block, 0, stream, a, b);  \
    else                                                                                  \
      hipLaunchKernelGGL((bat::bseg_kernel<S_, 1, M_>), grid, block, 0, stream, a, b);    \
    return hipGetLastError();                                                             \
  }
  RT_BSEG_FOR_EACH(RT_BSEG_CASE)
#undef RT_BSEG_CASE
  // one replica per lane: replicas per wave a power of two, at most 64, so
  // that the launch has about one wave per SIMD (1,024) where it can
  // (measured on 16,384 replicas of 72 instances: 64 per wave 270 ms, 16
  // per wave 203 ms, 8 per wave 210 ms, 4 per wave 333 ms)
  const int32_t lpw = bat_lanes_per_wave(a.n_work);
  const int64_t waves = (a.n_work + lpw - 1) / lpw;
  const dim3 wgrid((unsigned)((waves * 64 + bat::kBlock - 1) / bat::kBlock));
  hipLaunchKernelGGL(bat::bat_kernel, wgrid, block, 0, stream, a, b, lpw);
  return hipGetLastError();
}

// Lanes a launch of class c over n_work replicas spans (the scratch owners;
// the one-replica-per-lane kernel numbers its replicas densely, so n_work of
// them fit).
int64_t bat_lanes(const SimClass& c, int64_t n_work) {
  const int64_t lanes = n_work * (int64_t)c.S;
  return (lanes + bat::kBlock - 1) / bat::kBlock * bat::kBlock;
}

}  // namespace rt
