/*
 * Plain sequential CPU oracle: see rt_oracle.h for the contract.
 *
 * TEST INFRASTRUCTURE ONLY (tests, the smoke check and the CPU-baseline leg
 * of the benchmark).  Written for clarity, not speed: one request at a time,
 * every instance scored from scratch, one growable FIFO array per instance.
 */
#include "rt_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* The cost equation (Section III-A)                                         */
/* ------------------------------------------------------------------------ */

/* Ordering of costs for the argmin: smaller first, both zeros equal, NaN
 * after +inf.  Costs are non-negative whenever the weights are, so the IEEE
 * bit pattern of a positive float orders like its value. */
static uint32_t cost_key(float c) {
  uint32_t u;
  if (c != c) return 0x7fc00000u;
  if (c == 0.0f) return 0u;
  memcpy(&u, &c, sizeof u);
  return u;
}

/* cost = w_b * backlog * sigma  +  work * (1 + rho * press+) * sigma  +  w_q * queue
 * with work = w_s * (request tokens) * tau, press+ = (occupancy + k) / cap.
 * C evaluates each product and sum left to right in float32, which is the
 * written order of the equation. */
static float cost_eq(const orc_router* rp, float backlog_s, float work, float sg, int64_t kv_occ,
                     int64_t k, float inv_cap, int64_t queue) {
  float press = (float)(kv_occ + k) * inv_cap;
  float load = rp->w_b * backlog_s * sg;
  float size = work * (1.0f + rp->rho * press) * sg;
  return load + size + rp->w_q * (float)queue;
}

/* Per-request priced work of a pool: prompt tokens at the prefill price
 * (Section III-A prices prefill candidates like decode ones, with p_r tau_pre
 * in place of the decode work), predicted output tokens at the decode
 * price. */
static float pool_work(const orc_router* rp, int32_t pool, int32_t p, int32_t ohat) {
  if (pool == ORC_PREFILL) return rp->w_s * (float)p * rp->tau_pre_s;
  return rp->w_s * (float)ohat * rp->tau_dec_s;
}

/* Tokens the request adds to an instance's cache if admitted there. */
static int64_t pool_need(int32_t pool, int32_t p, int32_t ohat) {
  return pool == ORC_PREFILL ? (int64_t)p : (int64_t)p + (int64_t)ohat;
}

void orc_candidates(uint32_t u, uint32_t v, int32_t n, int32_t* c1, int32_t* c2) {
  const uint64_t first = ((uint64_t)u * (uint64_t)n) >> 32;
  *c1 = (int32_t)first;
  if (n < 2) {
    *c2 = *c1;
    return;
  }
  /* the v-th of the n - 1 instances other than the first, in index order */
  const uint64_t k = ((uint64_t)v * (uint64_t)(n - 1)) >> 32;
  *c2 = (int32_t)(k < first ? k : k + 1);
}

int orc_score(const orc_router* rp, int32_t pool, int32_t n_inst, const float* backlog_s,
              const int32_t* queue, const int32_t* kv_occ, int64_t kv_cap, int64_t inst_stride,
              int64_t n_req, const int32_t* prompt_len, const int32_t* pred_out_len,
              const uint8_t* slo_class, const uint32_t* sample_bits, int32_t* out_idx, float* out_score,
              float* out_second) {
  if (!rp || n_inst < 1 || n_req < 0 || kv_cap < 1 || (pool != ORC_PREFILL && pool != ORC_DECODE))
    return -1;
  if (n_req > 0 && (!backlog_s || !queue || !kv_occ || !prompt_len || !pred_out_len || !slo_class ||
                    !out_idx || !out_score))
    return -1;
  if (inst_stride != 0 && inst_stride < n_inst) return -1;
  const float inv_cap = 1.0f / (float)kv_cap;
  for (int64_t i = 0; i < n_req; ++i) {
    const int32_t p = prompt_len[i], oh = pred_out_len[i];
    const uint8_t c = slo_class[i];
    if (p < 1 || c >= ORC_MAX_CLASSES ||
        (pool == ORC_DECODE && (oh < 1 || (int64_t)p + oh > INT32_MAX))) {
      out_idx[i] = -1;
      out_score[i] = NAN;
      if (out_second) out_second[i] = NAN;
      continue;
    }
    const float sg = rp->sigma[c];
    const float work = pool_work(rp, pool, p, oh);
    const int64_t k = pool_need(pool, p, oh);
    const int64_t row = i * inst_stride;
    int32_t best = -1;
    float best_c = 0.0f, second_c = INFINITY;
    int32_t c1 = -1, c2 = -1;
    if (sample_bits) orc_candidates(sample_bits[2 * i], sample_bits[2 * i + 1], n_inst, &c1, &c2);
    for (int32_t j = 0; j < n_inst; ++j) {
      if (sample_bits && j != c1 && j != c2) continue; /* not offered */
      float c_j = cost_eq(rp, backlog_s[row + j], work, sg, kv_occ[row + j], k, inv_cap, queue[row + j]);
      if (best < 0 || cost_key(c_j) < cost_key(best_c)) {
        if (best >= 0) second_c = best_c;
        best = j;
        best_c = c_j;
      } else if (cost_key(c_j) < cost_key(second_c)) {
        second_c = c_j;
      }
    }
    out_idx[i] = best;
    out_score[i] = best_c;
    if (out_second) out_second[i] = second_c;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Replica simulation (Algorithm 1 per admission; Section III-D and          */
/* Section VI serial-service model)                                          */
/* ------------------------------------------------------------------------ */

typedef struct {
  int64_t busy;  /* time the instance finishes everything admitted so far */
  int64_t queue; /* admitted and not yet finished                         */
  int64_t kv;    /* cache tokens held by those requests                   */
  int64_t pend;  /* tokens the router's ledger still prices for them      */
  /* FIFO of in-flight requests in admission order: release time, cache
   * tokens and priced tokens of each; entries [head, size) are in flight. */
  int64_t *t_rel, *fp, *pt;
  int64_t head, size, cap;
} inst_t;

static int push(inst_t* s, int64_t t_rel, int64_t fp, int64_t pt) {
  if (s->size == s->cap) {
    int64_t nc = s->cap ? 2 * s->cap : 16;
    int64_t* a = (int64_t*)realloc(s->t_rel, (size_t)nc * sizeof(int64_t));
    if (!a) return -1;
    s->t_rel = a;
    a = (int64_t*)realloc(s->fp, (size_t)nc * sizeof(int64_t));
    if (!a) return -1;
    s->fp = a;
    a = (int64_t*)realloc(s->pt, (size_t)nc * sizeof(int64_t));
    if (!a) return -1;
    s->pt = a;
    s->cap = nc;
  }
  s->t_rel[s->size] = t_rel;
  s->fp[s->size] = fp;
  s->pt[s->size] = pt;
  s->size++;
  s->queue += 1;
  s->kv += fp;
  s->pend += pt;
  return 0;
}

/* Remove every request whose service has ended by `now` (a release at
 * exactly `now` happens before the arrival at `now` is routed). */
static int64_t retire(inst_t* s, int64_t now, int64_t* violations) {
  int64_t popped = 0;
  while (s->head < s->size && s->t_rel[s->head] <= now) {
    s->queue -= 1;
    s->kv -= s->fp[s->head];
    s->pend -= s->pt[s->head];
    s->head++;
    popped++;
    if (s->queue < 0 || s->kv < 0 || s->pend < 0) (*violations)++;
  }
  return popped;
}

static void free_pool(inst_t* a, int32_t n) {
  if (!a) return;
  for (int32_t j = 0; j < n; ++j) {
    free(a[j].t_rel);
    free(a[j].fp);
    free(a[j].pt);
  }
  free(a);
}

/* backlog(d) as Section III-A defines it (the work the instance has already
 * taken on, in seconds).  True mode reads the
 * simulation clock (busy-until minus now); proxy mode prices the in-flight
 * ledger with the router's own constants (Section VI). */
/* The proxy's ledger backlog of an instance with `queue` requests and `pend`
 * priced tokens in flight (the same in both service models). */
static float ledger_backlog(const orc_point* pt, int32_t pool, int64_t queue, int64_t pend) {
  const orc_router* rp = &pt->router;
  if (pool == ORC_PREFILL) return rp->tau_pre_s * (float)pend + rp->pre_base_s * (float)queue;
  return rp->tau_dec_s * (float)pend;
}

static float backlog_of(const orc_point* pt, int32_t pool, const inst_t* s, int64_t now) {
  if (pt->backlog_mode == ORC_BACKLOG_TRUE) {
    int64_t d = s->busy - now;
    if (d < 0) d = 0;
    return (float)d * 1e-9f;
  }
  return ledger_backlog(pt, pool, s->queue, s->pend);
}

/* Own choice for one pool from its instances' features (backlog in
 * seconds, requests in flight, cache tokens held).  Returns the argmin over
 * the offered instances (every instance, or under the sampled policy the two
 * candidates drawn from `words`, returned in cand[]); fills cost[] (learned
 * policies only) and reports whether the best two offered costs are equal or
 * within tie_rel. */
static int32_t choose(const orc_point* pt, int32_t pool, int32_t n, int64_t r, const float* backlog,
                      const int64_t* queue, const int64_t* kv, int32_t p, int32_t ohat, uint8_t c,
                      const uint32_t* words, double tie_rel, float* cost, int32_t* cand, int* tie, int* close) {
  *tie = 0;
  *close = 0;
  cand[0] = cand[1] = -1;
  if (pt->policy == ORC_ROUND_ROBIN) return (int32_t)(r % n);
  if (pt->policy == ORC_LEAST_LOADED || pt->policy == ORC_LENGTH_THRESHOLD) {
    /* the part of the pool this request may use: everything, except under
     * the threshold policy on the decode pool, where long predicted outputs
     * take the upper half and the others the lower half */
    int32_t lo = 0, hi = n;
    if (pt->policy == ORC_LENGTH_THRESHOLD && pool == ORC_DECODE && n > 1) {
      const int32_t half = (n + 1) / 2;
      if (ohat >= pt->len_threshold) lo = half;
      else hi = half;
    }
    int32_t b = lo;
    for (int32_t j = lo + 1; j < hi; ++j)
      if (queue[j] < queue[b]) b = j;
    return b;
  }
  const orc_router* rp = &pt->router;
  const float sg = rp->sigma[c];
  const float work = pool_work(rp, pool, p, ohat);
  const int64_t k = pool_need(pool, p, ohat);
  const int64_t cap = pool == ORC_PREFILL ? pt->kv_cap_pre : pt->kv_cap_dec;
  const float inv_cap = 1.0f / (float)cap;
  const int sampled = pt->policy == ORC_LEARNED_SAMPLED;
  if (sampled) orc_candidates(words[0], words[1], n, &cand[0], &cand[1]);
  int32_t b = -1, b2 = -1;
  for (int32_t j = 0; j < n; ++j) {
    cost[j] = cost_eq(rp, backlog[j], work, sg, kv[j], k, inv_cap, queue[j]);
    if (sampled && j != cand[0] && j != cand[1]) continue; /* not offered */
    if (b < 0) {
      b = j;
    } else if (cost_key(cost[j]) < cost_key(cost[b])) {
      b2 = b;
      b = j;
    } else if (b2 < 0 || cost_key(cost[j]) < cost_key(cost[b2])) {
      b2 = j;
    }
  }
  if (b2 >= 0) {
    if (cost_key(cost[b2]) == cost_key(cost[b]))
      *tie = 1;
    else if ((double)cost[b2] - (double)cost[b] <= tie_rel * fabs((double)cost[b]))
      *close = 1;
  }
  return b;
}

/* The serial model's features of one pool at time `now`. */
static void serial_features(const orc_point* pt, int32_t pool, const inst_t* inst, int32_t n, int64_t now,
                            float* backlog, int64_t* queue, int64_t* kv) {
  for (int32_t j = 0; j < n; ++j) {
    backlog[j] = backlog_of(pt, pool, &inst[j], now);
    queue[j] = inst[j].queue;
    kv[j] = inst[j].kv;
  }
}

/* Adopt an external placement g in place of the own choice m. */
static int32_t follow(const orc_point* pt, int32_t m, int32_t g, int32_t n, const float* cost,
                      const int32_t* cand, double tie_rel, int64_t* near_tie, int64_t* mismatch, int64_t* first,
                      int64_t r) {
  if (g == m) return m;
  int ok = 0;
  const int offered = pt->policy == ORC_LEARNED || (pt->policy == ORC_LEARNED_SAMPLED && (g == cand[0] || g == cand[1]));
  if (g >= 0 && g < n && offered) {
    double gap = (double)cost[g] - (double)cost[m];
    ok = gap <= tie_rel * fabs((double)cost[m]);
  }
  if (ok) {
    (*near_tie)++;
  } else {
    (*mismatch)++;
    if (*first < 0) *first = r;
  }
  return (g >= 0 && g < n) ? g : m;
}

int orc_sim_replica(const orc_point* pt, int64_t n, const int64_t* arrival_ns,
                    const int32_t* prompt_len, const int32_t* out_len,
                    const int32_t* pred_out_len, const uint8_t* slo_class, const uint32_t* sample_bits,
                    const int32_t* follow_pre, const int32_t* follow_dec, double tie_rel,
                    int32_t* i_pre, int32_t* i_dec, int64_t* ttft_ns, int64_t* span_ns,
                    orc_stats* st) {
  if (!pt || !st || n < 0) return -1;
  if (pt->n_prefill < 1 || pt->n_decode < 1 || pt->n_classes < 1 ||
      pt->n_classes > ORC_MAX_CLASSES || pt->kv_cap_pre < 1 || pt->kv_cap_dec < 1)
    return -1;
  if (pt->policy == ORC_LENGTH_THRESHOLD && pt->len_threshold < 1) return -1;
  if (n > 0 && (!arrival_ns || !prompt_len || !out_len || !pred_out_len || !slo_class || !i_pre ||
                !i_dec || !ttft_ns || !span_ns))
    return -1;
  if (pt->policy == ORC_LEARNED_SAMPLED && n > 0 && !sample_bits) return -1;
  memset(st, 0, sizeof *st);
  st->first_mismatch = -1;
  const int32_t P = pt->n_prefill, D = pt->n_decode;
  inst_t* pre = (inst_t*)calloc((size_t)P, sizeof(inst_t));
  inst_t* dec = (inst_t*)calloc((size_t)D, sizeof(inst_t));
  float* cost_pre = (float*)calloc((size_t)P, sizeof(float));
  float* cost_dec = (float*)calloc((size_t)D, sizeof(float));
  const int32_t N = P > D ? P : D;
  float* f_backlog = (float*)calloc((size_t)N, sizeof(float));
  int64_t* f_queue = (int64_t*)calloc((size_t)N, sizeof(int64_t));
  int64_t* f_kv = (int64_t*)calloc((size_t)N, sizeof(int64_t));
  int rc = 0;
  if (!pre || !dec || !cost_pre || !cost_dec || !f_backlog || !f_queue || !f_kv) {
    rc = -2;
    goto done;
  }

  int64_t last_arrival = 0;
  int have_arrival = 0;
  for (int64_t r = 0; r < n; ++r) {
    const int64_t now = arrival_ns[r];
    const int32_t p = prompt_len[r], o = out_len[r], oh = pred_out_len[r];
    const uint8_t c = slo_class[r];
    /* Data checks: a rejected request is not routed and leaves no state. */
    if (p < 1 || o < 1 || oh < 1 || (int64_t)p + o > INT32_MAX || (int64_t)p + oh > INT32_MAX ||
        c >= pt->n_classes || now < 0 || (have_arrival && now < last_arrival)) {
      st->invalid++;
      i_pre[r] = i_dec[r] = -1;
      ttft_ns[r] = span_ns[r] = -1;
      continue;
    }
    last_arrival = now;
    have_arrival = 1;

    /* 1. completions up to now leave both pools. */
    for (int32_t j = 0; j < P; ++j) st->retired_pre += retire(&pre[j], now, &st->violations);
    for (int32_t j = 0; j < D; ++j) st->retired_dec += retire(&dec[j], now, &st->violations);

    /* 2. argmin of each pool, computed independently on the same state. */
    int tie, close;
    int32_t cand_pre[2], cand_dec[2];
    const uint32_t* w = sample_bits ? sample_bits + 4 * r : NULL;
    serial_features(pt, ORC_PREFILL, pre, P, now, f_backlog, f_queue, f_kv);
    int32_t ip = choose(pt, ORC_PREFILL, P, r, f_backlog, f_queue, f_kv, p, oh, c, w, tie_rel, cost_pre, cand_pre,
                        &tie, &close);
    st->tie_pre += tie;
    st->close_pre += close;
    serial_features(pt, ORC_DECODE, dec, D, now, f_backlog, f_queue, f_kv);
    int32_t id = choose(pt, ORC_DECODE, D, r, f_backlog, f_queue, f_kv, p, oh, c, w ? w + 2 : NULL, tie_rel,
                        cost_dec, cand_dec, &tie, &close);
    st->tie_dec += tie;
    st->close_dec += close;
    if (follow_pre)
      ip = follow(pt, ip, follow_pre[r], P, cost_pre, cand_pre, tie_rel, &st->near_tie_pre, &st->mismatch_pre,
                  &st->first_mismatch, r);
    if (follow_dec)
      id = follow(pt, id, follow_dec[r], D, cost_dec, cand_dec, tie_rel, &st->near_tie_dec, &st->mismatch_dec,
                  &st->first_mismatch, r);

    /* 3. prefill on ip, transfer the KV, decode on id: one request at a time
     * per instance, in admission order. */
    const int64_t s_pre = pt->pre_base_ns + (int64_t)p * pt->pre_tok_ns;
    const int64_t s_dec = (int64_t)(o - 1) * pt->dec_tok_ns;
    const int64_t xfer = (int64_t)p * pt->xfer_tok_ns;
    inst_t* a = &pre[ip];
    const int64_t pf_end = (now > a->busy ? now : a->busy) + s_pre;
    if (a->size > a->head && pf_end < a->t_rel[a->size - 1]) st->violations++;
    a->busy = pf_end;
    if (push(a, pf_end, p, p)) {
      rc = -2;
      goto done;
    }
    if (a->kv > pt->kv_cap_pre) st->over_cap_pre++;
    if (a->queue > st->max_queue_pre) st->max_queue_pre = a->queue;

    inst_t* b = &dec[id];
    const int64_t kv_at = pf_end + xfer;
    const int64_t dec_end = (kv_at > b->busy ? kv_at : b->busy) + s_dec;
    if (b->size > b->head && dec_end < b->t_rel[b->size - 1]) st->violations++;
    b->busy = dec_end;
    if (push(b, dec_end, (int64_t)p + o, oh)) {
      rc = -2;
      goto done;
    }
    if (b->kv > pt->kv_cap_dec) st->over_cap_dec++;
    if (b->queue > st->max_queue_dec) st->max_queue_dec = b->queue;

    /* 4. record the outcome. */
    i_pre[r] = ip;
    i_dec[r] = id;
    ttft_ns[r] = pf_end - now;
    span_ns[r] = dec_end - pf_end;
  }

  for (int32_t j = 0; j < P; ++j) st->end_inflight_pre += pre[j].queue;
  for (int32_t j = 0; j < D; ++j) st->end_inflight_dec += dec[j].queue;
  /* Drain: after every release everything must return to zero. */
  for (int32_t j = 0; j < P; ++j) {
    retire(&pre[j], INT64_MAX, &st->violations);
    if (pre[j].queue || pre[j].kv || pre[j].pend) st->violations++;
  }
  for (int32_t j = 0; j < D; ++j) {
    retire(&dec[j], INT64_MAX, &st->violations);
    if (dec[j].queue || dec[j].kv || dec[j].pend) st->violations++;
  }

done:
  free_pool(pre, P);
  free_pool(dec, D);
  free(cost_pre);
  free(cost_dec);
  free(f_backlog);
  free(f_queue);
  free(f_kv);
  return rc;
}

/* ------------------------------------------------------------------------ */
/* Goodput: SLO attainment under per-class TTFT/TPOT targets (Table II,      */
/* Section IV-B).  TPOT = decode span / (o - 1); a one-token answer has no    */
/* inter-token time and meets its TPOT target.                               */
/* ------------------------------------------------------------------------ */
int64_t orc_goodput(const orc_point* pt, int64_t n, const int32_t* out_len,
                    const uint8_t* slo_class, const int64_t* ttft_ns, const int64_t* span_ns,
                    double* goodput) {
  int64_t met = 0;
  for (int64_t r = 0; r < n; ++r) {
    const uint8_t c = slo_class[r];
    if (ttft_ns[r] < 0 || c >= ORC_MAX_CLASSES) continue;
    const int ok_ttft = ttft_ns[r] <= pt->slo_ttft_ns[c];
    const int ok_tpot = out_len[r] <= 1 || span_ns[r] <= pt->slo_tpot_ns[c] * (int64_t)(out_len[r] - 1);
    if (ok_ttft && ok_tpot) met++;
  }
  if (goodput) *goodput = n > 0 ? (double)met / (double)n : 0.0;
  return met;
}


/* ------------------------------------------------------------------------ */
/* Continuous batching at the prefill and the decode stage alike (Section VI): processor sharing with a */
/* batch-dependent speed.  See rt_oracle.h for the model.                   */
/* ------------------------------------------------------------------------ */

/* A batch member: the virtual time at which it finishes (virtual time
 * counts the stand-alone service each member of the batch has received). */
typedef struct {
  double f;
  int64_t r;
} bmember;

/* A KV transfer on its way to a decode instance: the time it lands. */
typedef struct {
  double t;
  int64_t r;
} bjoin;

typedef struct {
  double v, t_last;  /* virtual time, valid at time t_last                  */
  bmember* act;      /* the batch, sorted by (f, r)                          */
  int64_t nact, cap;
  bjoin* wait;       /* decode only: transfers in flight, sorted by (t, r)   */
  int64_t nwait, wcap;
  int64_t owed_wait; /* decode only: stand-alone work (ns) of the requests
                        routed here that have not joined the batch yet      */
  int64_t queue, kv, pend;
} binst;

/* Per-request time factor of a batch of b: 1 + beta (b - 1). */
static double slowdown(double beta, int64_t b) { return 1.0 + beta * (double)(b - 1); }

static int grow(void** a, int64_t* cap, size_t sz) {
  int64_t nc = *cap ? 2 * *cap : 16;
  void* p = realloc(*a, (size_t)nc * sz);
  if (!p) return -1;
  *a = p;
  *cap = nc;
  return 0;
}

static int batch_insert(binst* s, double f, int64_t r) {
  if (s->nact == s->cap && grow((void**)&s->act, &s->cap, sizeof(bmember))) return -1;
  int64_t i = s->nact;
  while (i > 0 && (s->act[i - 1].f > f || (s->act[i - 1].f == f && s->act[i - 1].r > r))) {
    s->act[i] = s->act[i - 1];
    i--;
  }
  s->act[i].f = f;
  s->act[i].r = r;
  s->nact++;
  return 0;
}

static int wait_insert(binst* s, double t, int64_t r) {
  if (s->nwait == s->wcap && grow((void**)&s->wait, &s->wcap, sizeof(bjoin))) return -1;
  int64_t i = s->nwait;
  while (i > 0 && (s->wait[i - 1].t > t || (s->wait[i - 1].t == t && s->wait[i - 1].r > r))) {
    s->wait[i] = s->wait[i - 1];
    i--;
  }
  s->wait[i].t = t;
  s->wait[i].r = r;
  s->nwait++;
  return 0;
}

/* Bring the instance's virtual time to time t, with no event in between:
 * each of the b members receives dv of service. */
static void b_advance(binst* s, double beta, double t) {
  if (s->nact > 0) s->v += (t - s->t_last) / slowdown(beta, s->nact);
  s->t_last = t;
}

/* A member joins with stand-alone work w: it finishes once the virtual
 * clock has advanced by w. */
static int b_join(binst* s, double w, int64_t r) { return batch_insert(s, s->v + w, r); }

/* Time of the instance's next completion (+inf when idle).  The remaining
 * virtual work is clamped at 0, so a completion never lies before t_last. */
static double b_next(const binst* s, double beta) {
  if (s->nact == 0) return INFINITY;
  double rem = s->act[0].f - s->v;
  if (rem < 0.0) rem = 0.0;
  return s->t_last + rem * slowdown(beta, s->nact);
}

typedef struct {
  const orc_point* pt;
  binst *pre, *dec;
  const int32_t *p, *o, *oh;
  const int32_t* idec;    /* decode placements */
  double *pf_end, *dec_end;
  orc_stats* st;
} bsim;

/* Stand-alone (batch of one) service of request r in each stage: the serial
 * model's service times. */
static int64_t work_pre(const bsim* b, int64_t r) { return b->pt->pre_base_ns + (int64_t)b->p[r] * b->pt->pre_tok_ns; }
static int64_t work_dec(const bsim* b, int64_t r) { return (int64_t)(b->o[r] - 1) * b->pt->dec_tok_ns; }

/* Process every event at or before time T in time order (completions before
 * transfer landings at equal times, lower instance first, prefill pool
 * before decode pool), then bring every instance's virtual time to T
 * (skipped for T = +inf, the final drain). */
static int b_run_to(bsim* b, double T) {
  const int32_t P = b->pt->n_prefill, D = b->pt->n_decode;
  for (;;) {
    double te = INFINITY;
    int32_t k = -1;
    int landing = 0;
    for (int32_t j = 0; j < P + D; ++j) {
      const double tc = j < P ? b_next(&b->pre[j], b->pt->beta_pre) : b_next(&b->dec[j - P], b->pt->beta_dec);
      if (tc < te) {
        te = tc;
        k = j;
      }
    }
    for (int32_t d = 0; d < D; ++d)
      if (b->dec[d].nwait > 0 && b->dec[d].wait[0].t < te) {
        te = b->dec[d].wait[0].t;
        k = P + d;
        landing = 1;
      }
    if (k < 0 || te > T) break;
    if (!landing) {
      /* every member sharing the smallest finish virtual time leaves */
      const int is_pre = k < P;
      binst* s = is_pre ? &b->pre[k] : &b->dec[k - P];
      const double fmin = s->act[0].f;
      s->v = fmin;
      s->t_last = te;
      int64_t m = 0;
      while (m < s->nact && s->act[m].f == fmin) m++;
      for (int64_t i = 0; i < m; ++i) {
        const int64_t r = s->act[i].r;
        s->queue -= 1;
        if (is_pre) {
          s->kv -= b->p[r];
          s->pend -= b->p[r];
          b->pf_end[r] = te;
          b->st->retired_pre++;
          /* the KV leaves for the decode instance and lands a transfer later */
          if (wait_insert(&b->dec[b->idec[r]], te + (double)((int64_t)b->p[r] * b->pt->xfer_tok_ns), r)) return -2;
        } else {
          s->kv -= (int64_t)b->p[r] + b->o[r];
          s->pend -= b->oh[r];
          b->dec_end[r] = te;
          b->st->retired_dec++;
        }
        if (s->queue < 0 || s->kv < 0 || s->pend < 0) b->st->violations++;
      }
      for (int64_t i = m; i < s->nact; ++i) s->act[i - m] = s->act[i];
      s->nact -= m;
    } else {
      /* a KV lands: its request joins the decode batch */
      binst* s = &b->dec[k - P];
      const int64_t r = s->wait[0].r;
      for (int64_t i = 1; i < s->nwait; ++i) s->wait[i - 1] = s->wait[i];
      s->nwait--;
      b_advance(s, b->pt->beta_dec, te);
      s->owed_wait -= work_dec(b, r);
      if (b_join(s, (double)work_dec(b, r), r)) return -2;
    }
  }
  if (T < INFINITY) {
    for (int32_t j = 0; j < P; ++j) b_advance(&b->pre[j], b->pt->beta_pre, T);
    for (int32_t d = 0; d < D; ++d) b_advance(&b->dec[d], b->pt->beta_dec, T);
  }
  return 0;
}

/* Features of one pool.  Clock backlog (backlog(d) of Section III-A, the
 * work the instance has taken on and not yet done, under batching): the stand-alone
 * work (ns) the instance still owes, summed over the batch in member order,
 * each member's max(f - v, 0) (clamped as in b_next), plus, on a decode
 * instance, the whole work of the requests routed there that have not
 * joined (an exact integer), in seconds.  Ledger backlog: as in the serial
 * model. */
static void batched_features(const bsim* b, int32_t pool, float* backlog, int64_t* queue, int64_t* kv) {
  const orc_point* pt = b->pt;
  const int32_t n = pool == ORC_PREFILL ? pt->n_prefill : pt->n_decode;
  for (int32_t j = 0; j < n; ++j) {
    const binst* s = pool == ORC_PREFILL ? &b->pre[j] : &b->dec[j];
    queue[j] = s->queue;
    kv[j] = s->kv;
    if (pt->backlog_mode == ORC_BACKLOG_TRUE) {
      double w = 0.0;
      for (int64_t i = 0; i < s->nact; ++i) {
        const double left = s->act[i].f - s->v;
        w += left < 0.0 ? 0.0 : left;
      }
      w += (double)s->owed_wait;
      backlog[j] = (float)w * 1e-9f;
    } else {
      backlog[j] = ledger_backlog(pt, pool, s->queue, s->pend);
    }
  }
}

static void free_binst(binst* a, int32_t n) {
  if (!a) return;
  for (int32_t j = 0; j < n; ++j) {
    free(a[j].act);
    free(a[j].wait);
  }
  free(a);
}

int orc_sim_replica_batched(const orc_point* pt, int64_t n, const int64_t* arrival_ns,
                            const int32_t* prompt_len, const int32_t* out_len, const int32_t* pred_out_len,
                            const uint8_t* slo_class, const uint32_t* sample_bits, const int32_t* follow_pre,
                            const int32_t* follow_dec, double tie_rel, int32_t* i_pre, int32_t* i_dec,
                            int64_t* ttft_ns, int64_t* span_ns, orc_stats* st) {
  if (!pt || !st || n < 0) return -1;
  if (pt->n_prefill < 1 || pt->n_decode < 1 || pt->n_classes < 1 || pt->n_classes > ORC_MAX_CLASSES ||
      pt->kv_cap_pre < 1 || pt->kv_cap_dec < 1 || !(pt->beta_pre >= 0.0) || !(pt->beta_dec >= 0.0) ||
      !isfinite(pt->beta_pre) || !isfinite(pt->beta_dec))
    return -1;
  if (pt->policy == ORC_LENGTH_THRESHOLD && pt->len_threshold < 1) return -1;
  if (n > 0 && (!arrival_ns || !prompt_len || !out_len || !pred_out_len || !slo_class || !i_pre || !i_dec ||
                !ttft_ns || !span_ns))
    return -1;
  if (pt->policy == ORC_LEARNED_SAMPLED && n > 0 && !sample_bits) return -1;
  memset(st, 0, sizeof *st);
  st->first_mismatch = -1;
  const int32_t P = pt->n_prefill, D = pt->n_decode;
  const int32_t N = P > D ? P : D;
  bsim b;
  memset(&b, 0, sizeof b);
  b.pt = pt;
  b.p = prompt_len;
  b.o = out_len;
  b.oh = pred_out_len;
  b.idec = i_dec;
  b.st = st;
  b.pre = (binst*)calloc((size_t)P, sizeof(binst));
  b.dec = (binst*)calloc((size_t)D, sizeof(binst));
  b.pf_end = (double*)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
  b.dec_end = (double*)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
  float* f_backlog = (float*)calloc((size_t)N, sizeof(float));
  int64_t* f_queue = (int64_t*)calloc((size_t)N, sizeof(int64_t));
  int64_t* f_kv = (int64_t*)calloc((size_t)N, sizeof(int64_t));
  float* cost_pre = (float*)calloc((size_t)P, sizeof(float));
  float* cost_dec = (float*)calloc((size_t)D, sizeof(float));
  int rc = 0;
  if (!b.pre || !b.dec || !b.pf_end || !b.dec_end || !f_backlog || !f_queue || !f_kv || !cost_pre || !cost_dec) {
    rc = -2;
    goto done;
  }

  int64_t last_arrival = 0;
  int have_arrival = 0;
  for (int64_t r = 0; r < n; ++r) {
    const int64_t now = arrival_ns[r];
    const int32_t p = prompt_len[r], o = out_len[r], oh = pred_out_len[r];
    const uint8_t c = slo_class[r];
    /* the serial model's data checks */
    if (p < 1 || o < 1 || oh < 1 || (int64_t)p + o > INT32_MAX || (int64_t)p + oh > INT32_MAX ||
        c >= pt->n_classes || now < 0 || (have_arrival && now < last_arrival)) {
      st->invalid++;
      i_pre[r] = i_dec[r] = -1;
      continue;
    }
    last_arrival = now;
    have_arrival = 1;

    /* 1. every completion and transfer landing up to the arrival */
    if ((rc = b_run_to(&b, (double)now)) != 0) goto done;

    /* 2. each pool's argmin on that state */
    int tie, close;
    int32_t cand_pre[2], cand_dec[2];
    const uint32_t* w = sample_bits ? sample_bits + 4 * r : NULL;
    batched_features(&b, ORC_PREFILL, f_backlog, f_queue, f_kv);
    int32_t ip = choose(pt, ORC_PREFILL, P, r, f_backlog, f_queue, f_kv, p, oh, c, w, tie_rel, cost_pre, cand_pre,
                        &tie, &close);
    st->tie_pre += tie;
    st->close_pre += close;
    batched_features(&b, ORC_DECODE, f_backlog, f_queue, f_kv);
    int32_t id = choose(pt, ORC_DECODE, D, r, f_backlog, f_queue, f_kv, p, oh, c, w ? w + 2 : NULL, tie_rel,
                        cost_dec, cand_dec, &tie, &close);
    st->tie_dec += tie;
    st->close_dec += close;
    if (follow_pre)
      ip = follow(pt, ip, follow_pre[r], P, cost_pre, cand_pre, tie_rel, &st->near_tie_pre, &st->mismatch_pre,
                  &st->first_mismatch, r);
    if (follow_dec)
      id = follow(pt, id, follow_dec[r], D, cost_dec, cand_dec, tie_rel, &st->near_tie_dec, &st->mismatch_dec,
                  &st->first_mismatch, r);
    i_pre[r] = ip;
    i_dec[r] = id;

    /* 3. admission: the prefill batch takes the request now; the decode
     * instance holds its cache and counts it from now, and takes it into its
     * batch when its KV lands */
    binst* a = &b.pre[ip];
    if (b_join(a, (double)work_pre(&b, r), r)) {
      rc = -2;
      goto done;
    }
    a->queue += 1;
    a->kv += p;
    a->pend += p;
    if (a->kv > pt->kv_cap_pre) st->over_cap_pre++;
    if (a->queue > st->max_queue_pre) st->max_queue_pre = a->queue;
    binst* d = &b.dec[id];
    d->owed_wait += work_dec(&b, r);
    d->queue += 1;
    d->kv += (int64_t)p + o;
    d->pend += oh;
    if (d->kv > pt->kv_cap_dec) st->over_cap_dec++;
    if (d->queue > st->max_queue_dec) st->max_queue_dec = d->queue;
  }
  for (int32_t j = 0; j < P; ++j) st->end_inflight_pre += b.pre[j].queue;
  for (int32_t j = 0; j < D; ++j) st->end_inflight_dec += b.dec[j].queue;
  /* 4. drain: everything in flight finishes; then every count is zero */
  {
    const int64_t kept_pre = st->retired_pre, kept_dec = st->retired_dec;
    if ((rc = b_run_to(&b, INFINITY)) != 0) goto done;
    st->retired_pre = kept_pre;
    st->retired_dec = kept_dec;
  }
  for (int32_t j = 0; j < P; ++j)
    if (b.pre[j].queue || b.pre[j].kv || b.pre[j].pend || b.pre[j].nact) st->violations++;
  for (int32_t j = 0; j < D; ++j)
    if (b.dec[j].queue || b.dec[j].kv || b.dec[j].pend || b.dec[j].nact || b.dec[j].nwait || b.dec[j].owed_wait)
      st->violations++;
  /* 5. outcomes, rounded to whole ns (nearest, ties to even) */
  for (int64_t r = 0; r < n; ++r) {
    if (i_pre[r] < 0) {
      ttft_ns[r] = span_ns[r] = -1;
      continue;
    }
    if (!(b.pf_end[r] >= (double)arrival_ns[r]) || !(b.dec_end[r] >= b.pf_end[r])) st->violations++;
    ttft_ns[r] = llrint(b.pf_end[r] - (double)arrival_ns[r]);
    span_ns[r] = llrint(b.dec_end[r] - b.pf_end[r]);
  }

done:
  free_binst(b.pre, P);
  free_binst(b.dec, D);
  free(b.pf_end);
  free(b.dec_end);
  free(f_backlog);
  free(f_queue);
  free(f_kv);
  free(cost_pre);
  free(cost_dec);
  return rc;
}
