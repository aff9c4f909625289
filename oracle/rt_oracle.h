/*
 * Plain sequential CPU oracle for the learned prefill/decode router and its
 * serial-service discrete-event simulation.
 *
 * TEST INFRASTRUCTURE ONLY.  This library exists to check the HIP path: only
 * the test suite, the smoke check and the benchmark's CPU-baseline leg may
 * load it.  It shares no code, header or constant with the GPU library, and
 * the product path never calls it.
 *
 * What it computes (the paper: Section III-A cost equation and Algorithm 1;
 * Section III-D and Section VI for the simulator; Section IV-B for the SLO
 * targets):
 *   - orc_score:        score every instance of one pool for each request and
 *                       take the argmin (lowest index on equal cost);
 *   - orc_sim_replica:  one replica of the disaggregated prefill -> KV
 *                       transfer -> decode pipeline, one request at a time in
 *                       arrival order, FIFO serial service per instance;
 *                       optionally in "follow" mode, where it adopts
 *                       externally supplied placements and accounts every
 *                       divergence from its own choice;
 *   - orc_sim_replica_batched: the same replica with both stages
 *                       batched continuously (processor sharing with a
 *                       batch-dependent slowdown);
 *   - orc_goodput:      fraction of a replica's requests meeting both the
 *                       TTFT and the TPOT target of their class.
 *
 * Every floating-point step is evaluated in float32 in the order the cost
 * equation is written, left to right, one rounding per operation (the
 * library is built with -ffp-contract=off, so no fused multiply-add).
 * Simulated times are int64 nanoseconds in the serial model and float64
 * nanoseconds inside the batched one.
 */
#ifndef RT_ORACLE_H
#define RT_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ORC_MAX_CLASSES 8

/* ORC_LEARNED_SAMPLED: the learned score over two randomly drawn candidates per pool
 * (the sampled variant Section V-E and Section VI name as the mitigation for
 * scarce pools).  The random words are inputs (see orc_candidates). */
/* ORC_LENGTH_THRESHOLD: the predicted-length threshold baseline (Section
 * IV-C), read as size-interval assignment: prefill least loaded; decode least
 * loaded within the lower part [0, ceil(D/2)) for o^ < len_threshold, within
 * the upper part [ceil(D/2), D) otherwise (both parts are instance 0 when
 * D == 1). */
enum { ORC_LEARNED = 0, ORC_ROUND_ROBIN = 1, ORC_LEAST_LOADED = 2, ORC_LEARNED_SAMPLED = 3, ORC_LENGTH_THRESHOLD = 4 };
enum { ORC_BACKLOG_TRUE = 0, ORC_BACKLOG_PROXY = 1 };
enum { ORC_PREFILL = 0, ORC_DECODE = 1 };

typedef struct {
  float w_b, w_s, w_q, rho;   /* hand-set weights of the cost equation        */
  float tau_pre_s, tau_dec_s; /* priced seconds per prompt / output token      */
  float pre_base_s;           /* priced prefill base (in-flight ledger only)   */
  float sigma[ORC_MAX_CLASSES]; /* SLO amplifier per class                     */
} orc_router;

typedef struct {
  int32_t n_prefill, n_decode, n_classes;
  int32_t policy, backlog_mode;
  orc_router router;
  int64_t pre_base_ns, pre_tok_ns, dec_tok_ns, xfer_tok_ns;
  int64_t kv_cap_pre, kv_cap_dec;
  int64_t slo_ttft_ns[ORC_MAX_CLASSES], slo_tpot_ns[ORC_MAX_CLASSES];
  int32_t len_threshold; /* ORC_LENGTH_THRESHOLD only */
  int32_t service;       /* ORC_SERIAL or ORC_BATCHED (orc_sim_replica_batched) */
  double beta_pre, beta_dec; /* ORC_BATCHED: per-request slowdown per extra batch member */
} orc_point;

enum { ORC_SERIAL = 0, ORC_BATCHED = 1 };

typedef struct {
  int64_t invalid;                   /* requests rejected by the data checks   */
  int64_t near_tie_pre, near_tie_dec; /* follow mode: accepted divergences      */
  int64_t mismatch_pre, mismatch_dec; /* follow mode: divergences beyond tol.   */
  int64_t first_mismatch;            /* request index, -1 if none              */
  int64_t tie_pre, tie_dec;          /* decisions whose best two costs are equal
                                        (lowest index taken)                   */
  int64_t close_pre, close_dec;      /* decisions whose best two costs differ by
                                        a positive gap within the tolerance    */
  int64_t over_cap_pre, over_cap_dec; /* admissions with occupancy above cap    */
  int64_t max_queue_pre, max_queue_dec;
  int64_t retired_pre, retired_dec;  /* FIFO pops before the last arrival      */
  int64_t violations;                /* internal invariant failures (must be 0) */
  int64_t end_inflight_pre, end_inflight_dec; /* after the last arrival       */
} orc_stats;

/* The two candidates a pool of n >= 1 instances offers for one request,
 * from the request's two random words u, v of that pool: the first is
 * floor(u * n / 2^32); the second is drawn the same way from v among the
 * n - 1 others (floor(v * (n - 1) / 2^32), counted past the first), so that
 * the two differ whenever n >= 2; with n == 1 both are instance 0. */
void orc_candidates(uint32_t u, uint32_t v, int32_t n, int32_t* c1, int32_t* c2);

/* Score n_inst instances of one pool for each of n_req requests.
 *   backlog_s/queue/kv_occ: instance snapshot; request i uses row
 *   i*inst_stride (inst_stride 0 = one snapshot shared by all requests).
 *   out_idx[i] = argmin (lowest index on equal cost), out_score[i] = its cost;
 *   out_second[i] (may be NULL) = second-lowest cost (+inf if n_inst == 1).
 *   sample_bits (may be NULL): [n_req][2] words u, v; when given, only the
 *   two candidates orc_candidates draws from them are scored, out_idx is the
 *   cheaper of the two (lower index on equal cost) and out_second the other
 *   one's cost (+inf if n_inst == 1).
 *   A request with prompt_len < 1, slo_class >= ORC_MAX_CLASSES or (decode
 *   pool) pred_out_len < 1 or prompt_len + pred_out_len >= 2^31 gets idx -1
 *   and NaN scores.
 * Returns 0, or -1 on a bad argument. */
int orc_score(const orc_router* rp, int32_t pool, int32_t n_inst, const float* backlog_s,
              const int32_t* queue, const int32_t* kv_occ, int64_t kv_cap, int64_t inst_stride,
              int64_t n_req, const int32_t* prompt_len, const int32_t* pred_out_len,
              const uint8_t* slo_class, const uint32_t* sample_bits, int32_t* out_idx, float* out_score,
              float* out_second);

/* Simulate one replica of n requests (arrays indexed 0..n-1).
 *   follow_pre/follow_dec: NULL for a free run, else externally chosen
 *   placements to adopt (see the header comment); tie_rel is the relative
 *   tolerance under which a divergent learned placement is accepted (under
 *   the sampled policy only a placement on one of the two candidates).
 *   sample_bits: [n][4] words for ORC_LEARNED_SAMPLED (words 0, 1 draw the
 *   prefill candidates, words 2, 3 the decode ones); NULL otherwise.
 *   Outputs: i_pre, i_dec, ttft_ns = prefill end - arrival,
 *   span_ns = decode end - prefill end; all -1 for a rejected request (a
 *   length < 1, a token total p + o or p + o^ >= 2^31, a class out of range,
 *   a negative arrival or one earlier than the previous accepted arrival).
 * Returns 0, -1 on a bad argument, -2 on allocation failure. */
int orc_sim_replica(const orc_point* pt, int64_t n, const int64_t* arrival_ns,
                    const int32_t* prompt_len, const int32_t* out_len,
                    const int32_t* pred_out_len, const uint8_t* slo_class, const uint32_t* sample_bits,
                    const int32_t* follow_pre, const int32_t* follow_dec, double tie_rel,
                    int32_t* i_pre, int32_t* i_dec, int64_t* ttft_ns, int64_t* span_ns,
                    orc_stats* st);

/* The same replica under continuous batching at the prefill and the decode stage alike (the service
 * model Section VI adds to the serial one): every instance serves all its
 * admitted requests at once, each at 1 / (1 + beta * (b - 1)) of its
 * stand-alone speed while b requests share the instance (beta_pre for
 * prefill, beta_dec for decode, finite and >= 0; a batch of one runs at full
 * speed, so the model reduces to the serial one wherever requests never
 * overlap).  A request's stand-alone work is its serial service time.  It
 * joins its prefill instance's batch at its arrival and its decode
 * instance's batch when its KV lands there (prefill end + transfer); it holds
 * cache and ledger tokens and counts in the queue of both instances from its
 * admission to the end of that stage.
 * Each instance keeps a virtual clock v (stand-alone service received by
 * every member since the instance's start), advanced by dt / (1 + beta (b-1))
 * at each of its events, and a batch of members sorted by finish virtual
 * time f = v at joining + work (then by request index); its next completion
 * lies at t_last + max(f_min - v, 0) * (1 + beta (b - 1)), and every member
 * with f == f_min leaves then.
 * Clock backlog is the stand-alone work the instance still owes, in
 * seconds: the sum over the batch, in member order, of each member's
 * remaining work max(f - v, 0), plus (decode) the int64 sum of the decode
 * work of the requests routed there that have not joined; ledger backlog as
 * in the serial model.
 * Times are float64 ns, events at equal times in the order: completions,
 * then KV landings, then the arrival being routed; the lower-numbered
 * instance first (prefill pool before decode pool), landings in request
 * order.  ttft and span are rounded to whole ns (nearest, ties to even).
 * Same arguments and outputs as orc_sim_replica; follow mode and
 * sample_bits as there.  Returns -1 also for a negative or non-finite
 * beta. */
int orc_sim_replica_batched(const orc_point* pt, int64_t n, const int64_t* arrival_ns,
                            const int32_t* prompt_len, const int32_t* out_len, const int32_t* pred_out_len,
                            const uint8_t* slo_class, const uint32_t* sample_bits, const int32_t* follow_pre,
                            const int32_t* follow_dec, double tie_rel, int32_t* i_pre, int32_t* i_dec,
                            int64_t* ttft_ns, int64_t* span_ns, orc_stats* st);

/* Number of requests meeting both SLO targets of their class; *goodput is
 * that count over n (0 when n == 0). */
int64_t orc_goodput(const orc_point* pt, int64_t n, const int32_t* out_len,
                    const uint8_t* slo_class, const int64_t* ttft_ns, const int64_t* span_ns,
                    double* goodput);

#ifdef __cplusplus
}
#endif
#endif
