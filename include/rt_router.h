/*
 * rt_router: replica-batched simulation of a learned prefill/decode router
 * for disaggregated LLM serving, on AMD Instinct MI355X (gfx950).
 *
 * Method (arxiv 2609.16206, "Calibrate, Then Route"):
 *   - Section III-A, cost equation: every candidate instance d of a pool is
 *     scored by an estimate of the completion time request r would see there,
 *       cost(d) = w_b * backlog(d) * sigma(s_r)
 *               + w_s * o_r * tau_dec * (1 + rho * press+(d)) * sigma(s_r)
 *               + w_q * queue(d),
 *     prefill candidates the same way with p_r * tau_pre; the request goes to
 *     the argmin of each pool.
 *   - Algorithm 1: per admission, argmin over the prefill pool, argmin over
 *     the decode pool, prefill, KV transfer, decode, record the outcome.
 *   - Section III-D and Section VI: a deterministic discrete-event simulator
 *     with explicit pools, KV transfer and SLO accounting; serial service
 *     (one request at a time per instance).  Backlog is either read from the
 *     simulation clock or priced by the router's in-flight ledger with its own
 *     constants (the deployed proxy's estimator).
 *   - Section IV-B: SLO targets per class (TTFT, TPOT); goodput = SLO
 *     attainment (Table II).
 *
 * Conventions shared by every entry point
 *   - Sizes are element counts.  Simulated time is int64 nanoseconds; fields
 *     named *_s are float32 seconds.
 *   - Buffers named "device" are device pointers owned by the caller (for
 *     example the storage of torch tensors on the current HIP device); the
 *     library never frees them.  Parameter structs are host memory, read
 *     during the call only.
 *   - Work is enqueued on `hip_stream` (a hipStream_t; NULL = the null stream)
 *     and returns before it completes, except where a function says it
 *     synchronizes.
 *   - Argument errors are reported synchronously with a negative rt_status
 *     before anything is launched; rt_last_error() then describes the
 *     problem.  No C++ exception crosses this interface.
 *   - Per-request data errors are not argument errors: such a request is
 *     rejected in place (its outputs are set to -1) and a sticky bit is set
 *     in the simulator's device flag word (rt_sim_data_status).
 *   - Arithmetic: every float operation of the cost equation is a single
 *     float32 operation in the order the equation is written (left to right;
 *     no fused multiply-add), integer-to-float conversions round to nearest
 *     even, and press+ is (occupancy + need) times the float32 reciprocal of
 *     the cache capacity.  Equal costs resolve to the lowest instance index.
 *   - A simulator handle is used by one host thread at a time.
 */
#ifndef RT_ROUTER_H
#define RT_ROUTER_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RT_OK = 0,
  RT_EINVAL = -1,       /* a null pointer, a negative size or an out-of-range parameter */
  RT_ENOMEM = -2,       /* device or host allocation failed                              */
  RT_EDEVICE = -3,      /* a HIP runtime call failed                                     */
  RT_ERANGE = -4,       /* a size beyond a documented limit                              */
  RT_EUNSUPPORTED = -5, /* a pool shape the library has no kernel for                   */
  RT_EDATA = -6         /* the device flag word reports rejected requests                */
} rt_status;

typedef enum {
  RT_POLICY_LEARNED = 0,      /* the marginal-cost scorer (Section III-A)              */
  RT_POLICY_ROUND_ROBIN = 1,  /* request r goes to instance r mod N (Section IV-C)     */
  RT_POLICY_LEAST_LOADED = 2, /* fewest in-flight requests, lowest index on ties       */
  RT_POLICY_LEARNED_SAMPLED = 3, /* the scorer over two randomly drawn candidates per pool: the
                                   sampled variant that Section V-E and Section VI give
                                   as the mitigation for scarce pools (candidates: see
                                   rt_sim_run_replicas)                                */
  RT_POLICY_LENGTH_THRESHOLD = 4 /* the predicted-length threshold baseline of Section
                                   IV-C, read as size-interval assignment: requests
                                   with o^_r >= len_threshold use the upper part of the
                                   decode pool, the others the lower part (see
                                   rt_sim_run_replicas); least loaded within a part   */
} rt_policy;

typedef enum {
  RT_BACKLOG_TRUE = 0,  /* backlog = busy-until minus now, from the simulation clock   */
  RT_BACKLOG_PROXY = 1  /* backlog = the router's ledger: tau * priced tokens in flight
                           (+ pre_base_s per in-flight request on the prefill pool)     */
} rt_backlog_mode;

typedef enum { RT_POOL_PREFILL = 0, RT_POOL_DECODE = 1 } rt_pool;

typedef enum {
  RT_SERVICE_SERIAL = 0,  /* one request at a time per instance, in admission order
                             (the serial-service model of Section III-D / VI)        */
  RT_SERVICE_BATCHED = 1  /* continuous batching at the prefill and the decode stage alike (the model Section VI
                             adds): every admitted request is served at once, each at
                             1 / (1 + beta (b - 1)) of its stand-alone speed while b
                             requests share the instance (see rt_sim_run_replicas)  */
} rt_service;

#define RT_MAX_CLASSES 8
/* Instances per pool.  The widest pool of every workload here is 1,024
 * decode instances; the simulation kernels keep each instance's state and
 * the front of its queue in registers, and eight waves of 64 lanes at five
 * instances a lane hold two pools of 1,024, which is the most one workgroup
 * holds that way. */
#define RT_MAX_POOL 1024

/* The router's priced view (Section III-A, Section III-B).  All finite and
 * >= 0, so every cost is >= 0. */
typedef struct {
  float w_b, w_s, w_q, rho;     /* hand-set weights                                   */
  float tau_pre_s, tau_dec_s;   /* priced seconds per prompt / predicted output token */
  float pre_base_s;             /* priced prefill base, used by the proxy ledger only */
  float sigma[RT_MAX_CLASSES];  /* SLO amplifier sigma(s) per class                   */
} rt_router_params;

/* True service physics and SLO targets (Section VI constants, Section IV-B
 * targets).  Service of request r: prefill pre_base_ns + p_r * pre_tok_ns;
 * KV transfer p_r * xfer_tok_ns (a pure delay); decode (o_r - 1) * dec_tok_ns.
 * All >= 0 and <= 2^40; capacities >= 1 (soft: occupancy above capacity is
 * priced, never blocked).  Simulated times must stay below 2^52 ns. */
typedef struct {
  int64_t pre_base_ns, pre_tok_ns, dec_tok_ns, xfer_tok_ns;
  int64_t kv_cap_pre, kv_cap_dec;                 /* cache tokens per instance */
  int64_t slo_ttft_ns[RT_MAX_CLASSES], slo_tpot_ns[RT_MAX_CLASSES];
} rt_physics;

/* One parameter point: pool shape, policy, router constants and physics. */
typedef struct {
  int32_t n_prefill, n_decode; /* 1 .. RT_MAX_POOL                        */
  int32_t n_classes;           /* 1 .. RT_MAX_CLASSES                     */
  int32_t policy;              /* rt_policy                               */
  int32_t backlog_mode;        /* rt_backlog_mode                         */
  rt_router_params router;
  rt_physics phys;
  int32_t len_threshold;       /* RT_POLICY_LENGTH_THRESHOLD: predicted output
                                  tokens at which a request counts as long
                                  (>= 1); unread by the other policies      */
  int32_t service;             /* rt_service                              */
  double beta_pre, beta_dec;   /* RT_SERVICE_BATCHED: slowdown per extra
                                  batch member in prefill / decode, finite
                                  and >= 0 (the measured decode curve of
                                  Section VI: 0.029 / 7)                    */
  int32_t batch_cap;           /* RT_SERVICE_BATCHED: room per instance for
                                  batch members and for KV transfers in
                                  flight; 0 = 256, else a power of two in
                                  [2, 65536]                               */
  int32_t reserved;            /* set to 0                                */
} rt_point;

typedef struct rt_sim rt_sim; /* opaque: device copies of the points, scratch, flag word */

/* Create a simulator for n_points parameter points on HIP device `device`.
 * Copies the points (host memory) to the device.  Returns RT_EINVAL for a bad
 * point (the message names it), RT_EUNSUPPORTED for a pool wider than
 * RT_MAX_POOL, RT_EDEVICE/RT_ENOMEM on runtime failures.  *out is set only on
 * success.  Synchronizes the device once. */
rt_status rt_sim_create(const rt_point* points, int32_t n_points, int32_t device, rt_sim** out);

/* Free the simulator and its device memory.  Waits for the device first.
 * NULL is accepted. */
rt_status rt_sim_destroy(rt_sim* sim);

/* A batch of independent replicas, structure of arrays, all device memory. */
typedef struct {
  int64_t n_replicas;          /* >= 0                                                   */
  int64_t n_requests;          /* total length of the request arrays                      */
  const int64_t* offsets;      /* [n_replicas+1]; replica i = requests [offsets[i],
                                  offsets[i+1]); non-decreasing, offsets[n] <= n_requests,
                                  each replica < 2^31 requests                            */
  const int32_t* param_point;  /* [n_replicas], each in [0, n_points); NULL = point 0      */
  const int64_t* arrival_ns;   /* >= 0, non-decreasing within a replica                   */
  const int32_t* prompt_len;   /* p_r >= 1                                                */
  const int32_t* out_len;      /* o_r >= 1, true output length: physics only, the router
                                  never reads it                                          */
  const int32_t* pred_out_len; /* o^_r >= 1, predicted output length                      */
  const uint8_t* slo_class;    /* s_r < the point's n_classes                             */
  const uint32_t* sample_bits; /* [n_requests][4] random words for RT_POLICY_LEARNED_SAMPLED:
                                  words 0, 1 draw request r's prefill candidates, words
                                  2, 3 its decode candidates; required when a replica
                                  uses that policy, else may be NULL (never read)         */
} rt_trace;

/* Per-request outputs, device memory, each of length trace->n_requests
 * (entries outside every replica are left untouched). */
typedef struct {
  int32_t* i_pre;           /* chosen prefill instance                          */
  int32_t* i_dec;           /* chosen decode instance                           */
  int64_t* ttft_ns;         /* prefill end - arrival (first token at prefill end) */
  int64_t* decode_span_ns;  /* decode end - prefill end; TPOT = span / (o_r - 1)  */
} rt_sim_out;

/* Simulate every replica of `trace` (Algorithm 1 per admission, serial
 * service per instance).  Per replica, requests are admitted in index order
 * at their arrival time; first every instance releases the requests that
 * finished at or before that time, then each pool is scored on that state and
 * its argmin taken (the two argmins are independent), then the request is
 * served: prefill ends at max(arrival, prefill busy-until) + service, its KV
 * reaches the decode instance a transfer delay later, and decode ends at
 * max(KV arrival, decode busy-until) + service; instances serve in admission
 * order.  A request is rejected in place (outputs -1, no state change, flag
 * bit set) if p_r, o_r or o^_r < 1, p_r + o_r or p_r + o^_r >= 2^31, its class
 * is out of range, or its arrival is negative or earlier than the replica's
 * previous accepted arrival.
 * Under RT_POLICY_LEARNED_SAMPLED a pool of n instances offers two candidates
 * drawn from the request's two words u, v of that pool:
 *   c1 = floor(u * n / 2^32);  n == 1: c2 = c1;  else with
 *   x = floor(v * (n - 1) / 2^32), c2 = x + (x >= c1 ? 1 : 0)
 * (two distinct instances, every ordered pair equally likely up to a bias of
 * n / 2^32), and the request goes to the cheaper of the two, the lower index
 * on equal cost.  With n <= 2 this is the full argmin.
 * Under RT_POLICY_LENGTH_THRESHOLD the prefill pool is least loaded (fewest
 * requests in flight, lowest index); the decode pool of D instances is cut
 * into a lower part [0, ceil(D/2)) and an upper part [ceil(D/2), D) (with
 * D == 1 both parts are instance 0), a request with o^_r >= len_threshold
 * goes to the least loaded instance of the upper part, any other request to
 * the least loaded of the lower part.
 * A point with service RT_SERVICE_BATCHED changes how instances serve, not
 * how the router scores (the cost equation and every policy read the same
 * features).  Its request joins its prefill instance's batch at its arrival
 * and its decode instance's batch when its KV lands there (prefill end +
 * transfer); while b requests share an instance, each receives stand-alone
 * service at 1 / (1 + beta (b - 1)) of full speed (beta_pre, beta_dec), and
 * it leaves when it has received its stand-alone work (the serial service
 * time).  It holds its cache and ledger tokens and counts in the queue of
 * both instances from its admission to the end of each stage, as in the
 * serial model.  Each instance keeps a virtual clock v (stand-alone service
 * received by each member), advanced by dt / (1 + beta (b - 1)) at each of
 * its events; members are ordered by finish virtual time f = v at joining +
 * work, then request index; the next completion lies at
 * t_last + max(f_min - v, 0) (1 + beta (b - 1)), and every member with
 * f == f_min leaves then.  Clock backlog is the stand-alone work still owed
 * (Section III-A's backlog under batching), in seconds: the batch's
 * remaining work plus, on a decode instance, the decode work of requests
 * routed there that have not joined (an exact integer sum, added last).
 * The kernels keep the batch's remaining work as a running float64 total
 * per instance (+ each joining member's work; - b * dv at every
 * virtual-time step dv, in event order; reset to 0 when the batch empties;
 * clamped at 0 when read); it equals the sum over members of max(f - v, 0)
 * up to rounding, so a placement can differ from one made on that sum only
 * where two costs lie within rounding of each other.  Ledger backlog is
 * unchanged.  Times
 * are float64 ns; at equal times completions come first, then KV landings,
 * then the arrival being routed.  TTFT and decode span are rounded to whole
 * ns (nearest, ties to even).  An instance holds at most batch_cap members
 * and batch_cap KV transfers in flight; a replica that would exceed either
 * stops there (its outputs are not valid) and sets flag bit 3.
 * The call reads offsets and param_point back to the host to plan the launch
 * (it synchronizes `hip_stream` for that), validates them (RT_EINVAL), then
 * enqueues the simulation on `hip_stream` and returns.  Scratch memory grows
 * with n_requests (for serial points: 64 bytes per request, 128 for points
 * with the proxy backlog, 192 when a call holds both kinds), and for
 * batched replicas with about 68 + 32 batch_cap bytes per instance slot: a
 * replica of a point with P + D <= 64 takes S slots, S the smallest of 4, 8,
 * 16, 32, 64 that holds P + D; one with ceil(P / 2) + ceil(D / 2) <= 64
 * (at most 128 instances) takes 128; a larger point takes P + D slots (each
 * kind sized by the largest pool and batch_cap among the call's points of
 * that kind).  It is owned by `sim`. */
rt_status rt_sim_run_replicas(rt_sim* sim, const rt_trace* trace, rt_sim_out* out, void* hip_stream);

/* For callers that cannot allocate memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): the same
 * simulation as rt_sim_run_replicas, with the same arguments and outputs,
 * bit for bit, for serial-service points, calling no hipMalloc, hipFree or
 * other allocating routine.  Its FIFO record planes and its work list live
 * in a fixed 64 MiB device array that the library holds on every GPU it has
 * run on until the process ends (its address is resolved once per device,
 * by rt_sim_create), and its launch is planned in fixed host arrays.
 * Limits, each returned as RT_ERANGE before anything is launched: at most
 * 65,536 replicas per call and 4,096 points per simulator, and at most
 * 64 MiB of scratch: 64 bytes per request of trace->n_requests (128 for
 * points with the proxy backlog, 192 when a call holds both kinds), plus
 * 4 bytes per replica, plus a fixed 192 KiB at most (dummy records ahead
 * of the record planes).  A point with
 * continuous-batching service returns RT_EUNSUPPORTED.  Every kernel class
 * runs on `hip_stream` in turn (rt_sim_run_replicas runs them side by side
 * on streams of its own).  Nothing in the array needs to start at zero:
 * every record is written before it is read.  All calls on one GPU share
 * the array, so calls that overlap on one GPU (on different streams, or
 * from different threads without ordering) race and their outputs are not
 * valid; calls on one stream are ordered.  The host-side planning arrays
 * are shared by all threads and guarded by a lock: the call waits for the
 * offsets read-back and for the work list's upload before it returns. */
rt_status rt_sim_run_replicas_noalloc(rt_sim* sim, const rt_trace* trace, rt_sim_out* out, void* hip_stream);

/* Per-replica goodput, the SLO attainment that Table II reports, under the
 * per-class TTFT and TPOT targets of Section IV-B: the fraction of the
 * replica's requests that meet both
 * their class's TTFT target (ttft <= TTFT_c) and TPOT target
 * (span <= TPOT_c * (o_r - 1); always met when o_r == 1).  Rejected requests
 * count as missed; an empty replica has goodput 0.  goodput: [n_replicas]
 * device doubles; met: [n_replicas] device int64 counts or NULL.  Reads the
 * trace (offsets and param_point on the device) and the outputs of
 * rt_sim_run_replicas; enqueue it on the same stream after that call. */
rt_status rt_goodput(const rt_sim* sim, const rt_trace* trace, const rt_sim_out* out,
                     double* goodput, int64_t* met, void* hip_stream);

/* Synchronize `hip_stream`, return the sticky device flag word in *flags
 * (may be NULL) and clear it.  Returns RT_EDATA if any bit was set:
 *   bit 0: a request was rejected (length, class or arrival order);
 *   bit 1: rt_goodput met a replica whose offsets or point id are
 *          inconsistent (its goodput is 0 and its met count -1);
 *   bit 2: a simulated time reached 2^52 ns (about 52 days), beyond which
 *          the kernels' exact integer arithmetic no longer holds (the
 *          outputs of such a run are not valid);
 *   bit 3: a replica of a batched point outgrew its point's batch_cap (its
 *          outputs are not valid; run it again with a larger batch_cap). */
rt_status rt_sim_data_status(rt_sim* sim, void* hip_stream, uint32_t* flags);

/* Measurement hook.  rt_sim_timing(sim, 1) resets the totals and makes every
 * later rt_sim_run_replicas call record a HIP event pair on its stream: one
 * after its launch preparation, just before the first simulation kernel, one
 * after the last.  rt_sim_kernel_time waits for the last recorded pair and
 * returns the summed elapsed milliseconds and the number of timed calls since
 * timing was enabled.  rt_sim_timing(sim, 0) stops recording.  Host memory
 * outputs; either may be NULL. */
rt_status rt_sim_timing(rt_sim* sim, int32_t enable);
rt_status rt_sim_kernel_time(rt_sim* sim, double* total_ms, int64_t* calls);

/* Standalone batched scorer: the cost equation and per-pool argmin for
 * n_req independent requests against an instance snapshot (Section III-A).
 *   pool: RT_POOL_DECODE prices o^_r * tau_dec with need p_r + o^_r;
 *         RT_POOL_PREFILL prices p_r * tau_pre with need p_r (o^_r unread).
 *   backlog_s / queue / kv_occ: device arrays, instance j of request i at
 *         [i * inst_stride + j]; inst_stride 0 = one snapshot shared by all
 *         requests, else inst_stride >= n_inst.  backlog_s finite >= 0,
 *         queue >= 0, kv_occ >= 0.
 *   prompt_len / pred_out_len / slo_class: device arrays [n_req].
 *   out_idx [n_req] device: argmin, lowest index on equal cost;
 *   out_score [n_req] device: its cost.
 * A request with p_r < 1, (decode) o^_r < 1 or p_r + o^_r >= 2^31, or
 * slo_class >= RT_MAX_CLASSES gets out_idx -1 and a NaN score.
 * Limits: 1 <= n_inst <= RT_MAX_POOL, kv_cap >= 1, n_req >= 0. */
rt_status rt_score_argmin(const rt_router_params* prm, int32_t pool, int32_t n_inst,
                          const float* backlog_s, const int32_t* queue, const int32_t* kv_occ,
                          int32_t kv_cap, int64_t inst_stride, int64_t n_req,
                          const int32_t* prompt_len, const int32_t* pred_out_len,
                          const uint8_t* slo_class, int32_t* out_idx, float* out_score,
                          void* hip_stream);

/* Message describing the last non-OK status returned on this host thread
 * ("" if none).  Valid until the next call on the thread. */
const char* rt_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* RT_ROUTER_H */
