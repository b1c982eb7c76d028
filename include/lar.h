/*
 * lar.h -- C ABI of the MI355X SFS TTFT estimator and latency-aware router.
 *
 * The library estimates, for every (scenario z, query q, model instance j), the
 * time-to-first-token of q at j by Serving Framework Simulation (SFS, Sec. 4.1):
 * the instance's resident requests plus the new query are replayed through the
 * serving scheduler's token batches -- one decode token per decoding sequence,
 * then prefill chunks in arrival (FCFS) order under a per-batch token budget B
 * and a cap M on running sequences -- and the modelled batch times
 *     T = a + b*P + c*D + d*C + e*A                  (batch-time model, Sec. 4.1)
 * are summed up to and including the batch in which q produces its first decode
 * token (the first-output-token batch and the SFS TTFT sum, Sec. 4.1).
 * P = prefill tokens, D = decode tokens, C = context of the decoding sequences,
 * A = sum over chunks of chunk*context + chunk*(chunk+1)/2.  In the paper's
 * notation a = beta_0, b = c = beta_1, d = beta_2, e = beta_3.  Every binary64
 * operation is one round-to-nearest-even operation in the order written, with no
 * fused multiply-add; sums over batches are left folds in batch order.
 *
 * Routing follows the Lagrangian objective of Sec. 3 with the utility of Eq. 2:
 *     u_j = (acc_j - w_cost*cost_j) - w_lat*TTFT_j,   choice = lowest j with max u,
 * or the constrained objective of Eq. 3 (the *_constrained calls): the lowest j of
 * maximal utility acc_j - w_cost*cost_j among the instances with TTFT_j <= tau,
 * and, when none is within the target tau, the lowest j of minimal TTFT_j.
 *
 * Conventions
 *  - Every call returns lar_status (LAR_OK == 0, errors < 0).
 *  - Pointers marked "dev" are device (HBM) pointers; "host" are host pointers.
 *    The caller owns all array arguments (contiguous, int32 / int64 / float64 as
 *    declared).  The context owns its device state, allocated by lar_create and
 *    lar_load_state; the estimate / route / commit / trace / stats calls allocate
 *    nothing.
 *  - Calls enqueue work on the context's HIP stream and return without waiting;
 *    outputs are valid once the caller synchronises the stream (or lar_sync).
 *  - Errors found on the host (bad arguments) return at once with nothing
 *    enqueued; lar_error_string() gives the detail.  Errors found by kernels
 *    (queue overflow, iteration cap, instance not advanced, prompt too long) set a
 *    sticky device flag, reported by lar_sync / lar_read_state; once observed it is
 *    returned by every later call until lar_load_state resets it.
 *  - A batch of zero queries (n_q == 0, n == 0) is valid: the call returns LAR_OK,
 *    enqueues nothing and leaves the state as it was (a trace of zero queries does
 *    not advance the instances either).  A negative count is LAR_E_ARG.
 *    lar_stats and lar_ontime_utility average over the queries and need n_q >= 1.
 *  - A context is not thread-safe.
 *
 * Time unit: milliseconds.  Layouts are row-major.
 */
#ifndef LAR_H
#define LAR_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lar_ctx lar_ctx;
typedef int32_t lar_status;

enum {
  LAR_OK = 0,
  LAR_E_ARG = -1,      /* invalid argument                                      */
  LAR_E_STATE = -2,    /* invalid snapshot, or an instance clock behind t       */
  LAR_E_CAPACITY = -3, /* waiting queue of an instance would exceed queue_cap   */
  LAR_E_ITER = -4,     /* a simulation needed more than max_iters batches       */
  LAR_E_HIP = -5,      /* HIP runtime failure                                   */
  LAR_E_SYNC = -6      /* workgroups of one scenario could not run together     */
};

/* Which batch yields the first token (the first-output-token batch, Sec. 4.1). */
enum {
  LAR_FIRST_TOKEN_DECODE_BATCH = 0,  /* default: first batch in which q decodes     */
  LAR_FIRST_TOKEN_PREFILL_BATCH = 1  /* alternate reading: batch completing q's prefill */
};

/* Per-instance batch-time coefficients (ms) and scheduler limits (Sec. 4.1). */
typedef struct {
  double a, b, c, d, e;   /* T = a + b*P + c*D + d*C + e*A, all finite             */
  int32_t token_budget;   /* B: tokens per batch, max_seqs <= B <= 2^30 - 1        */
  int32_t max_seqs;       /* M: running sequences, 1 <= M <= lar_config.max_seqs_cap */
  int32_t col;            /* column of this instance in the acc / cost arrays, >= 0 */
  int32_t reserved;       /* must be 0                                              */
} lar_instance_params;

typedef struct {
  int32_t n_scen;         /* Z >= 1 routing scenarios (independent state copies)    */
  int32_t n_inst;         /* I >= 1 model instances                                 */
  int32_t max_seqs_cap;   /* upper bound on every instance's M, 1..1024             */
  int32_t queue_cap;      /* waiting requests per (scenario, instance), >= 1        */
  int32_t max_prompt;     /* largest query prompt accepted (tokens), >= 1           */
  int32_t flags;          /* LAR_FIRST_TOKEN_*                                      */
  int64_t max_iters;      /* batch cap of one estimate or one advance, >= 1         */
  void *stream;           /* hipStream_t to enqueue on; NULL = null stream          */
} lar_config;

/*
 * Create a context and allocate its device state.  *out is NULL on failure.
 * Read from the environment at creation (tests of the failure paths, not needed in
 * use): LAR_SYNC_TIMEOUT_MS bounds the wait of a multi-workgroup trace for its
 * other workgroups (default 10000 ms, then LAR_E_SYNC); LAR_TEST_SKIP_POST=m:q makes
 * workgroup m of every scenario skip its post for query q (so the others reach the
 * bound); LAR_TEST_TAG_START starts the realised-TTFT tag counter at that value (so
 * a test reaches its wrap).
 */
lar_status lar_create(lar_ctx **out, const lar_config *cfg);

/* Free the context (synchronises its stream first).  NULL is accepted. */
lar_status lar_destroy(lar_ctx *ctx);

/* Detail of the last error on this context; owned by the context. */
const char *lar_error_string(const lar_ctx *ctx);

/*
 * Load an instance snapshot (Sec. 4 setup; App. E, workload snapshots): for every
 * instance j, its resident requests in FCFS order, requests offsets[j] ..
 * offsets[j+1]-1 of the host arrays, each with remaining prefill rem_prefill,
 * predicted remaining decode rem_decode and context length context (0 = waiting).
 * The snapshot is copied into every scenario.  Validates: offsets non-decreasing
 * from 0; rem_prefill >= 0; rem_decode >= 1; context >= 0; rem_prefill == 0
 * implies context > 0; running (context > 0) before waiting; at most max_seqs
 * running (LAR_E_STATE), at most queue_cap waiting (LAR_E_CAPACITY); finite
 * clocks.  Resets the sticky device error.  Synchronises the stream.
 *   params   host [I]
 *   offsets  host [I+1]
 *   rem_prefill, rem_decode, context  host [offsets[I]]
 *   clock_ms host [I]  instance clocks
 */
lar_status lar_load_state(lar_ctx *ctx, const lar_instance_params *params,
                          const int32_t *offsets, const int32_t *rem_prefill,
                          const int32_t *rem_decode, const int32_t *context,
                          const double *clock_ms);

/*
 * Scheduler limits of an instance (the system appendix lists context limits,
 * KV-cache allocation and preemption among what the SFS simulation follows; Sec. 2
 * describes paged KV caches and chunked prefill).  Each is optional (0 = none):
 *   chunk_cap   a request receives at most this many prefill tokens per batch;
 *   max_ctx     context limit: a request's context (prompt + generated tokens) never
 *               exceeds it.  A request entering with cx + rp tokens has its predicted
 *               decode cut to max_ctx - (cx + rp); cx + rp < max_ctx is required.  An
 *               instance cannot take a query whose prompt is >= its max_ctx: its
 *               estimate is +infinity and the routes never choose it (a pool may mix
 *               small and large limits); a query that no instance can take is routed
 *               nowhere (choice -1) with the sticky LAR_E_ARG;
 *   kv_blocks   KV cache of kv_blocks blocks of block_size tokens (block_size a power
 *               of two, 1 .. 65536): a running request holds ceil(cx / block_size)
 *               blocks.  Requires max_ctx > 0 and kv_blocks * block_size >= max_ctx.
 * With limits, a batch gives each running request in list order one decode token
 * (decoding ones), then min(rp, chunk_cap, budget left) (partially prefilled ones).
 * When a request's new blocks do not fit, the last running request is preempted
 * (recompute), repeatedly, until they fit or the request itself is out: its blocks,
 * including those taken in this batch, and its tokens of this batch are returned,
 * and it becomes the first waiting request with its whole context to prefill again.
 * Waiting requests are admitted only in a batch without preemption, in FCFS order,
 * while budget is left, fewer than max_seqs run and the first chunk's blocks fit.
 * With every limit 0 the batches are the default ones bit for bit.
 */
typedef struct {
  int32_t chunk_cap;
  int32_t kv_blocks;
  int32_t block_size;
  int32_t max_ctx;
} lar_sched_limits;

/*
 * Put scheduler limits on every instance (host [I]), or remove them (NULL).  The
 * state is laid out for the scheduler in use, so a lar_load_state must follow
 * before any other call (until then they return LAR_E_STATE).  With limits set,
 * estimates and traces simulate each (query, instance) pair from the instance state
 * (the shared-trajectory shortcuts of the default scheduler are not used); the
 * snapshot validation also requires cx + rp < max_ctx for every request and at most
 * kv_blocks blocks held by the running ones (LAR_E_STATE).  Bad limits: LAR_E_ARG,
 * nothing changed.  Synchronises the stream.
 */
lar_status lar_set_scheduler(lar_ctx *ctx, const lar_sched_limits *limits);

/*
 * Re-install the snapshot of the last lar_load_state (kept in device memory) into
 * every scenario, with device-to-device copies enqueued on the stream: no host
 * traffic, no synchronisation.  Clears the sticky device error.  Use it to replay
 * a trace again from the same snapshot.
 */
lar_status lar_reload_state(lar_ctx *ctx);

/*
 * SFS what-if estimate (Sec. 4.1): TTFT of each query q (prompt q_prefill[q]
 * tokens, 1..max_prompt) arriving at time t_ms at every instance of every
 * scenario.  Pure: the state is not modified.  Every instance clock must be
 * >= t_ms (advance with lar_commit first), else the sticky LAR_E_STATE is set.
 * Under scheduler limits an instance whose context limit is at or below the prompt
 * cannot take the query: +infinity there (iters 0), no error.
 *   q_prefill dev [Q]
 *   ttft_ms   dev [Z][Q][I]  float64, TTFT = (clock + T_1 + ... + T_l) - t_ms
 *   iters     dev [Z][Q][I]  int32, l = number of batches simulated; may be NULL
 */
lar_status lar_estimate_ttft(lar_ctx *ctx, int32_t n_q, const int32_t *q_prefill, double t_ms,
                             double *ttft_ms, int32_t *iters);

/*
 * Route (Lagrangian objective, Sec. 3, with the utility of Eq. 2):
 *   choice[z][q] = lowest j maximising (acc[q][col_j] - w_cost[z]*cost[q][col_j])
 *                                        - w_lat[z]*ttft_ms[z][q][j].
 *   ttft_ms     dev [Z][Q][I]
 *   acc, cost   dev [Q][n_cols]; col_j = params[j].col must be < n_cols
 *   w_cost      dev [Z]   (lambda of Eq. 2)
 *   w_lat       dev [Z]   latency weight per ms (delta of the objective, per ms)
 *   choice      dev [Z][Q] int32
 *   chosen_ttft dev [Z][Q] TTFT at the choice; may be NULL
 *   utility     dev [Z][Q] acc - w_cost*cost at the choice (Eq. 2); may be NULL
 * An instance whose TTFT is +infinity (it cannot take the query) is no candidate, and
 * neither is a NaN utility; a row without any candidate gets choice -1 and sets the
 * sticky LAR_E_ARG.
 */
lar_status lar_route(lar_ctx *ctx, int32_t n_q, const double *ttft_ms, const double *acc,
                     const double *cost, int32_t n_cols, const double *w_cost,
                     const double *w_lat, int32_t *choice, double *chosen_ttft,
                     double *utility);

/*
 * Route under the constrained objective (Eq. 3, Sec. 3): per (z, q),
 *   F = { j : ttft_ms[z][q][j] <= tau_ms[q] };
 *   choice[z][q] = lowest j in F maximising acc[q][col_j] - w_cost[z]*cost[q][col_j]
 *                  (Eq. 2) if F is not empty, else lowest j minimising ttft_ms[z][q][j].
 *   ttft_ms  dev [Z][Q][I];  tau_ms dev [Q] TTFT targets (e.g. from lar_ttft_targets)
 *   acc, cost dev [Q][n_cols];  w_cost dev [Z] (lambda of Eq. 2)
 *   choice dev [Z][Q];  chosen_ttft, utility dev [Z][Q] as in lar_route (may be NULL)
 * Errors: LAR_E_ARG for a null required pointer or n_cols not covering every
 * instance's column.  An instance whose TTFT is +infinity is no candidate in either
 * branch; a row without any candidate gets choice -1 and sets the sticky LAR_E_ARG.
 */
lar_status lar_route_constrained(lar_ctx *ctx, int32_t n_q, const double *ttft_ms,
                                 const double *tau_ms, const double *acc, const double *cost,
                                 int32_t n_cols, const double *w_cost, int32_t *choice,
                                 double *chosen_ttft, double *utility);

/*
 * Per-query TTFT targets (appendix on TTFT latency assignment):
 *   tau_ms[i] = min{1120, max{150, u_ms[i] + (155 + 3.5e-3*q_prefill[i])*v[i]}},
 * evaluated in that order (155 + 3.5e-3*p first, then times v, then plus u), each
 * operation binary64 round-to-nearest-even.  The caller draws u ~ U(1, 5) ms and
 * v ~ U(0.98, 1.02) per query (seeded).  Needs no loaded state.
 *   q_prefill dev [n] int32;  u_ms, v dev [n];  tau_ms dev [n] (output)
 */
lar_status lar_ttft_targets(lar_ctx *ctx, int32_t n, const int32_t *q_prefill,
                            const double *u_ms, const double *v, double *tau_ms);

/*
 * Commit one routed query and replay the instances to t_next_ms.  The paper's
 * router takes a fresh snapshot of every instance after each engine iteration
 * (appendix on the system, query workload snapshots); here the instances are
 * instead replayed by the same token-batch simulation (Sec. 4.1) between
 * arrivals, which stands in for those snapshots.  In scenario z,
 * the query (q_prefill >= 1 prompt tokens, q_decode predicted decode tokens,
 * raised to 1) joins the FCFS tail of instance choice[z] as a waiting request
 * (choice == NULL or choice[z] < 0: nothing is appended); then on every instance
 * every batch that starts before t_next_ms runs, and an idle instance's clock
 * jumps to t_next_ms.  A full waiting queue sets the sticky LAR_E_CAPACITY.  Under
 * scheduler limits the predicted decode is cut to what the context limit leaves,
 * and a prompt at or above that limit is not appended (sticky LAR_E_ARG).
 *   choice dev [Z] or NULL
 */
lar_status lar_commit(lar_ctx *ctx, const int32_t *choice, int32_t q_prefill, int32_t q_decode,
                      double t_next_ms);

/*
 * One routing step with every query value in device memory, so that a caller can
 * capture it once in a HIP graph and replay it per arriving query after writing the
 * query into the same buffers.  Exactly the call sequence
 *   lar_estimate_ttft(1 query *q_prefill, t = *t_ms)
 *   lar_route (tau_ms == NULL) or lar_route_constrained (row of acc / cost)
 *   lar_commit(choice, *q_prefill, *q_decode, *t_next_ms)
 * with the values read when the step runs.  The instances must be advanced to *t_ms
 * (the previous step's *t_next_ms, or lar_commit(NULL, ...) before the first step).
 * Enqueues four kernels; allocates nothing, does not synchronise.
 *   q_prefill, q_decode dev [1] int32;  t_ms, t_next_ms dev [1]
 *   acc, cost dev [n_cols] (this query's row);  w_cost dev [Z]
 *   w_lat dev [Z] (Lagrangian objective) or tau_ms dev [1] (Eq. 3; w_lat unused)
 *   choice dev [Z] int32;  chosen_ttft, utility dev [Z] (may be NULL)
 * Device-found errors (prompt outside 1..max_prompt, queue full, iteration cap) are
 * sticky as for the separate calls.
 */
lar_status lar_route_step(lar_ctx *ctx, const int32_t *q_prefill, const int32_t *q_decode,
                          const double *t_ms, const double *t_next_ms, const double *acc,
                          const double *cost, int32_t n_cols, const double *w_cost,
                          const double *w_lat, const double *tau_ms, int32_t *choice,
                          double *chosen_ttft, double *utility);

/*
 * Sequential routing of N queries, exactly the call sequence
 *   for i in 0..N-1:
 *     lar_estimate_ttft(1 query q_prefill[i], t = q_t_ms[i])
 *     lar_route(row i of acc / cost)            -> choice[z][i]
 *     lar_commit(choice[.][i], q_prefill[i], q_decode[i], t_next)
 *   with t_next = q_t_ms[i+1], and t_after_ms for the last query.
 * The instances must already be advanced to q_t_ms[0].
 *   q_prefill, q_decode dev [N] int32;  q_t_ms dev [N] non-decreasing
 *   acc, cost dev [N][n_cols];  w_cost, w_lat dev [Z]
 *   choice dev [Z][N];  chosen_ttft, utility dev [Z][N] (may be NULL)
 *   realized_ttft dev [Z][N] (may be NULL): the TTFT each query sees in the replay
 *     (the estimates set against measured TTFTs in Fig. 2; Eq. 4 counts it): the
 *     end of the replayed batch that produces its first token (the same batch
 *     reading as the estimate) minus q_t_ms[i].  It can exceed the estimate:
 *     queries that arrive later take the budget a query leaves in its last prefill
 *     batch and decode beside it, which lengthens those batches (Sec. 4.1 batch
 *     time).  A query without its first token at t_after_ms gets it from a private
 *     copy of its instance run on with no further arrivals; the state the call
 *     leaves is not changed by this.  NaN marks a query the replay did not finish
 *     (only after a device error).  Each call tracks its own queries: a query
 *     routed by an earlier call, or committed by lar_commit, is not reported.
 */
lar_status lar_route_trace(lar_ctx *ctx, int32_t n_q, const int32_t *q_prefill,
                           const int32_t *q_decode, const double *q_t_ms, double t_after_ms,
                           const double *acc, const double *cost, int32_t n_cols,
                           const double *w_cost, const double *w_lat, int32_t *choice,
                           double *chosen_ttft, double *utility, double *realized_ttft);

/*
 * lar_route_trace under the constrained objective (Eq. 3; see
 * lar_route_constrained), with query i's TTFT target tau_ms[i]:
 *   for i in 0..N-1:
 *     lar_estimate_ttft(1 query q_prefill[i], t = q_t_ms[i])
 *     lar_route_constrained(row i, tau_ms[i]) -> choice[z][i]
 *     lar_commit(choice[.][i], q_prefill[i], q_decode[i], t_next)
 *   tau_ms dev [N]; the other arguments as in lar_route_trace (no w_lat).
 */
lar_status lar_route_trace_constrained(lar_ctx *ctx, int32_t n_q, const int32_t *q_prefill,
                                       const int32_t *q_decode, const double *q_t_ms,
                                       double t_after_ms, const double *tau_ms,
                                       const double *acc, const double *cost, int32_t n_cols,
                                       const double *w_cost, int32_t *choice,
                                       double *chosen_ttft, double *utility,
                                       double *realized_ttft);

/*
 * Per-scenario summary of a routed trace -- the two axes of the utility-latency
 * trade-off of Sec. 3, E[U] and E[L]:
 *   stats[z] = { mean acc, mean cost, mean (acc - w_cost[z]*cost) (Eq. 2),
 *                p50 TTFT, p99 TTFT }
 * at the chosen instances; means are left folds in query order divided by N,
 * percentiles nearest-rank (sorted[ceil(p*N/100) - 1]).
 *   choice, chosen_ttft dev [Z][N];  acc, cost dev [N][n_cols];  w_cost dev [Z]
 *   stats dev [Z][5] float64
 */
lar_status lar_stats(lar_ctx *ctx, int32_t n_q, const int32_t *choice, const double *chosen_ttft,
                     const double *acc, const double *cost, int32_t n_cols,
                     const double *w_cost, double *stats);

/*
 * OnTimeUtility (Eq. 4) of a routed trace, per scenario:
 *   out[z] = (1/N) * sum over i, in query order, of
 *            (acc[i][col_c] - w_cost[z]*cost[i][col_c]) if realized_ttft[z][i] <= tau_ms[i],
 *            c = choice[z][i]; queries past their target (or NaN) add nothing.
 *   choice dev [Z][N];  realized_ttft dev [Z][N] (the trace's realised TTFT)
 *   tau_ms dev [N];  acc, cost dev [N][n_cols];  w_cost dev [Z];  out dev [Z] float64
 */
lar_status lar_ontime_utility(lar_ctx *ctx, int32_t n_q, const int32_t *choice,
                              const double *realized_ttft, const double *tau_ms,
                              const double *acc, const double *cost, int32_t n_cols,
                              const double *w_cost, double *out);

/*
 * Copy scenario `scen`'s state out (synchronises): resident requests of every
 * instance in FCFS order as in lar_load_state, the clocks and the number of
 * batches replayed per instance since the load.  Under scheduler limits the
 * predicted decodes are the ones cut to the context limit, and a preempted request
 * is a waiting one (context 0) with its whole context to prefill again.  out_cap = capacity of the
 * request arrays; LAR_E_CAPACITY if they are too small (*n_total still set).
 *   offsets host [I+1]; rem_prefill, rem_decode, context host [out_cap]
 *   clock_ms host [I]; iterations_run host [I]
 */
lar_status lar_read_state(lar_ctx *ctx, int32_t scen, int32_t *offsets, int32_t *rem_prefill,
                          int32_t *rem_decode, int32_t *context, double *clock_ms,
                          int64_t *iterations_run, int64_t out_cap, int64_t *n_total);

/*
 * Snapshot board (appendix on the system: query workload snapshots, robustness to
 * incomplete snapshots).  Instances publish their resident requests while they
 * keep generating; the router takes only complete, unmodified copies and keeps
 * the last complete copy per instance.  Host memory only; no device work.
 *
 * lar_board_create: a board for n_inst >= 1 instances of at most max_requests
 *   resident requests each.  *out is NULL on failure (LAR_E_ARG).
 * lar_board_publish: instance `inst` replaces its snapshot (requests in FCFS
 *   order, as in lar_load_state, and its clock).  One publisher per instance at a
 *   time; publishers of different instances may run concurrently with each other
 *   and with lar_board_collect.  LAR_E_ARG for a bad instance, a count above
 *   max_requests or null arrays.
 * lar_board_collect: for every instance, copy its snapshot if a newer complete one
 *   is there (the slot's sequence number even before the copy and unchanged after
 *   it, up to 4 tries), else keep the cached copy; then write all cached copies in
 *   lar_load_state's layout (offsets host [I+1], request arrays host [out_cap],
 *   clock_ms host [I]).  fresh [I] (may be NULL): 1 where a new copy was taken;
 *   versions [I] (may be NULL): sequence number of each cached copy.
 *   LAR_E_STATE while some instance has no complete snapshot yet (the copies
 *   taken are cached all the same), LAR_E_CAPACITY if out_cap is too small.  One
 *   collector at a time.
 */
typedef struct lar_board lar_board;
lar_status lar_board_create(lar_board **out, int32_t n_inst, int32_t max_requests);
lar_status lar_board_destroy(lar_board *board);
lar_status lar_board_publish(lar_board *board, int32_t inst, int32_t n_req,
                             const int32_t *rem_prefill, const int32_t *rem_decode,
                             const int32_t *context, double clock_ms);
lar_status lar_board_collect(lar_board *board, int32_t *offsets, int32_t *rem_prefill,
                             int32_t *rem_decode, int32_t *context, double *clock_ms,
                             int64_t out_cap, int32_t *fresh, uint64_t *versions);

/*
 * Work of the last lar_route_trace / lar_route_trace_constrained call (synchronises):
 * per scenario, the number of token batches its estimates stand for -- for every
 * (query, instance) pair, the batches a literal SFS estimate would simulate from the
 * instance state to the query's first-token batch (Sec. 4.1).  The batches of the
 * replay between arrivals are in lar_read_state's iterations_run.  Zero before the
 * first trace.
 *   estimate_batches host [Z]
 */
lar_status lar_trace_work(lar_ctx *ctx, int64_t *estimate_batches);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): lar_estimate_ttft followed
 * by lar_route for one scenario, with no context.  Same results bit for bit.  The
 * snapshot is read from device memory and laid out on the device; every
 * intermediate buffer lives in one 32 MiB device array in the library, of which
 * each GPU holds its own copy, set up on the first call on that GPU (the stream's
 * device must be current) and kept until the process ends.  The call allocates
 * nothing and does not synchronise.  Calls that overlap on one GPU (other threads,
 * other streams) share that array and race: serialise them.
 *   cfg  host: n_inst I >= 1; max_seqs_cap (bound on every M, 1..1024); max_resident
 *        (bound on the requests of any one instance in the snapshot, >= 0);
 *        max_prompt (>= every q_prefill, >= 1); n_cols (columns of acc / cost);
 *        flags (LAR_FIRST_TOKEN_*); max_iters (>= 1); stream (hipStream_t, NULL =
 *        null stream).  The working memory, about
 *          I * (936 + 12 * max_seqs_cap + 16 * (max_resident + max_seqs_cap))
 *        bytes (each of its 21 arrays rounded up to 256 bytes), must fit the 32 MiB
 *        (else LAR_E_CAPACITY, nothing enqueued).
 *   params   dev [I] instance coefficients and limits, as for lar_load_state
 *   offsets  dev [I+1]; rem_prefill, rem_decode, context dev [offsets[I]]:
 *            the resident requests of every instance in FCFS order (lar_load_state's
 *            layout); the offsets must index these arrays
 *   clock_ms dev [I];  q_prefill dev [Q];  t_ms the arrival time (every clock >= t_ms)
 *   acc, cost dev [Q][n_cols];  w_cost, w_lat dev [1] (as lar_route)
 *   ttft_ms dev [Q][I];  iters dev [Q][I] or NULL;  choice dev [Q];
 *   chosen_ttft, utility dev [Q] or NULL
 *   status   dev [1] int32: set to 0 first, then to the first error found on the
 *            device -- LAR_E_ARG (bad coefficients or limits, a column >= n_cols,
 *            a prompt outside 1..max_prompt, or a prompt bound needing more than 64
 *            decode-only batches after its admission batch), LAR_E_STATE (an
 *            instance's requests break lar_load_state's rules, more than
 *            max_resident of them, or a clock behind t_ms), LAR_E_ITER.  An instance
 *            found invalid is treated as empty; the outputs are meaningful only when
 *            status is 0 after the stream completes.
 * Errors found on the host return at once with nothing enqueued;
 * lar_noalloc_error_string() gives this thread's last detail.  n_q == 0: LAR_OK,
 * nothing enqueued, status not written.
 */
typedef struct {
  int32_t n_inst;
  int32_t max_seqs_cap;
  int32_t max_resident;
  int32_t max_prompt;
  int32_t n_cols;
  int32_t flags;
  int64_t max_iters;
  void *stream;
} lar_whatif_config;

lar_status lar_whatif_noalloc(const lar_whatif_config *cfg, const lar_instance_params *params,
                              const int32_t *offsets, const int32_t *rem_prefill,
                              const int32_t *rem_decode, const int32_t *context,
                              const double *clock_ms, int32_t n_q, const int32_t *q_prefill,
                              double t_ms, const double *acc, const double *cost,
                              const double *w_cost, const double *w_lat, double *ttft_ms,
                              int32_t *iters, int32_t *choice, double *chosen_ttft,
                              double *utility, int32_t *status);
const char *lar_noalloc_error_string(void);

/*
 * Average-case TTFT estimate for routing without real-time workload information
 * (Sec. 4.2, Eqs. 10 and 11; the appendix on the limited-processor-sharing
 * abstraction, Eqs. 12 and 13).  Instance j of scenario z is a server of aggregate
 * capacity mu (service_rate) shared equally by at most k active queries, the others
 * waiting in FCFS order, with queries arriving at rate alpha (arrival_rate):
 *   LAR_LPS_POISSON (Poisson arrivals, memoryless work; Eqs. 10, 12):
 *       rho = alpha / mu,  W = rho^k / (mu - alpha);
 *   LAR_LPS_VARIABILITY (Eq. 13, squared coefficients of variation ca2 of the
 *   inter-arrival times and cs2 of the work):
 *       E[Q] = 1 / mu,  rho = alpha * E[Q],  W = ((ca2 + cs2) / 2) * ((rho^k * E[Q]) / (1 - rho));
 *   and for query q of p = q_prefill[q] prompt tokens (Eq. 11):
 *       ttft_ms[z][q][j] = (W + p / prefill_rate) + decode_ms.
 * rho^k is the product of k factors taken left to right; every operation is one
 * binary64 round-to-nearest-even operation in the order written.  Rates are per ms,
 * times in ms.  The model needs 0 <= alpha < mu, 1 <= k <= 65536, prefill_rate > 0,
 * decode_ms >= 0 (and ca2, cs2 >= 0, rho < 1 under LAR_LPS_VARIABILITY), all finite,
 * reserved == 0, and p >= 1: otherwise NaN there and the sticky LAR_E_ARG.  Needs no
 * loaded snapshot (route the result with lar_route / lar_route_constrained, which
 * take the instances' columns from lar_load_state: an empty snapshot will do).
 *   params    dev [Z][I]
 *   q_prefill dev [Q];  ttft_ms dev [Z][Q][I]
 */
typedef struct {
  double arrival_rate;   /* alpha, queries per ms                               */
  double service_rate;   /* mu, queries per ms at full load                      */
  double prefill_rate;   /* theta, prompt tokens per ms                           */
  double decode_ms;      /* mean time of a decode token batch, ms                 */
  double ca2, cs2;       /* squared coefficients of variation (Eq. 13 only)       */
  int32_t k;             /* queries served at once                                */
  int32_t reserved;      /* must be 0                                             */
} lar_lps_params;

enum { LAR_LPS_POISSON = 0, LAR_LPS_VARIABILITY = 1 };

lar_status lar_estimate_lps(lar_ctx *ctx, const lar_lps_params *params, int32_t mode,
                            int32_t n_q, const int32_t *q_prefill, double *ttft_ms);

/* Synchronise the stream; return the sticky device error, if any. */
lar_status lar_sync(lar_ctx *ctx);

#ifdef __cplusplus
}
#endif

#endif /* LAR_H */
