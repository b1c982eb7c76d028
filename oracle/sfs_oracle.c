/*
 * sfs_oracle.c -- plain, slow CPU oracle of the SFS TTFT estimator and the
 * latency-aware router.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may load this file's library.  It shares no code,
 * header, table or helper with the HIP path; it is compiled with gcc and
 * -ffp-contract=off so every binary64 operation is a single round-to-nearest-even
 * operation, with no fused multiply-add.
 *
 * What it computes (Sec. 4 "Estimating query latencies across model instances"):
 *
 *   * Resident set of an instance (Sec. 4, Setup): an ordered list, in arrival
 *     (FCFS) order, of requests r with remaining prefill tokens rp, predicted
 *     remaining decode tokens rd, and context length cx (tokens already in the KV
 *     cache).  A request is active ("running") iff cx > 0, otherwise it is queued
 *     ("waiting").  Running requests precede waiting ones; at most M run.
 *
 *   * Token batch (Sec. 4.1, paragraph on SFS): at most one decode token per
 *     decoding sequence plus prefill chunks of one or more sequences; decode of a
 *     sequence starts only after its whole prefill.  The simulated scheduler
 *     (App. E, latency estimation paragraph: queue order, admission limit,
 *     token-budget constraint) is: every running request with rp == 0 decodes one
 *     token; the remaining budget goes to prefill chunks in FCFS order, a waiting
 *     request being admitted only while fewer than M requests run; the scan stops
 *     at the first request it cannot serve (head-of-line blocking).
 *
 *   * Batch time (Eq. for the token-batch processing time, Sec. 4.1):
 *       T = a + b*P + c*D + d*C + e*A,
 *     P = sum of prefill tokens, D = number of decode tokens,
 *     C = sum over decoding sequences of their context (KV reads),
 *     A = sum over chunks of chunk*cx + chunk*(chunk+1)/2 (prefill attention).
 *     The paper's coefficients are a = beta_0, b = c = beta_1, d = beta_2,
 *     e = beta_3.  Evaluated as ((((a + b*P) + c*D) + d*C) + e*A).
 *
 *   * SFS estimate (Eqs. for the first-output-token batch and the SFS TTFT sum):
 *     append the new query to the tail of a copy of the resident list, simulate
 *     batches from the instance clock s, and stop at the first batch in which the
 *     query produces a decode token; TTFT = (s + T_1 + ... + T_l) - t, the sum a
 *     left fold in batch order.  Reading A (flag 1) stops instead at the batch in
 *     which the query's prefill completes.
 *
 *   * Route (Eq. for the Lagrangian routing objective with the utility of Eq. 2):
 *       u_j = (acc_j - w_cost*cost_j) - w_lat*TTFT_j,
 *     choice = the lowest j attaining the maximum.  Under scheduler limits an
 *     instance whose context limit cannot hold the query's prompt cannot serve it:
 *     its estimate is +infinity and it is no candidate; a query no instance can
 *     take is an error.
 *
 *   * Commit / advance (replay of the instances between snapshots, App. E on
 *     workload snapshots): append the routed query as a waiting request of the
 *     chosen instance, then on every instance run each batch that starts before
 *     the next arrival time; an idle instance's clock jumps to that time.
 *
 *   * Constrained route (Eq. 3, the primary objective of Sec. 3): among the
 *     instances whose estimated TTFT is within the query's target tau, the lowest
 *     j of maximal utility acc_j - w_cost*cost_j (Eq. 2); when none is within the
 *     target, the lowest j of minimal estimated TTFT.
 *
 *   * TTFT target of a query (appendix on TTFT latency assignment):
 *       tau = min{1120, max{150, u + (155 + 3.5e-3*p)*v}}  (ms),
 *     u ~ U(1, 5) ms and v ~ U(0.98, 1.02) drawn by the caller.
 *
 *   * Realised TTFT (the replay's own first-token times, against which Fig. 2 of
 *     the paper sets the estimates): each routed query is tagged in the replay;
 *     the first batch that produces its first token (the same reading as the
 *     estimate) ends at its first-token time, and realised TTFT = that time minus
 *     the arrival.  Queries still waiting for it when the trace ends are finished
 *     on a copy of their instance with no further arrivals.
 *
 *   * OnTimeUtility (Eq. 4): (1/N) * sum over queries, in query order, of the
 *     utility at the chosen instance when its realised TTFT is within the target,
 *     else 0.
 *
 *   * Scheduler limits (appendix on the system: the simulation follows the
 *     engine's context limits, KV-cache allocation and preemption; Sec. 2 on paged
 *     KV caches and chunked prefill).  The paper names them without defining them;
 *     the reading taken here, per instance and each optional:
 *       - chunk cap H: a request receives at most H prefill tokens per batch;
 *       - context limit X: a request's context (prompt plus generated tokens) never
 *         exceeds X, so its remaining decode is at most X - (cx + rp); a request
 *         needs cx + rp < X;
 *       - KV cache of K blocks of S tokens: a running request holds
 *         ceil(cx / S) blocks, and a batch that gives it n more tokens needs
 *         ceil((cx + n) / S) of them.  Requires X > 0 and K*S >= X.
 *     With limits set, a batch serves the running requests in list order, first
 *     one decode token to each decoding one, then a chunk min(rp, H, budget left)
 *     to each partially prefilled one.  When a request's blocks do not fit, the
 *     last running request is preempted, repeatedly, until they fit: it frees its
 *     blocks (with any taken in this batch), loses the tokens given to it in this
 *     batch, and becomes the first waiting request with its whole context to
 *     prefill again (recompute).  A request that preempts itself gets nothing.
 *     Only in a batch without preemption are waiting requests admitted, in FCFS
 *     order, each while budget is left, fewer than M run and the blocks of its
 *     first chunk fit; the first that cannot be admitted stops the admissions.
 *     With no limit set this is the batch described above.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/*
 * Threads.  The estimates of one query at the different instances are
 * independent (each works on its own copy of one instance), and so is the replay
 * of each instance between two arrivals; the loops over instances below, and the
 * (query, instance) pairs of orc_estimate_matrix, may therefore run on several
 * threads.  Every thread runs exactly the same sequential code on its own
 * instance, and the results are combined in instance order afterwards, so a
 * threaded run is bit-identical to a single-threaded one.  Default: 1 thread.
 */
static int g_threads = 1;

void orc_set_threads(int n) { g_threads = n < 1 ? 1 : n; }
int orc_get_threads(void) { return g_threads; }

#define ORC_OK 0
#define ORC_E_ARG (-1)
#define ORC_E_STATE (-2)
#define ORC_E_CAPACITY (-3)
#define ORC_E_ITER (-4)

typedef struct {
  double a, b, c, d, e;
  int32_t budget;
  int32_t max_seqs;
} orc_params;

typedef struct {
  orc_params pr;
  int64_t n;        /* resident requests */
  int64_t alloc;    /* allocated entries */
  int32_t *rp, *rd, *cx;
  int32_t *qid;     /* routed query still waiting for its first token, else -1 */
  int32_t *dec, *chunk; /* tokens of the batch being built, per request */
  int32_t *blk;         /* KV blocks taken in the batch being built, per request */
  double clock;
  int64_t iters;    /* batches run by advance() since creation */
  /* first-token tracking of the replay (realised == NULL: off) */
  double *realized;     /* [N] realised TTFT per query */
  const double *q_t;    /* [N] arrival times */
  int32_t reading;
  int64_t tracked;      /* residents with qid >= 0 */
  /* scheduler limits (has_sched == 0: none, the default batch) */
  int has_sched;
  int32_t chunk_cap;    /* H, 0 = none */
  int32_t kv_blocks;    /* K, 0 = unlimited */
  int32_t block_size;   /* S */
  int32_t max_ctx;      /* X, 0 = none */
  int64_t preemptions;  /* requests preempted since creation */
} orc_queue;

typedef struct {
  int64_t P, D, C, A;
} orc_feat;

/* ---------------------------------------------------------------- storage */

static int q_reserve(orc_queue *q, int64_t need) {
  if (need <= q->alloc) return ORC_OK;
  int64_t cap = q->alloc ? q->alloc : 16;
  while (cap < need) cap *= 2;
  int32_t **arrs[7] = {&q->rp, &q->rd, &q->cx, &q->qid, &q->dec, &q->chunk, &q->blk};
  for (int k = 0; k < 7; ++k) {
    int32_t *p = (int32_t *)realloc(*arrs[k], (size_t)cap * sizeof(int32_t));
    if (!p) return ORC_E_ARG;
    *arrs[k] = p;
  }
  q->alloc = cap;
  return ORC_OK;
}

static int params_ok(const orc_params *pr) {
  return pr->max_seqs >= 1 && pr->budget >= pr->max_seqs;
}

/* Resident-list invariants: rp >= 0, rd >= 1, cx >= 0, rp == 0 implies cx > 0,
   running (cx > 0) before waiting (cx == 0), at most M running. */
static int state_ok(const orc_params *pr, int64_t n, const int32_t *rp, const int32_t *rd,
                    const int32_t *cx) {
  int64_t running = 0;
  int seen_waiting = 0;
  for (int64_t r = 0; r < n; ++r) {
    if (rp[r] < 0 || rd[r] < 1 || cx[r] < 0) return 0;
    if (rp[r] == 0 && cx[r] == 0) return 0;
    if (cx[r] > 0) {
      if (seen_waiting) return 0;
      ++running;
    } else {
      seen_waiting = 1;
    }
  }
  return running <= pr->max_seqs;
}

orc_queue *orc_queue_new(const orc_params *pr, int64_t n, const int32_t *rp,
                         const int32_t *rd, const int32_t *cx, double clock, int *status) {
  *status = ORC_OK;
  if (!params_ok(pr) || n < 0) { *status = ORC_E_ARG; return NULL; }
  if (!state_ok(pr, n, rp, rd, cx)) { *status = ORC_E_STATE; return NULL; }
  orc_queue *q = (orc_queue *)calloc(1, sizeof(orc_queue));
  if (!q) { *status = ORC_E_ARG; return NULL; }
  q->pr = *pr;
  if (q_reserve(q, n + 1) != ORC_OK) { free(q); *status = ORC_E_ARG; return NULL; }
  for (int64_t r = 0; r < n; ++r) {
    q->rp[r] = rp[r]; q->rd[r] = rd[r]; q->cx[r] = cx[r]; q->qid[r] = -1;
  }
  q->n = n;
  q->clock = clock;
  q->iters = 0;
  return q;
}

void orc_queue_free(orc_queue *q) {
  if (!q) return;
  free(q->rp); free(q->rd); free(q->cx); free(q->qid); free(q->dec); free(q->chunk);
  free(q->blk);
  free(q);
}

static orc_queue *q_clone(const orc_queue *src) {
  int st;
  orc_queue *q = orc_queue_new(&src->pr, src->n, src->rp, src->rd, src->cx, src->clock, &st);
  if (!q) return NULL;
  q->iters = src->iters;
  for (int64_t r = 0; r < src->n; ++r) q->qid[r] = src->qid[r];
  q->realized = src->realized;
  q->q_t = src->q_t;
  q->reading = src->reading;
  q->tracked = src->tracked;
  q->has_sched = src->has_sched;
  q->chunk_cap = src->chunk_cap;
  q->kv_blocks = src->kv_blocks;
  q->block_size = src->block_size;
  q->max_ctx = src->max_ctx;
  return q;
}

/* KV blocks that hold `tokens` cached tokens. */
static int64_t blocks_for(const orc_queue *q, int64_t tokens) {
  return (tokens + q->block_size - 1) / q->block_size;
}

/* Put the scheduler limits (chunk_cap, kv_blocks, block_size, max_ctx; see the
   header) on a queue.  The residents must fit them: cx + rp < max_ctx for each, and
   the running ones' blocks within kv_blocks.  Each resident's remaining decode is
   cut to what the context limit leaves. */
int orc_queue_set_sched(orc_queue *q, const int32_t *lim4) {
  const int32_t H = lim4[0], K = lim4[1], S = lim4[2], X = lim4[3];
  if (H < 0 || K < 0 || X < 0) return ORC_E_ARG;
  if (K > 0 && (S < 1 || X < 1 || (int64_t)K * S < X)) return ORC_E_ARG;
  q->has_sched = 1;
  q->chunk_cap = H;
  q->kv_blocks = K;
  q->block_size = K > 0 ? S : 1;
  q->max_ctx = X;
  int64_t held = 0;
  for (int64_t r = 0; r < q->n; ++r) {
    const int64_t total = (int64_t)q->cx[r] + q->rp[r];
    if (X > 0) {
      if (total >= X) return ORC_E_STATE;
      if (q->rd[r] > X - total) q->rd[r] = (int32_t)(X - total);
    }
    if (q->cx[r] > 0) held += blocks_for(q, q->cx[r]);
  }
  if (K > 0 && held > K) return ORC_E_STATE;
  return ORC_OK;
}

int64_t orc_queue_size(const orc_queue *q) { return q->n; }

int64_t orc_queue_preemptions(const orc_queue *q) { return q->preemptions; }

int64_t orc_queue_waiting(const orc_queue *q) {
  int64_t w = 0;
  for (int64_t r = 0; r < q->n; ++r) w += (q->cx[r] == 0);
  return w;
}

/* Copy the resident list out (FCFS order); arrays must hold orc_queue_size(). */
void orc_queue_get(const orc_queue *q, int32_t *rp, int32_t *rd, int32_t *cx, double *clock,
                   int64_t *iters) {
  for (int64_t r = 0; r < q->n; ++r) { rp[r] = q->rp[r]; rd[r] = q->rd[r]; cx[r] = q->cx[r]; }
  *clock = q->clock;
  *iters = q->iters;
}

/* ---------------------------------------------------------------- one batch */

static orc_feat features(const orc_queue *q) {
  orc_feat f = {0, 0, 0, 0};
  for (int64_t r = 0; r < q->n; ++r) {
    int64_t ch = q->chunk[r];
    f.P += ch;
    f.D += q->dec[r];
    f.C += (int64_t)q->dec[r] * q->cx[r];
    f.A += ch * (int64_t)q->cx[r] + ch * (ch + 1) / 2;
  }
  return f;
}

/* Preempt the last running request (index *running - 1): its blocks, with those
   taken in this batch, return to the pool, the tokens given to it in this batch
   return to the budget, and it becomes the first waiting request, to prefill its
   whole context again. */
static void preempt_last(orc_queue *q, int64_t *running, int64_t *left, int64_t *free_blk) {
  const int64_t v = *running - 1;
  *free_blk += blocks_for(q, q->cx[v]) + q->blk[v];
  *left += q->dec[v] + q->chunk[v];
  q->dec[v] = 0;
  q->chunk[v] = 0;
  q->blk[v] = 0;
  q->rp[v] += q->cx[v];
  q->cx[v] = 0;
  *running = v;
  q->preemptions += 1;
}

/* The batch under scheduler limits (see the header). */
static orc_feat compose_sched(orc_queue *q) {
  const int64_t n = q->n;
  const int kv = q->kv_blocks > 0;
  const int64_t cap = q->chunk_cap > 0 ? q->chunk_cap : INT64_MAX;
  int64_t left = q->pr.budget, running = 0, free_blk = q->kv_blocks;
  int preempted = 0;
  for (int64_t r = 0; r < n; ++r) {
    q->dec[r] = 0;
    q->chunk[r] = 0;
    q->blk[r] = 0;
    if (q->cx[r] > 0) {
      ++running;
      if (kv) free_blk -= blocks_for(q, q->cx[r]);
    }
  }
  /* running requests in list order: decode tokens first */
  for (int64_t r = 0; r < running; ++r) {
    if (q->rp[r] != 0) continue;
    const int64_t need = kv ? blocks_for(q, q->cx[r] + 1) - blocks_for(q, q->cx[r]) : 0;
    while (free_blk < need && r < running) {   /* until it fits, or r itself is out */
      preempt_last(q, &running, &left, &free_blk);
      preempted = 1;
    }
    if (r >= running) break;
    q->dec[r] = 1;
    q->blk[r] = (int32_t)need;
    free_blk -= need;
    left -= 1;
  }
  /* then prefill chunks of the partially prefilled ones */
  for (int64_t r = 0; r < running; ++r) {
    if (q->rp[r] == 0) continue;
    int64_t g = q->rp[r] < cap ? q->rp[r] : cap;
    if (left < g) g = left;
    if (g == 0) continue;
    const int64_t need = kv ? blocks_for(q, q->cx[r] + g) - blocks_for(q, q->cx[r]) : 0;
    while (free_blk < need && r < running) {   /* until it fits, or r itself is out */
      preempt_last(q, &running, &left, &free_blk);
      preempted = 1;
    }
    if (r >= running) break;
    q->chunk[r] = (int32_t)g;
    q->blk[r] = (int32_t)need;
    free_blk -= need;
    left -= g;
  }
  /* admissions, FCFS, in a batch without preemption */
  if (!preempted) {
    const int64_t first_waiting = running;
    for (int64_t r = first_waiting; r < n; ++r) {
      if (left == 0 || running == q->pr.max_seqs) break;
      int64_t g = q->rp[r] < cap ? q->rp[r] : cap;
      if (left < g) g = left;
      const int64_t need = kv ? blocks_for(q, g) : 0;
      if (need > free_blk) break;
      q->chunk[r] = (int32_t)g;
      q->blk[r] = (int32_t)need;
      free_blk -= need;
      left -= g;
      running += 1;
    }
  }
  return features(q);
}

/* Build the next token batch: dec[r] in {0,1}, chunk[r] >= 0; return its features. */
static orc_feat compose(orc_queue *q) {
  if (q->has_sched) return compose_sched(q);
  const int64_t n = q->n;
  int64_t left = q->pr.budget;
  int64_t running = 0;
  for (int64_t r = 0; r < n; ++r) {
    q->dec[r] = 0;
    q->chunk[r] = 0;
    if (q->cx[r] > 0) ++running;
  }
  /* decodes first: one token per running request whose prefill is complete */
  for (int64_t r = 0; r < n; ++r) {
    if (q->cx[r] > 0 && q->rp[r] == 0) {
      q->dec[r] = 1;
      left -= 1;
    }
  }
  /* then prefill chunks in FCFS order */
  for (int64_t r = 0; r < n; ++r) {
    if (q->rp[r] == 0) continue;
    if (left == 0) break;
    if (q->cx[r] == 0) {            /* waiting: needs a free sequence slot */
      if (running == q->pr.max_seqs) break;
      running += 1;
    }
    int64_t ch = q->rp[r] < left ? q->rp[r] : left;
    q->chunk[r] = (int32_t)ch;
    left -= ch;
  }
  return features(q);
}

static double batch_time(const orc_params *pr, orc_feat f) {
  double t = pr->a;
  t = t + pr->b * (double)f.P;
  t = t + pr->c * (double)f.D;
  t = t + pr->d * (double)f.C;
  t = t + pr->e * (double)f.A;
  return t;
}

/* Apply the batch built by compose(): decode tokens extend the context and consume
   predicted decode; chunks extend the context and consume prefill; requests with
   no decode left leave, the others keep their order. */
static void apply(orc_queue *q) {
  int64_t w = 0;
  for (int64_t r = 0; r < q->n; ++r) {
    if (q->dec[r]) { q->cx[r] += 1; q->rd[r] -= 1; }
    if (q->chunk[r]) { q->cx[r] += q->chunk[r]; q->rp[r] -= q->chunk[r]; }
    if (q->rd[r] > 0) {
      q->rp[w] = q->rp[r]; q->rd[w] = q->rd[r]; q->cx[w] = q->cx[r]; q->qid[w] = q->qid[r];
      ++w;
    }
  }
  q->n = w;
}

/* First tokens of the batch built by compose(), which ends at q->clock: a tracked
   query gets its first token in this batch when it decodes in it (reading 0; it
   has not decoded before, or it would no longer be tracked) or when the batch
   completes its prefill (reading 1).  Its realised TTFT is the batch's end minus
   its arrival time, and it is tracked no longer. */
static void record_first_tokens(orc_queue *q) {
  for (int64_t r = 0; r < q->n; ++r) {
    const int32_t i = q->qid[r];
    if (i < 0) continue;
    int first;
    if (q->reading == 1)
      first = q->chunk[r] > 0 && q->chunk[r] == q->rp[r];
    else
      first = q->dec[r] == 1;
    if (first) {
      q->realized[i] = q->clock - q->q_t[i];
      q->qid[r] = -1;
      q->tracked -= 1;
    }
  }
}

/* One batch of the replayed instance; returns its time and features. */
double orc_queue_step(orc_queue *q, int64_t *feat4) {
  orc_feat f = compose(q);
  double T = batch_time(&q->pr, f);
  q->clock = q->clock + T;
  if (q->realized) record_first_tokens(q);
  apply(q);
  q->iters += 1;
  if (feat4) { feat4[0] = f.P; feat4[1] = f.D; feat4[2] = f.C; feat4[3] = f.A; }
  return T;
}

/* Run every batch that starts before t; an empty instance idles until t. */
int orc_queue_advance(orc_queue *q, double t, int64_t max_iters) {
  int64_t k = 0;
  while (q->n > 0 && q->clock < t) {
    if (k == max_iters) return ORC_E_ITER;
    orc_queue_step(q, NULL);
    ++k;
  }
  if (q->n == 0 && q->clock < t) q->clock = t;
  return ORC_OK;
}

/* Append a routed query as a waiting request; query index i >= 0 is tracked
   until its first token (when tracking is on), i = -1 is not. */
/* Predicted decode of a new request of p prompt tokens: at least 1, and no more
   than the context limit leaves (0 when p does not fit the limit). */
static int32_t decode_of(const orc_queue *q, int32_t p, int32_t dhat) {
  int32_t d = dhat < 1 ? 1 : dhat;
  if (q->has_sched && q->max_ctx > 0) {
    if (p >= q->max_ctx) return 0;
    if (d > q->max_ctx - p) d = q->max_ctx - p;
  }
  return d;
}

static int append_tagged(orc_queue *q, int32_t p, int32_t dhat, int64_t queue_cap, int32_t i) {
  if (p < 1 || decode_of(q, p, dhat) < 1) return ORC_E_ARG;
  if (orc_queue_waiting(q) + 1 > queue_cap) return ORC_E_CAPACITY;
  if (q_reserve(q, q->n + 2) != ORC_OK) return ORC_E_ARG;
  q->rp[q->n] = p;
  q->rd[q->n] = decode_of(q, p, dhat);
  q->cx[q->n] = 0;
  q->qid[q->n] = q->realized ? i : -1;
  if (q->realized && i >= 0) q->tracked += 1;
  q->n += 1;
  return ORC_OK;
}

int orc_queue_append(orc_queue *q, int32_t p, int32_t dhat, int64_t queue_cap) {
  return append_tagged(q, p, dhat, queue_cap, -1);
}

/* SFS estimate for a query of p prompt tokens arriving at t (the instance must
   already be advanced to t).  Pure: the queue is not modified. */
int orc_queue_estimate(const orc_queue *q, int32_t p, int32_t dhat, double t, int32_t reading,
                       int64_t max_iters, double *ttft, int32_t *iters) {
  if (p < 1) return ORC_E_ARG;
  if (q->clock < t) return ORC_E_STATE;
  if (decode_of(q, p, dhat) < 1) {   /* the context limit cannot hold the prompt */
    *ttft = INFINITY;
    *iters = 0;
    return ORC_OK;
  }
  orc_queue *w = q_clone(q);
  if (!w) return ORC_E_ARG;
  w->rp[w->n] = p;
  w->rd[w->n] = decode_of(q, p, dhat);
  w->cx[w->n] = 0;
  w->n += 1;
  double E = w->clock;
  int64_t l = 0;
  int done = 0;
  while (!done) {
    if (l == max_iters) { orc_queue_free(w); return ORC_E_ITER; }
    orc_feat f = compose(w);
    const int64_t me = w->n - 1;             /* the query stays last in the list */
    if (reading == 1)
      done = w->chunk[me] > 0 && w->chunk[me] == w->rp[me];
    else
      done = w->dec[me] == 1;
    E = E + batch_time(&w->pr, f);
    ++l;
    apply(w);
  }
  orc_queue_free(w);
  *ttft = E - t;
  *iters = (int32_t)l;
  return ORC_OK;
}

/* ---------------------------------------------------------------- routing */

/* Lagrangian objective over one row; ties go to the lowest instance index. */
int32_t orc_route_row(int32_t n_inst, const double *ttft, const double *acc_row,
                      const double *cost_row, const int32_t *col, double w_cost, double w_lat,
                      double *best_u) {
  int32_t best = -1;
  double bu = 0.0;
  for (int32_t j = 0; j < n_inst; ++j) {
    if (ttft[j] == INFINITY) continue;   /* the instance cannot take the query */
    double pen = w_cost * cost_row[col[j]];
    double u = acc_row[col[j]] - pen;
    double lat = w_lat * ttft[j];
    u = u - lat;
    if (best < 0 || u > bu) { best = j; bu = u; }
  }
  if (best_u) *best_u = bu;
  return best;
}

/* Eq. 3: argmax of the utility over the feasible set {j : ttft_j <= tau}; if that
 * set is empty, argmin of the estimated TTFT.  Lowest index on ties. */
int32_t orc_route_row_constrained(int32_t n_inst, const double *ttft, double tau,
                                  const double *acc_row, const double *cost_row,
                                  const int32_t *col, double w_cost) {
  int32_t best = -1;
  double bu = 0.0;
  for (int32_t j = 0; j < n_inst; ++j) {
    if (!(ttft[j] <= tau)) continue;
    double pen = w_cost * cost_row[col[j]];
    double u = acc_row[col[j]] - pen;
    if (best < 0 || u > bu) { best = j; bu = u; }
  }
  if (best >= 0) return best;
  double bt = 0.0;
  for (int32_t j = 0; j < n_inst; ++j) {
    if (ttft[j] == INFINITY) continue;   /* the instance cannot take the query */
    if (best < 0 || ttft[j] < bt) { best = j; bt = ttft[j]; }
  }
  return best;
}

/* TTFT target (appendix on TTFT latency assignment), evaluated in the written
 * order: lin = 155 + 3.5e-3*p, raw = u + lin*v, then the clip to [150, 1120]. */
double orc_ttft_target(int32_t p, double u_ms, double v) {
  double lin = 155.0 + 3.5e-3 * (double)p;
  double raw = u_ms + lin * v;
  double lo = raw > 150.0 ? raw : 150.0;
  return lo < 1120.0 ? lo : 1120.0;
}

void orc_ttft_targets(int32_t n, const int32_t *p, const double *u_ms, const double *v,
                      double *tau) {
  for (int32_t i = 0; i < n; ++i) tau[i] = orc_ttft_target(p[i], u_ms[i], v[i]);
}

/* ---------------------------------------------------------------- trace */

/* The lowest-indexed error of a loop over instances (what a sequential loop that
   stops at its first error returns), or ORC_OK. */
static int first_error(const int *jst, int32_t n) {
  for (int32_t j = 0; j < n; ++j)
    if (jst[j] != ORC_OK) return jst[j];
  return ORC_OK;
}

/* Replay every instance to t; the instances are independent. */
static int advance_all(orc_queue **qs, int32_t n_inst, double t, int64_t max_iters, int *jst) {
#pragma omp parallel for num_threads(g_threads) schedule(dynamic, 1)
  for (int32_t j = 0; j < n_inst; ++j) jst[j] = orc_queue_advance(qs[j], t, max_iters);
  return first_error(jst, n_inst);
}

/*
 * What-if matrix (the SFS estimate of Sec. 4.1 for many queries at once): for
 * every query i < n_q and instance j < n_inst, the literal estimate of a query of
 * p[i] prompt tokens (predicted decode d[i]) arriving at t at instance j, into
 * ttft[i*n_inst + j] and iters[i*n_inst + j].  The instances must already be
 * advanced to t.  Returns the error of the lowest (i, j) in row-major order that
 * fails, or ORC_OK.
 */
int orc_estimate_matrix(int32_t n_inst, orc_queue *const *qs, int32_t n_q, const int32_t *p,
                        const int32_t *d, double t, int32_t reading, int64_t max_iters,
                        double *ttft, int32_t *iters) {
  if (n_inst < 1 || n_q < 0) return ORC_E_ARG;
  int64_t n = (int64_t)n_q * n_inst;
  int *pst = (int *)malloc((size_t)(n > 0 ? n : 1) * sizeof(int));
  if (!pst) return ORC_E_ARG;
#pragma omp parallel for num_threads(g_threads) schedule(dynamic, 16)
  for (int64_t k = 0; k < n; ++k) {
    int64_t i = k / n_inst, j = k % n_inst;
    pst[k] = orc_queue_estimate(qs[j], p[i], d[i], t, reading, max_iters, &ttft[k], &iters[k]);
  }
  int st = ORC_OK;
  for (int64_t k = 0; k < n && st == ORC_OK; ++k) st = pst[k];
  free(pst);
  return st;
}

/*
 * Sequential routing trace of one scenario:
 *   advance every instance to t_0;
 *   for each query i: estimate every instance at t_i, route, append the query to
 *   the chosen instance, advance every instance to t_{i+1} (t_N := t_{N-1}).
 * The route is the Lagrangian one, or Eq. 3 when tau (per query) is given.
 * Outputs per query: choice, TTFT at the choice, utility of Eq. 2 at the choice
 * (acc - w_cost*cost), and optionally the whole TTFT / iteration rows.
 * The final state is written to the out_* arrays when out_offsets != NULL (each
 * out array must hold out_cap entries).  realized [N] (may be NULL) receives the
 * realised TTFT of every query (NaN where an error stopped the trace first).
 * sched [n_inst][4] (may be NULL) puts scheduler limits on every instance.
 */
int orc_trace(int32_t n_inst, const orc_params *params, const int32_t *col,
              const int32_t *offsets, const int32_t *rp, const int32_t *rd, const int32_t *cx,
              const double *clock, int32_t n_q, const int32_t *q_p, const int32_t *q_d,
              const double *q_t, const double *acc, const double *cost, int32_t n_cols,
              double w_cost, double w_lat, const double *tau, int32_t reading,
              int64_t max_iters, int64_t queue_cap, int32_t *choice, double *ttft_chosen,
              double *util_chosen,
              double *ttft_all, int32_t *iters_all, int32_t *out_offsets, int32_t *out_rp,
              int32_t *out_rd, int32_t *out_cx, double *out_clock, int64_t *out_iters,
              int64_t out_cap, double *realized, const int32_t *sched,
              int32_t *failed_query) {
  int st = ORC_OK;
  *failed_query = -1;
  if (n_inst < 1 || n_q < 0 || n_cols < 1) return ORC_E_ARG;
  for (int32_t j = 0; j < n_inst; ++j)
    if (col[j] < 0 || col[j] >= n_cols) return ORC_E_ARG;
  orc_queue **qs = (orc_queue **)calloc((size_t)n_inst, sizeof(orc_queue *));
  double *row = (double *)malloc((size_t)n_inst * sizeof(double));
  int *jst = (int *)malloc((size_t)n_inst * sizeof(int));
  if (!qs || !row || !jst) { free(qs); free(row); free(jst); return ORC_E_ARG; }
  for (int32_t j = 0; j < n_inst && st == ORC_OK; ++j) {
    int64_t lo = offsets[j], hi = offsets[j + 1];
    qs[j] = orc_queue_new(&params[j], hi - lo, rp + lo, rd + lo, cx + lo, clock[j], &st);
    if (st == ORC_OK && sched) st = orc_queue_set_sched(qs[j], sched + 4 * (int64_t)j);
    if (st == ORC_OK && orc_queue_waiting(qs[j]) > queue_cap) st = ORC_E_CAPACITY;
    if (st == ORC_OK && realized) {
      qs[j]->realized = realized;
      qs[j]->q_t = q_t;
      qs[j]->reading = reading;
    }
  }
  if (realized)
    for (int32_t i = 0; i < n_q; ++i) realized[i] = NAN;
  if (st == ORC_OK && n_q > 0) st = advance_all(qs, n_inst, q_t[0], max_iters, jst);
  for (int32_t i = 0; i < n_q && st == ORC_OK; ++i) {
#pragma omp parallel for num_threads(g_threads) schedule(dynamic, 1)
    for (int32_t j = 0; j < n_inst; ++j) {
      int32_t it = 0;
      jst[j] = orc_queue_estimate(qs[j], q_p[i], q_d[i], q_t[i], reading, max_iters, &row[j],
                                  &it);
      if (ttft_all) ttft_all[(int64_t)i * n_inst + j] = row[j];
      if (iters_all) iters_all[(int64_t)i * n_inst + j] = it;
    }
    st = first_error(jst, n_inst);
    if (st != ORC_OK) { *failed_query = i; break; }
    const double *arow = acc + (int64_t)i * n_cols;
    const double *crow = cost + (int64_t)i * n_cols;
    int32_t m = tau ? orc_route_row_constrained(n_inst, row, tau[i], arow, crow, col, w_cost)
                    : orc_route_row(n_inst, row, arow, crow, col, w_cost, w_lat, NULL);
    choice[i] = m;
    if (m < 0) {   /* no instance's context limit holds the prompt */
      st = ORC_E_ARG;
      *failed_query = i;
      break;
    }
    if (ttft_chosen) ttft_chosen[i] = row[m];
    if (util_chosen) {
      double pen = w_cost * crow[col[m]];
      util_chosen[i] = arow[col[m]] - pen;
    }
    st = append_tagged(qs[m], q_p[i], q_d[i], queue_cap, i);
    double t_next = (i + 1 < n_q) ? q_t[i + 1] : q_t[i];
    if (st == ORC_OK) st = advance_all(qs, n_inst, t_next, max_iters, jst);
    if (st != ORC_OK) *failed_query = i;
  }
  /* queries without their first token at the end: run a copy of each instance on,
     with no further arrivals, until its last tracked query has it */
  for (int32_t j = 0; j < n_inst && st == ORC_OK && realized; ++j) {
    if (qs[j]->tracked == 0) continue;
    orc_queue *w = q_clone(qs[j]);
    if (!w) { st = ORC_E_ARG; break; }
    for (int64_t k = 0; w->tracked > 0; ++k) {
      if (k == max_iters) { st = ORC_E_ITER; break; }
      orc_queue_step(w, NULL);
    }
    orc_queue_free(w);
  }
  if (st == ORC_OK && out_offsets) {
    int64_t pos = 0;
    out_offsets[0] = 0;
    for (int32_t j = 0; j < n_inst; ++j) {
      if (pos + qs[j]->n > out_cap) { st = ORC_E_CAPACITY; break; }
      orc_queue_get(qs[j], out_rp + pos, out_rd + pos, out_cx + pos, &out_clock[j],
                    &out_iters[j]);
      pos += qs[j]->n;
      out_offsets[j + 1] = (int32_t)pos;
    }
  }
  for (int32_t j = 0; j < n_inst; ++j) orc_queue_free(qs[j]);
  free(qs);
  free(row);
  free(jst);
  return st;
}

/* ---------------------------------------------------------------- LPS */

/*
 * Average-case TTFT without real-time workload information (Sec. 4.2, Eqs. 10 and
 * 11; the appendix on the limited-processor-sharing abstraction, Eqs. 12 and 13).
 * An instance is one server of aggregate capacity mu (queries per ms) shared
 * equally by at most k active queries; further queries wait in FCFS order.  Queries
 * arrive at rate alpha (queries per ms); the model needs alpha < mu.
 *
 *   mode 0, Poisson arrivals and memoryless work (Eqs. 10 and 12):
 *       rho = alpha / mu,   W = rho^k / (mu - alpha)
 *   mode 1, the variability-corrected approximation (Eq. 13), with the mean work
 *   E[Q] = 1/mu and squared coefficients of variation ca2 (inter-arrival times) and
 *   cs2 (work):
 *       E[Q] = 1 / mu,  rho = alpha * E[Q],
 *       W = ((ca2 + cs2) / 2) * ((rho^k * E[Q]) / (1 - rho))
 *   and the TTFT estimate (Eq. 11) of a query of p prompt tokens, with prefill
 *   throughput theta (tokens per ms) and mean decode batch time t_dec (ms):
 *       L = (W + p / theta) + t_dec.
 * rho^k is the product of k factors rho taken left to right.  Each operation is one
 * binary64 round-to-nearest-even operation in the order written.  Parameters outside
 * the model (k < 1, alpha < 0, alpha >= mu, rho >= 1, theta <= 0, t_dec < 0, negative
 * variation coefficients, non-finite values) and p < 1 give NaN, and so does
 * k > 65536 (a concurrency cap far beyond any serving engine's, which bounds the work
 * of the product).
 */
static double pow_left(double r, int32_t k) {
  double x = r;
  for (int32_t m = 1; m < k; ++m) x = x * r;
  return x;
}

double orc_lps_wait(double alpha, double mu, int32_t k, int32_t mode, double ca2, double cs2) {
  if (!(isfinite(alpha) && isfinite(mu) && alpha >= 0.0 && alpha < mu && k >= 1 && k <= 65536))
    return NAN;
  if (mode == 0) {
    const double rho = alpha / mu;
    return pow_left(rho, k) / (mu - alpha);
  }
  if (mode != 1 || !(isfinite(ca2) && isfinite(cs2) && ca2 >= 0.0 && cs2 >= 0.0)) return NAN;
  const double eq = 1.0 / mu;
  const double rho = alpha * eq;
  if (!(rho < 1.0)) return NAN;
  const double h = (ca2 + cs2) / 2.0;
  double t = pow_left(rho, k) * eq;
  t = t / (1.0 - rho);
  return h * t;
}

double orc_lps_ttft(double alpha, double mu, int32_t k, int32_t mode, double ca2, double cs2,
                    double theta, double t_dec, int32_t p) {
  const double w = orc_lps_wait(alpha, mu, k, mode, ca2, cs2);
  if (isnan(w) || p < 1 || !(isfinite(theta) && theta > 0.0) ||
      !(isfinite(t_dec) && t_dec >= 0.0))
    return NAN;
  return (w + (double)p / theta) + t_dec;
}

/* The LPS estimate of every query i < n_q at every instance j < n_inst (parameters
   per instance), into out[i*n_inst + j]. */
void orc_lps_matrix(int32_t n_inst, const double *alpha, const double *mu, const int32_t *k,
                    const double *ca2, const double *cs2, const double *theta,
                    const double *t_dec, int32_t mode, int32_t n_q, const int32_t *p,
                    double *out) {
  for (int32_t i = 0; i < n_q; ++i)
    for (int32_t j = 0; j < n_inst; ++j)
      out[(int64_t)i * n_inst + j] = orc_lps_ttft(alpha[j], mu[j], k[j], mode, ca2[j], cs2[j],
                                                  theta[j], t_dec[j], p[i]);
}

/* ---------------------------------------------------------------- stats */

static int cmp_double(const void *x, const void *y) {
  double a = *(const double *)x, b = *(const double *)y;
  return (a > b) - (a < b);
}

/*
 * Per-scenario summary of a routed trace (the two axes of the utility-latency
 * trade-off, E[U] and E[L], of Sec. 3): mean accuracy, mean cost and mean utility
 * (Eq. 2) at the chosen instances, each a left fold in query order divided by N,
 * and the nearest-rank 50th and 99th percentiles of the chosen TTFTs.
 */
int orc_stats(int32_t n_q, const int32_t *choice, const double *ttft_chosen, const double *acc,
              const double *cost, int32_t n_cols, const int32_t *col, double w_cost,
              double *out5) {
  if (n_q < 1) return ORC_E_ARG;
  double sa = 0.0, sc = 0.0, su = 0.0;
  for (int32_t i = 0; i < n_q; ++i) {
    double ac = acc[(int64_t)i * n_cols + col[choice[i]]];
    double co = cost[(int64_t)i * n_cols + col[choice[i]]];
    double pen = w_cost * co;
    double u = ac - pen;
    sa = sa + ac;
    sc = sc + co;
    su = su + u;
  }
  double *s = (double *)malloc((size_t)n_q * sizeof(double));
  if (!s) return ORC_E_ARG;
  memcpy(s, ttft_chosen, (size_t)n_q * sizeof(double));
  qsort(s, (size_t)n_q, sizeof(double), cmp_double);
  int64_t k50 = ((int64_t)50 * n_q + 99) / 100 - 1;
  int64_t k99 = ((int64_t)99 * n_q + 99) / 100 - 1;
  out5[0] = sa / (double)n_q;
  out5[1] = sc / (double)n_q;
  out5[2] = su / (double)n_q;
  out5[3] = s[k50];
  out5[4] = s[k99];
  free(s);
  return ORC_OK;
}

/* Eq. 4: left fold in query order of the utility (Eq. 2) at the chosen instance
 * for queries whose realised TTFT is within the target, divided by N. */
int orc_ontime_utility(int32_t n_q, const int32_t *choice, const double *ttft_real,
                       const double *tau, const double *acc, const double *cost, int32_t n_cols,
                       const int32_t *col, double w_cost, double *out) {
  if (n_q < 1) return ORC_E_ARG;
  double s = 0.0;
  for (int32_t i = 0; i < n_q; ++i) {
    if (!(ttft_real[i] <= tau[i])) continue;
    double ac = acc[(int64_t)i * n_cols + col[choice[i]]];
    double co = cost[(int64_t)i * n_cols + col[choice[i]]];
    double pen = w_cost * co;
    s = s + (ac - pen);
  }
  *out = s / (double)n_q;
  return ORC_OK;
}
