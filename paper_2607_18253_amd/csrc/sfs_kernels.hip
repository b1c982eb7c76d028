// sfs_kernels.hip -- HIP kernels of the SFS estimator and router for gfx950.
//
//   k_traj   one wave per (scenario, instance): background trajectory up to the
//            batch in which a new FCFS-tail query is first served, plus the
//            decode-only batches after it.  Exact for every tail query: the query
//            is last in FCFS order and only takes budget and slots the background
//            leaves, so all batches before its admission batch are the same with or
//            without it, and after that batch the background only decodes.
//   k_est    one thread per (scenario, instance, chunk of queries), instance
//            fastest: each query's own continuation from the shared trajectory
//            (Sec. 4.1, the first-output-token batch and the TTFT sum).
//   k_route  one wave per (scenario, query) row: Lagrangian utility and argmax
//            with ties to the lowest instance (Sec. 3, Eq. 2).
//   k_commit one wave per (scenario, instance): append the routed query, then
//            replay batches until the clock reaches the next arrival.
//   k_trace_cl  a whole sequential trace in one launch: G workgroups per scenario,
//            one wave per instance (states in LDS), per query a workgroup and a
//            cross-workgroup argmax, then commit + replay + the next estimate from a
//            cached admission point (frontier) of each instance.
//   k_trace_mem the same trace with the states in HBM, for pools too large for LDS.
//   k_drain, k_track_begin, k_track_end  first-token tracking around a trace
//            (realised TTFT of each query in the replay).
//   k_stats  two blocks per scenario: means in query order; nearest-rank p50/p99.
//   k_targets, k_ontime  TTFT targets per query; OnTimeUtility (Eq. 4).
// Under scheduler limits the same calls dispatch to sfs_limits.hip.
#include "sfs_device.h"
#include "sfs_launch.h"
#include "sfs_route.h"
#include "sfs_walk.h"

namespace lar {

// ------------------------------------------------------------------ k_traj
// NC: some instance has d != 0, so the walk keeps context sums per batch; without
// them an instance with d != 0 runs the engine.
template <int KS, bool NC>
__global__ __launch_bounds__(kWave) void k_traj(DevState S, DevParams pr, DevTraj tr, int Z, int I,
                                               const double* t_ptr, double t_val,
                                               int64_t max_iters, int32_t* err) {
  const int qid = blockIdx.x;
  if (qid >= Z * I) return;
  const int j = qid % I;
  const double t = t_ptr ? *t_ptr : t_val;
  const int ln = lane_id();
  __shared__ alignas(16) int stage[stage_words<false>()];
  __shared__ WalkLds<NC> walk_lds;
  const QEnv e = make_env(S, pr, qid, j, stage);
  bool walked;
  if (e.need_C) {
    if constexpr (NC)
      walked = e.need_A ? walk_traj<KS, NC, true, true>(S, e, qid, tr, Z * I, t, max_iters, err,
                                                        walk_lds)
                        : walk_traj<KS, NC, true, false>(S, e, qid, tr, Z * I, t, max_iters, err,
                                                         walk_lds);
    else
      walked = false;
  } else {
    walked = e.need_A ? walk_traj<KS, NC, false, true>(S, e, qid, tr, Z * I, t, max_iters, err,
                                                       walk_lds)
                      : walk_traj<KS, NC, false, false>(S, e, qid, tr, Z * I, t, max_iters, err,
                                                        walk_lds);
  }
  if (walked) return;
  // the engine, for queues outside what the walk covers
  Queue<KS> w;
  w.load(S, e, qid);
  double E = w.clock;
  int ok = 1;
  if (E < t) {
    ok = 0;
    if (ln == 0) set_error(err, kErrState);
  }
  int64_t pre = 0;
  while (ok && !w.tail_admitted_next(e)) {
    if (pre >= max_iters) {   // the admission batch would exceed the cap
      ok = 0;
      break;
    }
    if (w.quiet(e)) {
      pre += w.quiet_run(e, E, __builtin_inf(), pre, max_iters);
      if (pre >= max_iters) continue;
    }
    const StepOut o = w.step(e);
    E = __dadd_rn(E, batch_time(e.k, o.P, o.D, o.C, o.A));
    ++pre;
  }
  const int64_t aP = w.pre_sum, aD = w.n_dec;
  const int64_t aC = e.need_C ? w.c0sum + aD * w.g : 0;
  int64_t aA = 0;
  if (ok) {
    w.refill(e);
    if (e.need_A) aA = w.pre_attention_all(e);
  }
  if (ln == 0) {
    tr.E[qid] = E;
    tr.pre[qid] = (int32_t)pre;
    tr.P[qid] = aP;
    tr.D[qid] = aD;
    tr.C[qid] = aC;
    tr.A[qid] = aA;
    tr.left[qid] = (int)((int64_t)e.k.B - aD - aP);
    tr.ok[qid] = ok;
  }
  const bool readonly = w.nwin == w.n_pre;
  typename Queue<KS>::Tail tl{};
  if (ok) {
    if (readonly) tl = w.tail_begin(e);
    else w.step(e);   // the admission batch itself (background only)
  }
  const int ZI = Z * I;
  const int K = tail_count(tr);
  for (int kk = 0; kk < K; ++kk) {
    int64_t D = 0, C = 0;
    if (ok) {
      if (readonly) {
        D = tl.D;
        C = e.need_C ? tl.c0 + D * (int64_t)(w.g + tl.k) : 0;
        w.tail_next(e, tl);
      } else {
        D = w.n_dec;
        C = e.need_C ? w.c0sum + D * w.g : 0;
        if (D > 0) w.step(e);   // decode-only batch
      }
    }
    if (ln == 0) {
      tr.tailD[(int64_t)kk * ZI + qid] = (int32_t)D;
      tr.tailC[(int64_t)kk * ZI + qid] = C;
    }
  }
}

// ------------------------------------------------------------------ k_est
// One block per (scenario, chunk of kEstChunk queries, 256 instances), one thread
// per instance: the thread keeps its instance's trajectory in registers and walks
// the chunk's queries (their prompt lengths staged in LDS), so each wave writes 64
// consecutive estimates per query.
constexpr int kEstChunk = 16;

__global__ __launch_bounds__(256) void k_est(DevParams pr, DevTraj tr, int Z, int Q, int I,
                                            const int32_t* q_prefill, const double* t_ptr,
                                            double t_val, int max_prompt,
                                            int reading, int64_t max_iters, double* ttft,
                                            int32_t* iters, int32_t* err) {
  __shared__ int s_p[kEstChunk];
  const int n_chunks = (Q + kEstChunk - 1) / kEstChunk;
  const int col_blocks = (I + 255) / 256;
  const int cb = (int)(blockIdx.x % (unsigned)col_blocks);
  const int zc = (int)(blockIdx.x / (unsigned)col_blocks);
  const int c = zc % n_chunks;
  const int z = zc / n_chunks;
  const int q0 = c * kEstChunk;
  const int q1 = Q - q0 < kEstChunk ? Q : q0 + kEstChunk;
  if ((int)threadIdx.x < q1 - q0) s_p[threadIdx.x] = q_prefill[q0 + threadIdx.x];
  __syncthreads();
  const int j = cb * 256 + (int)threadIdx.x;
  if (j >= I) return;
  const int qid = z * I + j;
  const int ZI = Z * I;
  const double t = t_ptr ? *t_ptr : t_val;
  const Coef k = load_coef(pr, j);
  const int ok = tr.ok[qid];
  const double E0 = tr.E[qid];
  const int64_t it0 = (int64_t)tr.pre[qid] + 1;
  const int lft = tr.left[qid];
  // P <= B and D <= M fit in 32 bits
  const int P0 = (int)tr.P[qid], D0 = (int)tr.D[qid];
  const int64_t C0 = tr.C[qid], A0 = tr.A[qid];
  const int K = tail_count(tr);
  // the first decode-tail batch, which nearly every query reaches
  const int D1 = K > 0 ? tr.tailD[qid] : 0;
  const int64_t C1 = K > 0 ? tr.tailC[qid] : 0;
  // Batch time of Sec. 4.1 with batch_time's operations: the context and attention
  // terms are converted only where their coefficient is non-zero (lanes whose
  // instances all have d = 0 or e = 0 skip them); otherwise the term is coef * 0.0.
  const bool need_C = k.d != 0.0, need_A = k.e != 0.0;
  const double dz = __dmul_rn(k.d, 0.0), ez = __dmul_rn(k.e, 0.0);
  auto bt_pd = [&](int P, int D) {
    return __dadd_rn(__dadd_rn(k.a, __dmul_rn(k.b, (double)P)), __dmul_rn(k.c, (double)D));
  };
  auto bt_ca = [&](double t, int64_t C, int64_t A) {
    double td = dz, te = ez;
    if (need_C) td = __dmul_rn(k.d, (double)C);
    if (need_A) te = __dmul_rn(k.e, (double)A);
    return __dadd_rn(__dadd_rn(t, td), te);
  };
  for (int q = q0; q < q1; ++q) {
    const int64_t o = ((int64_t)z * Q + q) * I + j;
    const int p = s_p[q - q0];
    if (p < 1 || p > max_prompt) {
      set_error(err, kErrArg);
      ttft[o] = __builtin_nan("");
      if (iters) iters[o] = -1;
      continue;
    }
    if (!ok) {
      set_error(err, kErrIter);   // a clock behind t was already reported as a state error
      ttft[o] = __builtin_nan("");
      if (iters) iters[o] = -1;
      continue;
    }
    int64_t it = it0;
    // admission batch: background features plus the query's first chunk (context 0)
    const int ch = p < lft ? p : lft;
    double E = __dadd_rn(
        E0, bt_ca(bt_pd(P0 + ch, D0), C0, need_A ? A0 + (int64_t)ch * (ch + 1) / 2 : 0));
    int rem = p - ch;
    int cxq = ch;
    bool done = reading == 1 && rem == 0;
    int kk = 0;
    while (!done) {
      if (kk >= K) {   // cannot happen for p <= max_prompt; guard the tail bounds
        set_error(err, kErrIter);
        E = __builtin_nan("");
        break;
      }
      const int Dk = kk == 0 ? D1 : tr.tailD[(int64_t)kk * ZI + qid];
      const int64_t Ck = kk == 0 ? C1 : tr.tailC[(int64_t)kk * ZI + qid];
      if (rem > 0) {
        const int room = k.B - Dk;
        const int c2 = rem < room ? rem : room;
        E = __dadd_rn(E, bt_ca(bt_pd(c2, Dk), Ck,
                               need_A ? (int64_t)c2 * cxq + (int64_t)c2 * (c2 + 1) / 2 : 0));
        rem -= c2;
        cxq += c2;
        done = reading == 1 && rem == 0;
      } else {
        E = __dadd_rn(E, bt_ca(bt_pd(0, Dk + 1), Ck + cxq, 0));
        done = true;
      }
      ++kk;
      ++it;
    }
    if (it > max_iters) set_error(err, kErrIter);
    ttft[o] = __dsub_rn(E, t);
    if (iters) iters[o] = (int32_t)it;
  }
}

// ------------------------------------------------------------------ k_route
__global__ __launch_bounds__(256) void k_route(int Z, int Q, int I, const double* ttft,
                                              int64_t ttft_zstride, const double* acc,
                                              const double* cost, int n_cols, const int32_t* col,
                                              const double* w_cost, const double* w_lat,
                                              const double* tau, int32_t* choice,
                                              double* chosen_ttft, double* utility,
                                              int64_t out_zstride, int out_q0, int32_t* err) {
  const int wid = uni((int)(threadIdx.x / kWave));   // wave-uniform: keeps per-wave data in SGPRs
  const int row = (int)blockIdx.x * (int)(blockDim.x / kWave) + wid;   // z * Q + q
  if ((int64_t)row >= (int64_t)Z * Q) return;   // (no barrier below: a whole wave leaves)
  const int z = row / Q;
  const int q = row % Q;
  const double wc = w_cost[z];
  const double wl = w_lat[z];
  const double* trow = ttft + (int64_t)z * ttft_zstride + (int64_t)q * I;
  const double* arow = acc + (int64_t)q * n_cols;
  const double* crow = cost + (int64_t)q * n_cols;
  const double tq = tau ? tau[q] : 0.0;
  double bu = 0.0;
  int bj = -1;
  // four instances per lane and pass, their loads issued before any is used
  for (int j0 = lane_id(); j0 < I; j0 += 4 * kWave) {
    int cc[4];
    double tt[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int j = j0 + u * kWave;
      cc[u] = j < I ? col[j] : 0;
      tt[u] = j < I ? trow[j] : 0.0;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int j = j0 + u * kWave;
      if (j < I) {
        const double eq2 = __dsub_rn(arow[cc[u]], __dmul_rn(wc, crow[cc[u]]));
        int k;
        const double v = cand_value(eq2, tt[u], wl, tau, tq, j, &k);
        if (better(v, k, bu, bj)) { bu = v; bj = k; }
      }
    }
  }
  // the row's best over the lanes (DPP; `better` is a total order, so the combining
  // order does not matter)
  lane_best(bu, bj, kWave);
  if (lane_id() == 0) {
    const int64_t o = (int64_t)z * out_zstride + out_q0 + q;
    bj = bj >= 0 ? key_index(bj) : -1;
    if (bj < 0) set_error(err, kErrArg);   // no instance can take the query
    choice[o] = bj;
    if (bj >= 0) {
      if (chosen_ttft) chosen_ttft[o] = trow[bj];
      if (utility) {
        const int c = col[bj];
        utility[o] = __dsub_rn(arow[c], __dmul_rn(wc, crow[c]));
      }
    }
  }
}

// ------------------------------------------------------------------ k_commit
// First-token tracking of a trace's replay: first-token time out[i] (this scenario's
// row; nullptr: off) of the queries tagged tag0 .. tag0 + N - 1.
struct Track {
  double* out;
  int tag0, N, reading;
};

// A quiet stretch of a replay (call when w.quiet(e) holds; clk < t_stop): folds the
// quiet batches before the next decode finish, stopping at t_stop or the cap, and
// returns true when it folded any (the caller re-checks its loop condition), false
// when the next batch must be stepped.  TRK, first token = first decode: when the
// last batch completed prefills, the next batch is their first decode batch; it is
// folded alone and their first tokens recorded at its end.
template <int KS, bool TRK>
__device__ __forceinline__ bool replay_quiet(Queue<KS>& w, const QEnv& e, double& clk,
                                             double t_stop, int64_t& n, int64_t max_iters,
                                             const int32_t* tags, const Track& tk) {
  if constexpr (TRK) {
    if (tk.reading == 0 && w.pend > 0) {
      StepOut pq;
      pq.h0 = w.head; pq.pn = w.pend; pq.nd = 0; pq.pt = w.ptag; pq.pt_ok = w.ptag_ok;
      if (w.quiet_run(e, clk, t_stop, n, n + 1) == 0) return false;
      ++n;
      w.pend = 0;
      w.realize(e, tags, pq, 0, clk, tk.out, tk.tag0, tk.N);
      return true;
    }
  }
  n += w.quiet_run(e, clk, t_stop, n, max_iters);
  return !(clk < t_stop) || n == max_iters;
}

// Append (p, d) when this queue is the chosen one, then replay every batch that
// starts before t; an idle queue's clock jumps to t.  TRK: the query is tracked
// (tag) and the first tokens of the replayed batches are recorded.
template <int KS, bool TRK>
__device__ __forceinline__ void commit_advance(Queue<KS>& w, const QEnv& e, bool chosen, int p,
                                               int d, double t, int qcap, int64_t max_iters,
                                               int32_t* err, int32_t* tags, int tag,
                                               const Track& tk) {
  const int ln = lane_id();
  if (chosen) {
    d = d < 1 ? 1 : d;
    if (p < 1) {
      if (ln == 0) set_error(err, kErrArg);
    } else if (w.n_pre - w.n_part + 1 > qcap) {
      if (ln == 0) set_error(err, kErrCapacity);
    } else {
      if constexpr (TRK) {
        w.append(e, p, d, tags, tag);
        w.ntrk += 1;
      } else {
        w.append(e, p, d);
      }
    }
  }
  double clock = w.clock;
  int64_t n = 0;
  while (w.resident() > 0 && clock < t) {
    if (n == max_iters) {
      if (ln == 0) set_error(err, kErrIter);
      break;
    }
    if (w.quiet(e) && replay_quiet<KS, TRK>(w, e, clock, t, n, max_iters, tags, tk)) continue;
    const StepOut o = w.template step<TRK>(e, tags);
    clock = __dadd_rn(clock, batch_time(e.k, o.P, o.D, o.C, o.A));
    ++n;
    if constexpr (TRK) w.realize(e, tags, o, tk.reading, clock, tk.out, tk.tag0, tk.N);
  }
  if (w.resident() == 0 && clock < t) clock = t;
  w.clock = clock;
  w.iters += n;
}

// Tracked queries still without a first token when the trace ends: a private copy
// of the queue runs on, with no further arrivals, until each has had it.  The
// queue's own state is left as the trace left it.
template <int KS>
__device__ __forceinline__ void drain(Queue<KS> w, const QEnv& e, const int32_t* tags,
                                      const Track& tk, int64_t max_iters, int32_t* err) {
  double clock = w.clock;
  int64_t n = 0;
  while (w.ntrk > 0) {
    if (n == max_iters) {
      if (lane_id() == 0) set_error(err, kErrIter);
      break;
    }
    if (w.quiet(e) &&
        replay_quiet<KS, true>(w, e, clock, __builtin_inf(), n, max_iters, tags, tk))
      continue;
    const StepOut o = w.template step<true>(e, tags);
    clock = __dadd_rn(clock, batch_time(e.k, o.P, o.D, o.C, o.A));
    ++n;
    w.realize(e, tags, o, tk.reading, clock, tk.out, tk.tag0, tk.N);
  }
}

template <int KS>
__global__ __launch_bounds__(kWave) void k_commit(DevState S, DevParams pr, int Z, int I,
                                                 const int32_t* choice, int64_t choice_zstride,
                                                 const int32_t* qp_ptr, const int32_t* qd_ptr,
                                                 int32_t qp_val, int32_t qd_val,
                                                 const double* t_ptr, double t_val,
                                                 int64_t max_iters, int32_t* err) {
  const int qid = blockIdx.x;
  if (qid >= Z * I) return;
  const int z = qid / I;
  const int j = qid % I;
  const double t = t_ptr ? *t_ptr : t_val;
  __shared__ alignas(16) int stage[stage_words<false>()];
  const QEnv e = make_env(S, pr, qid, j, stage);
  Queue<KS> w;
  w.load(S, e, qid);
  const bool chosen = choice && choice[(int64_t)z * choice_zstride] == j;
  const int p = qp_ptr ? *qp_ptr : qp_val;
  const int d = qd_ptr ? *qd_ptr : qd_val;
  const Track off{nullptr, 0, 0, 0};
  commit_advance<KS, false>(w, e, chosen, p, d, t, S.qcap, max_iters, err, nullptr, -1, off);
  w.store(S, e, qid);
}

// ------------------------------------------------------------------ k_trace
// From a state whose next batch admits a new tail query (clock folded to E after
// `it` batches): the admission batch -- the whole prefill list, the decodes, and the
// query's first chunk at context 0 -- then the query's further chunks and its first
// decode batch, over the background's decode-only batches.  The background comes
// from Queue::tail_begin/tail_next (read-only) when the whole prefill list is in the
// window, else from stepping the (private) state.
template <int KS>
__device__ __forceinline__ double finish_estimate(Queue<KS>& w, const QEnv& e, double E,
                                                  int64_t it, int p, double t, int reading,
                                                  int64_t max_iters, int32_t* err,
                                                  int64_t* it_out = nullptr) {
  const int ln = lane_id();
  const int aP = (int)w.pre_sum, aD = w.n_dec;
  const int64_t aC = e.need_C ? w.c0sum + (int64_t)aD * w.g : 0;
  const int64_t aA = e.need_A ? w.pre_attention_all(e) : 0;
  const int left = e.k.B - aD - aP;
  const int ch = p < left ? p : left;
  E = __dadd_rn(E, batch_time(e.k, aP + ch, aD, aC, aA + (int64_t)ch * (ch + 1) / 2));
  ++it;
  int rem = p - ch;
  int64_t cxq = ch;
  bool done = reading == 1 && rem == 0;
  if (!done) {
    const bool readonly = w.nwin == w.n_pre;
    typename Queue<KS>::Tail tl{};
    if (readonly) tl = w.tail_begin(e); else w.step(e);
    while (!done) {
      int Dk;
      int64_t Ck;
      if (readonly) {
        Dk = (int)tl.D;
        Ck = e.need_C ? tl.c0 + (int64_t)Dk * (w.g + tl.k) : 0;
      } else {
        Dk = w.n_dec;
        Ck = e.need_C ? w.c0sum + (int64_t)Dk * w.g : 0;
      }
      if (rem > 0) {
        const int room = e.k.B - Dk;
        const int c2 = rem < room ? rem : room;
        E = __dadd_rn(E, batch_time(e.k, c2, Dk, Ck, (int64_t)c2 * cxq + (int64_t)c2 * (c2 + 1) / 2));
        rem -= c2;
        cxq += c2;
        done = reading == 1 && rem == 0;
      } else {
        E = __dadd_rn(E, batch_time(e.k, 0, Dk + 1, Ck + cxq, 0));
        done = true;
      }
      ++it;
      if (!done) {
        if (readonly) w.tail_next(e, tl);
        else if (Dk > 0) w.step(e);
      }
    }
  }
  if (it > max_iters && ln == 0) set_error(err, kErrIter);
  if (it_out) *it_out = it;
  return __dsub_rn(E, t);
}

// SFS estimate of a query (p prompt tokens, arrival t) at one queue; the queue is
// not modified.  Returns NaN (and sets the error) when it cannot.
template <int KS>
__device__ __forceinline__ double estimate(const Queue<KS>& q, const QEnv& e, int p, double t,
                                           int reading, int64_t max_iters, int32_t* err,
                                           int64_t* it_out = nullptr) {
  const int ln = lane_id();
  if (q.clock < t) {
    if (ln == 0) set_error(err, kErrState);
    return __builtin_nan("");
  }
  Queue<KS> w = q;
  double E = w.clock;
  int64_t it = 0;
  while (!w.tail_admitted_next(e)) {
    if (it >= max_iters) {
      if (ln == 0) set_error(err, kErrIter);
      return __builtin_nan("");
    }
    if (w.quiet(e)) {
      it += w.quiet_run(e, E, __builtin_inf(), it, max_iters);
      if (it >= max_iters) continue;
    }
    const StepOut o = w.step(e);
    E = __dadd_rn(E, batch_time(e.k, o.P, o.D, o.C, o.A));
    ++it;
  }
  w.refill(e);
  return finish_estimate(w, e, E, it, p, t, reading, max_iters, err, it_out);
}

// The same trace for pools too large to keep in registers: each owned instance's
// state is loaded from HBM (L2) when it is needed and written back after its commit.
// Wave w owns instances j = w + v*nw; lane v holds the inputs of the v-th one.
// TRK: the replay also reports each query's realised TTFT.
template <int KS, int NW, bool TRK>
__global__ __launch_bounds__(NW * kWave) void k_trace_mem(LAR_TRACE_PARAMS) {
  __shared__ double s_u[2][NW], s_t[2][NW], s_q[2][NW];
  __shared__ int s_j[2][NW];
  __shared__ alignas(16) int stage[NW][stage_words<TRK>()];
  const int z = blockIdx.x;
  const int wid = uni((int)(threadIdx.x / kWave));   // wave-uniform: keeps per-wave data in SGPRs
  const int nw = blockDim.x / kWave;
  const int ln = lane_id();
  const double wc = w_cost[z];
  const double wl = w_lat[z];
  const int j_l = wid + ln * nw;
  const bool own_l = j_l < I;
  const int col_l = own_l ? pr.col[j_l] : 0;
  QueryIn nx = fetch_query(0, N, qp, qd, qt, t_after, tau, acc, cost, n_cols, col_l, own_l);
  const Track tk{TRK ? realized + (int64_t)z * N : nullptr, tag0, N, reading};
  unsigned long long wbatch = 0;   // batches of this wave's estimates
  for (int i = 0; i < N; ++i) {
    const QueryIn q = nx;
    nx = fetch_query(i + 1, N, qp, qd, qt, t_after, tau, acc, cost, n_cols, col_l, own_l);
    const bool p_ok = q.p >= 1 && q.p <= max_prompt;
    if (!p_ok && threadIdx.x == 0) set_error(err, kErrArg);
    double bu = 0.0, bt = 0.0, bq = 0.0;
    int bj = -1;
    for (int v = 0, j = wid; j < I; ++v, j += nw) {
      const QEnv e = make_env(S, pr, z * I + j, j, stage[wid]);
      Queue<KS> w;
      w.load(S, e, z * I + j);
      int64_t it = 0;
      const double ttft = p_ok ? estimate(w, e, q.p, q.t, reading, max_iters, err, &it)
                               : __builtin_nan("");
      wbatch += it;
      double eq2;
      int k;
      const double u = utility_lane(q, v, wc, wl, tau, ttft, j, &k, &eq2, i, acc, cost,
                                      n_cols, v < kWave ? 0 : pr.col[j]);
      if (better(u, k, bu, bj)) { bu = u; bj = k; bt = ttft; bq = eq2; }
    }
    const int m = trace_pick<NW>(bu, bj, bt, bq, i, z, N, choice, chosen_ttft, utility, s_u,
                                 s_t, s_q, s_j);
    if (m < 0 && threadIdx.x == 0) set_error(err, kErrArg);   // no candidate
    for (int j = wid; j < I; j += nw) {
      const QEnv e = make_env(S, pr, z * I + j, j, stage[wid]);
      Queue<KS> w;
      int32_t* tags = TRK ? S.r_tag + (int64_t)(z * I + j) * S.rcap : nullptr;
      w.template load<TRK>(S, e, z * I + j, tags);
      commit_advance<KS, TRK>(w, e, j == m, q.p, q.d, q.tn, S.qcap, max_iters, err, tags,
                              tag0 + i, tk);
      w.template store<TRK>(S, e, z * I + j);
    }
  }
  if (work && lane_id() == 0) atomicAdd(work + z, wbatch);
}

// Zeroes the per-scenario estimate-batch counters before a trace.
__global__ void k_clear_work(unsigned long long* w, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) w[i] = 0ull;
}

// Clears the exchange posts (tags included) of every scenario before a trace.
__global__ void k_clear_exchange(uint64_t* xs, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) xs[i] = 0;
}

// ------------------------------------------------------------------ frontier cache
// For a queue whose next batch would not admit a new tail query (a backlog), the
// state F at the admission point of such a query does not depend on the query (the
// query is last in FCFS order), and neither do the clock folded up to F, the
// background features of the admission batch, or the decode-only batches after it.
// The cache keeps F in LDS and those values in registers (tail batch k in lane
// k - 1), so an estimate is a short fold over them.  F stays valid while the world
// has not run past it; when the queue receives a query, F + query is walked to its
// next admission point (again exact by the FCFS argument).
struct FCache {
  bool valid;
  // Summary of the instance state when it admits a tail query in its very next
  // batch (no frontier needed): its batch counter and clock in g and E, the
  // admission batch's background in aP .. aA, and the decode batch after it (every
  // request left decodes there) in sD1 / sC1.  Valid while the state is unchanged.
  bool summ;
  int sD1;
  int64_t sC1;
  int snf;         // summary: the next batch in which a decoding request finishes
                   // (-1: not taken yet; replay_summary takes it from the state in LDS)
  int g;           // batch counter of F
  double E;        // clock folded up to F
  int aP, aD, left;
  int64_t aC, aA;  // admission-batch background features
  int tD;          // lane k: decode tokens of tail batch k + 1
  int64_t tC;      // lane k: their context sum
  int depth;       // tail batches held (lanes 0 .. depth - 1; at least the tail depth K)
};

__device__ __forceinline__ int64_t read_lane_i64(int64_t v, int l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(uint64_t)v, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), l);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Summary of the admission batch of w (which must satisfy tail_admitted_next).
template <int KS>
__device__ __forceinline__ void admission_summary(FCache& fc, const Queue<KS>& w, const QEnv& e,
                                                  double E) {
  fc.g = w.g;
  fc.E = E;
  fc.aP = (int)w.pre_sum;
  fc.aD = w.n_dec;
  fc.aC = e.need_C ? w.c0sum + (int64_t)w.n_dec * w.g : 0;
  fc.aA = e.need_A ? w.pre_attention_all(e) : 0;
  fc.left = e.k.B - fc.aD - fc.aP;
}

// Suffix sums over the lanes (lane l gets the sum over lanes l .. 63): the total
// minus the inclusive prefix, plus the lane's own value.
__device__ __forceinline__ int suffix_sum32(int x) {
  const int incl = scan_add32(x);
  return lane_last(incl) - incl + x;
}

__device__ __forceinline__ int64_t suffix_sum64(int64_t x) {
  const int64_t incl = scan_add64(x);
  const uint32_t t_hi = (uint32_t)lane_last((int)(uint32_t)((uint64_t)incl >> 32));
  const uint32_t t_lo = (uint32_t)lane_last((int)(uint32_t)(uint64_t)incl);
  const int64_t tot = (int64_t)(((uint64_t)t_hi << 32) | t_lo);
  return tot - incl + x;
}

// Record the decode-only tail read-only from w (whole prefill list in the window):
// lane k - 1 gets D and C of tail batch k (batch g + 1 + k), k = 1 .. kmax.  After the
// admission batch g + 1 every request decodes until its last batch: a decoding
// request until its slot's dl, a list entry until g + 1 + rd.  So a request is in
// tail batches 1 .. k_last, and D_k, and the cx0 sum behind C_k, are suffix sums
// over k_last: requests with k_last < kmax are binned in LDS (the staging area), the
// rest (most of them) counted with one wave reduction and put in the last bin.
template <int KS>
__device__ __forceinline__ void tail_readonly(FCache& fc, const Queue<KS>& w, const QEnv& e,
                                              int kmax) {
  const int ln = lane_id();
  const bool need_C = e.need_C;
  const int g1 = w.g + 1;   // the admission batch
  int* cnt = e.stg;                                                            // [64]
  unsigned long long* csum = reinterpret_cast<unsigned long long*>(e.stg + kWave);  // [64]
  cnt[ln] = 0;
  csum[ln] = 0ull;
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  int far_n = 0;
  int64_t far_c = 0;
  const int idx = ln - w.woff;
  if constexpr (KS >= 8) {
    // wide queues (the tail is taken on most chosen visits): the far requests are
    // counted by ballots and their cx0 summed per lane with selects; only the near
    // ones branch, to their bins
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int kl = w.dl[s] - g1;   // >= 1: survives the admission batch
      const bool far = kl >= kmax;
      far_n += popc(ballot(far));
      if (need_C) far_c += far ? (int64_t)w.dc[s] : 0;
      if (kl >= 1 && !far) {
        atomicAdd(&cnt[kl - 1], 1);
        if (need_C) atomicAdd(&csum[kl - 1], (unsigned long long)(int64_t)w.dc[s]);
      }
    }
    const bool ent = idx >= 0 && idx < w.nwin;   // rd >= 1
    const bool efar = ent && w.wrd >= kmax;
    far_n += popc(ballot(efar));
    if (need_C) far_c += efar ? (int64_t)(w.wcx + w.wrp) - g1 : 0;
    if (ent && !efar) {
      atomicAdd(&cnt[w.wrd - 1], 1);
      if (need_C) atomicAdd(&csum[w.wrd - 1], (unsigned long long)((int64_t)(w.wcx + w.wrp) - g1));
    }
    far_n = uni(far_n);
  } else {
    // narrow queues take the tail rarely; this form keeps their kernels' register
    // allocation (the form above measured slower there through it)
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int kl = w.dl[s] - g1;
      if (kl >= kmax) {
        ++far_n;
        far_c += w.dc[s];
      } else if (kl >= 1) {
        atomicAdd(&cnt[kl - 1], 1);
        if (need_C) atomicAdd(&csum[kl - 1], (unsigned long long)(int64_t)w.dc[s]);
      }
    }
    if (idx >= 0 && idx < w.nwin) {
      const int64_t c0 = (int64_t)(w.wcx + w.wrp) - g1;
      if (w.wrd >= kmax) {
        ++far_n;
        far_c += c0;
      } else {
        atomicAdd(&cnt[w.wrd - 1], 1);
        if (need_C) atomicAdd(&csum[w.wrd - 1], (unsigned long long)c0);
      }
    }
    far_n = wave_sum32(far_n);
  }
  if (need_C) far_c = wave_sum64(far_c);
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  int D = ln < kmax ? cnt[ln] : 0;
  int64_t c0 = need_C && ln < kmax ? (int64_t)csum[ln] : 0;
  if (ln == kmax - 1) {
    D += far_n;
    c0 += far_c;
  }
  __builtin_amdgcn_wave_barrier();   // the staging area is free again
  D = suffix_sum32(D);
  if (need_C) c0 = suffix_sum64(c0);
  fc.tD = ln < kmax ? D : 0;
  fc.tC = need_C && ln < kmax ? c0 + (int64_t)D * (w.g + ln + 1) : 0;
}

// The tail of F' (F + query walked to its next admission point, g' = w.g) from F's
// tail: F' holds F's background -- the same requests, decode-only after F's admission
// batch -- plus the query, so its tail batch k is F's tail batch k + sh (sh = g' - g_F
// batches between the two admission batches) plus the query's own term.  The query is
// the list's last entry (all of its prefill in the admission batch, then rd decodes) or
// a decoding request (its slot found by its sequence number).  F's tail must hold
// sh + K batches; F' then holds sh fewer.
template <int KS>
__device__ __forceinline__ void tail_shift(FCache& fc, const Queue<KS>& w, const QEnv& e, int sh,
                                           int seqq) {
  const int ln = lane_id();
  const int depth = fc.depth - sh;
  const int src = min(ln + sh, kWave - 1);
  int D = __shfl(fc.tD, src, kWave);
  int64_t C = 0;
  if (e.need_C) {
    const uint32_t lo = (uint32_t)__shfl((int)(uint32_t)(uint64_t)fc.tC, src, kWave);
    const uint32_t hi = (uint32_t)__shfl((int)(uint32_t)((uint64_t)fc.tC >> 32), src, kWave);
    C = (int64_t)(((uint64_t)hi << 32) | lo);
  }
  const int g1 = w.g + 1;   // the admission batch
  int kl = 0;               // the query decodes in tail batches 1 .. kl
  int64_t c0 = 0;           // its context in batch b is c0 + b - 1
  if (w.n_pre > 0) {
    const int q = w.woff + w.n_pre - 1;
    kl = __builtin_amdgcn_readlane(w.wrd, q);
    c0 = (int64_t)(__builtin_amdgcn_readlane(w.wcx, q) + __builtin_amdgcn_readlane(w.wrp, q)) - g1;
  } else {
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const uint64_t m = ballot(w.ds[s] == seqq && w.dl[s] > w.g);
      if (m) {
        const int l = __builtin_ctzll(m);
        kl = __builtin_amdgcn_readlane(w.dl[s], l) - g1;
        c0 = __builtin_amdgcn_readlane(w.dc[s], l);
      }
    }
  }
  if (ln < kl) {
    D += 1;
    if (e.need_C) C += c0 + (int64_t)(w.g + ln + 1);
  }
  fc.tD = ln < depth ? D : 0;
  fc.tC = e.need_C && ln < depth ? C : 0;
  fc.depth = depth;
}

// What the estimate needs of the instance after a visit: its batch counter and
// clock, and whether the working copy still equals it with the whole prefill list in
// the window and the query admitted in the very next batch (then the estimate reads
// the tail straight from it).
struct VisitOut {
  int g;
  double clock;
  bool direct;
};

// The admission batch of a summarised state (F, or the instance's own state under a
// summary) stepped from the summary, for that state + query (the list's last entry,
// p prompt tokens) with the whole list in the window: the batch serves every entry
// in full and gives the query min(p, left) tokens, so its features are the
// summary's plus the query's chunk, and the decoders alive after it are those of
// the first decode batch after it (D1 of them, context sum C1), plus the query when
// its prefill completes.  The completed entries take free decode slots in the order
// Queue::step gives them (staged in LDS), and the window and list move as there.
// The result is step()'s.
template <int KS>
__device__ __forceinline__ void admission_step(Queue<KS>& wk, const FCache& fc, const QEnv& e,
                                               int p, double& clk, int D1, int64_t C1) {
  const int ln = lane_id();
  const int g1 = wk.g + 1;
  const int ch = min(p, fc.left);
  clk = __dadd_rn(clk, batch_time(e.k, fc.aP + ch, fc.aD, fc.aC,
                                  e.need_A ? fc.aA + (int64_t)ch * (ch + 1) / 2 : 0));
  const bool qfull = ch == p;
  const int n_full = wk.n_pre - (qfull ? 0 : 1);
  int* stg = e.stg;
  const int idx = ln - wk.woff;
  if (idx >= 0 && idx < n_full) {
    stg[idx] = g1 + wk.wrd;
    stg[kWave + idx] = wk.wcx + wk.wrp - g1;
    stg[2 * kWave + idx] = wk.wseq;
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  int placed = 0;
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    if (placed < n_full) {
      const bool fr = wk.dl[s] <= g1;
      const uint64_t fm = ballot(fr);
      const int r = placed + mbcnt(fm);
      if (fr && r < n_full) {
        wk.dl[s] = stg[r]; wk.dc[s] = stg[kWave + r]; wk.ds[s] = stg[2 * kWave + r];
      }
      placed += popc(fm);
    }
  }
  __builtin_amdgcn_wave_barrier();
  wk.n_dec = D1 + (qfull ? 1 : 0);
  if (e.need_C) wk.c0sum = C1 - (int64_t)D1 * g1 + (qfull ? (int64_t)(p - g1) : 0);
  wk.woff += n_full;
  wk.nwin -= n_full;
  wk.head += n_full;
  if (wk.head >= e.rcap) wk.head -= e.rcap;
  wk.n_pre -= n_full;
  if (qfull) {
    wk.n_part = 0;
    wk.pre_sum = 0;
  } else {
    if (ln == wk.woff) {
      wk.wrp -= ch;
      wk.wcx += ch;
    }
    wk.n_part = 1;
    wk.pre_sum = p - ch;
  }
  wk.g = g1;
}

// F + query (p prompt tokens, rdq >= 1 decodes) walked towards its next admission
// point without stepping the background batch by batch.  F's admission batch is
// stepped: it serves every list entry of F in full and gives the query its first
// chunk.  After it the background is decode-only, and its batches are the cached
// tail of F (lane k - 1: decode tokens and context sum of tail batch k), which the
// query does not change (it is last in FCFS order and takes only what is left).  The
// query's chunks, then its decodes, are folded on top of those batches, one batch
// time each in batch order, until the state would admit a new tail query; then the
// queue is brought to that batch in one go (decoding requests are lazy: the batch
// counter moves and the live slots are recounted; the query, once its prefill is
// complete, takes a free slot).  Features, batch times and the resulting state are
// those of stepping every batch.  Stops early, at the last folded batch, when the
// cached batches run out or the cap is reached; the stepped walk then continues.
template <int KS>
__device__ __forceinline__ void walk_fast(Queue<KS>& wk, const FCache& fc, const QEnv& e, int p,
                                          int rdq, double& clk, int64_t& n, int kmax,
                                          int64_t max_iters) {
  const Coef& kc = e.k;
  const int ln = lane_id();
  if (wk.tail_admitted_next(e) || n >= max_iters) return;
  // F's admission batch, with the query's first chunk
  if (wk.nwin == wk.n_pre) {
    admission_step(wk, fc, e, p, clk, __builtin_amdgcn_readlane(fc.tD, 0), read_lane_i64(fc.tC, 0));
  } else {
    const StepOut o = wk.step(e);
    clk = __dadd_rn(clk, batch_time(kc, o.P, o.D, o.C, o.A));
  }
  ++n;
  if (wk.tail_admitted_next(e)) return;
  const int gA = wk.g;
  // the query: the list's only entry, or decoding since the admission batch
  int rem = 0, cxq = 0, k_done = -1, cx_done = 0, ctxq = 0;
  if (wk.n_pre > 0) {
    rem = (int)wk.pre_sum;
    cxq = __builtin_amdgcn_readlane(wk.wcx, wk.woff);
  } else {
    k_done = 0;
    cx_done = p;
    ctxq = p;
  }
  int folded = 0;
  for (int k = 1; k < kmax && n < max_iters; ++k) {   // lanes k - 1 and k are read
    const int Dk = __builtin_amdgcn_readlane(fc.tD, k - 1);
    int P = 0, D = Dk;
    int64_t C = read_lane_i64(fc.tC, k - 1), A = 0;
    if (rem > 0) {
      const int c = min(rem, kc.B - Dk);
      P = c;
      A = (int64_t)c * cxq + (int64_t)c * (c + 1) / 2;
      rem -= c;
      cxq += c;
      if (rem == 0) {
        k_done = k;
        cx_done = cxq;
        ctxq = cxq;
      }
    } else if (k_done >= 0 && k <= k_done + rdq) {   // the query decodes
      D += 1;
      C += ctxq;
      ctxq += 1;
    }
    clk = __dadd_rn(clk, batch_time(kc, P, D, e.need_C ? C : 0, e.need_A ? A : 0));
    ++n;
    folded = k;
    // the state for the next batch: the background's decoders of tail batch k + 1,
    // the query as a decoder then or as the list's only entry
    const int nd = __builtin_amdgcn_readlane(fc.tD, k) +
                   ((k_done >= 0 && k + 1 <= k_done + rdq) ? 1 : 0);
    if (nd + (rem > 0 ? 1 : 0) < kc.M && (int64_t)nd + rem < (int64_t)kc.B) break;
  }
  if (folded == 0) return;
  const int gN = gA + folded;
  if (k_done >= 1) {   // prefill completed during the fold: off the list, into a slot
    const int seqq = __builtin_amdgcn_readlane(wk.wseq, wk.woff);
    wk.woff += 1;
    wk.nwin -= 1;
    wk.head = wk.head + 1 == e.rcap ? 0 : wk.head + 1;
    wk.n_pre = 0;
    wk.n_part = 0;
    wk.pre_sum = 0;
    const int gc = gA + k_done;
    if (gc + rdq > gN) {   // still decoding; at most M - 1 others run, so a slot is free
      bool placed = false;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const uint64_t fm = ballot(wk.dl[s] <= gN);
        if (!placed && fm) {
          if (ln == __builtin_ctzll(fm)) {
            wk.dl[s] = gc + rdq;
            wk.dc[s] = cx_done - gc;
            wk.ds[s] = seqq;
          }
          placed = true;
        }
      }
    }
  } else if (rem > 0) {
    if (ln == wk.woff) {
      wk.wrp = rem;
      wk.wcx = cxq;
    }
    wk.pre_sum = rem;
  }
  wk.g = gN;
  int nd = 0;
  int64_t c0 = 0;
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const bool live = wk.dl[s] > gN;
    nd += popc(ballot(live));
    if (e.need_C && live) c0 += wk.dc[s];
  }
  wk.n_dec = nd;
  if (e.need_C) wk.c0sum = wave_sum64(c0);
}

// One visit of a wave to one owned queue for one query.  wk enters as the instance
// state (loaded from SL); the query is appended if it was routed here, the instance
// is replayed to tn and written back to SL (unless nothing changed), and the
// frontier cache (state F in LDS) is kept in step.
// Every batch -- replayed, walked to a new admission point, or recorded as tail --
// runs through the single Queue::step / quiet_run below, on wk.
template <int KS, bool TRK>
__device__ __forceinline__ VisitOut visit(Queue<KS>& wk, FCache& fc, const QEnv& e, bool chosen,
                                          int p, int d, double tn, int qcap, int kmax,
                                          int64_t max_iters, int32_t* err, LdsQueue<KS>& SL,
                                          LdsTags* SLt, LdsQueue<KS>& F, int32_t* tags, int tag,
                                          const Track& tk) {
  const int ln = lane_id();
  VisitOut vo;
  vo.direct = false;
  bool joined = false;
  if (chosen) {
    d = d < 1 ? 1 : d;
    if (p < 1) {
      if (ln == 0) set_error(err, kErrArg);
    } else if (wk.n_pre - wk.n_part + 1 > qcap) {
      if (ln == 0) set_error(err, kErrCapacity);
    } else {
      if constexpr (TRK) {
        wk.append(e, p, d, tags, tag);
        wk.ntrk += 1;
      } else {
        wk.append(e, p, d);
      }
      joined = true;
    }
  }
  enum { kReplay, kWalk, kTail };
  int phase = kReplay;
  const double clk0 = wk.clock;
  double clk = clk0;
  double stop_t = tn;
  int64_t n = 0;
  int kk = -1;
  int shift_g = -1;   // (wide queues) g of F when the walk starts from it, for the tail shift
  int seqq = 0;
  // (narrow queues, untracked) the query joined a state under a current summary: the
  // replay's first batch is that state's admission batch
  bool summ_step = false;
  if constexpr (KS <= 4 && !TRK)
    summ_step = joined && fc.summ && fc.g == wk.g && fc.E == clk0 && wk.nwin == wk.n_pre;
  for (;;) {
    bool stop;
    if (phase == kReplay) {
      stop = !(wk.resident() > 0 && clk < stop_t);
      if (!stop && n == max_iters) {
        if (ln == 0) set_error(err, kErrIter);
        stop = true;
      }
    } else if (phase == kWalk) {
      stop = wk.tail_admitted_next(e) || n == max_iters;
    } else {
      stop = kk == kmax;
    }
    if (stop) {
      if (phase == kReplay) {
        if (wk.resident() == 0 && clk < stop_t) clk = stop_t;
        wk.clock = clk;
        wk.iters += n;
        if (joined || n > 0 || clk != clk0) wk.template to_lds<TRK>(SL, SLt);   // it moved on
        vo.g = wk.g;
        vo.clock = clk;
        // the instance ran the admission batch, or sat idle at F and its clock jumped
        if (fc.valid && (wk.g > fc.g || (wk.g == fc.g && clk != fc.E))) fc.valid = false;
        const bool from_f = joined && fc.valid;
        if (from_f) {
          wk.from_lds(F);
          if constexpr (KS >= 8) {
            shift_g = fc.g;
            seqq = wk.next_seq;
          }
          wk.append(e, p, d);   // F shares the instance's ring: same slot, entry and tag
          clk = fc.E;
        } else if (!fc.valid) {
          wk.refill(e);
          if (wk.tail_admitted_next(e) && wk.nwin == wk.n_pre) {
            vo.direct = true;   // estimate straight from the instance state
            break;
          }
        } else {
          break;
        }
        phase = kWalk;
        stop_t = __builtin_inf();
        n = 0;
        // (pools of <= 256 slots per queue step cheaply enough; the larger code would
        // cost them more than the fold saves)
        if constexpr (KS >= 8)
          if (from_f) walk_fast(wk, fc, e, p, d, clk, n, kmax, max_iters);
        continue;
      }
      if (phase == kWalk) {
        if (!wk.tail_admitted_next(e)) {   // the cap ran out
          fc.valid = false;
          if (ln == 0) set_error(err, kErrIter);
          break;
        }
        wk.refill(e);
        admission_summary(fc, wk, e, clk);
        fc.valid = true;
        wk.to_lds(F);
        if (wk.nwin == wk.n_pre) {
          if constexpr (KS >= 8) {
            // (wide queues walk on most chosen visits: F's tail is shifted while it
            // holds enough batches, else taken afresh to the full lane width)
            if (shift_g >= 0 && fc.depth - (wk.g - shift_g) >= kmax) {
              tail_shift(fc, wk, e, wk.g - shift_g, seqq);
            } else {
              tail_readonly(fc, wk, e, kWave);
              fc.depth = kWave;
            }
          } else {
            tail_readonly(fc, wk, e, kmax);
          }
          break;
        }
        if constexpr (KS >= 8) fc.depth = kmax;
        phase = kTail;   // step the admission batch, then record kmax decode-only batches
        kk = -1;
        continue;
      }
      break;
    }
    if constexpr (KS <= 4 && !TRK) {
      if (summ_step && phase == kReplay) {   // the replay steps its first batch
        summ_step = false;
        admission_step(wk, fc, e, p, clk, fc.sD1, fc.sC1);
        ++n;
        continue;
      }
    }
    if (phase != kTail && wk.quiet(e)) {
      // a quiet run ends before the batch in which a decode finishes (or at the stop
      // time or the cap); that batch is then stepped below
      if (phase == kReplay) {
        if (replay_quiet<KS, TRK>(wk, e, clk, stop_t, n, max_iters, tags, tk)) continue;
      } else {
        n += wk.quiet_run(e, clk, stop_t, n, max_iters);
        if (!(clk < stop_t) || n == max_iters) continue;
      }
    }
    // (one step for every phase: TRK bookkeeping on the walk's copies is harmless)
    const StepOut o = wk.template step<TRK>(e, tags);
    if (phase != kTail) {
      clk = __dadd_rn(clk, batch_time(e.k, o.P, o.D, o.C, o.A));
      ++n;
      if constexpr (TRK)
        if (phase == kReplay)
          wk.realize(e, tags, o, tk.reading, clk, tk.out, tk.tag0, tk.N);
    } else {
      if (kk >= 0 && ln == kk) { fc.tD = o.D; fc.tC = o.C; }
      ++kk;
    }
  }
  return vo;
}

// SFS estimate of a query (p tokens, arrival t) from the admission batch summary and
// the decode-only tail: from the cache (tail in lanes) or, when the visit left the
// instance state in S with the query admitted in its very next batch, read-only
// from S.
template <int KS>
__device__ __forceinline__ double estimate_visit(const FCache& fc, const Queue<KS>& S,
                                                 const VisitOut& vo, const QEnv& e, int p,
                                                 double t, int reading, int kmax,
                                                 int64_t max_iters, int32_t* err,
                                                 int64_t* it_out = nullptr) {
  const int ln = lane_id();
  if (vo.clock < t) {
    if (ln == 0) set_error(err, kErrState);
    return __builtin_nan("");
  }
  const Coef& k = e.k;
  double E;
  int64_t it;
  int aP, aD, left;
  int64_t aC, aA;
  const bool cached = fc.valid;
  if (!cached && !vo.direct) return __builtin_nan("");   // the walk's cap ran out: error set
  if (cached) {
    E = fc.E; it = (int64_t)(fc.g - vo.g) + 1;
    aP = fc.aP; aD = fc.aD; left = fc.left; aC = fc.aC; aA = fc.aA;
  } else {
    E = S.clock; it = 1;
    aP = (int)S.pre_sum; aD = S.n_dec; left = k.B - aD - aP;
    aC = e.need_C ? S.c0sum + (int64_t)aD * S.g : 0;
    aA = e.need_A ? S.pre_attention_all(e) : 0;
  }
  const int ch = p < left ? p : left;
  E = __dadd_rn(E, batch_time(k, aP + ch, aD, aC, aA + (int64_t)ch * (ch + 1) / 2));
  int rem = p - ch;
  int64_t cxq = ch;
  bool done = reading == 1 && rem == 0;
  typename Queue<KS>::Tail tl{};
  if (!cached && !done) tl = S.tail_begin(e);
  int kk = 0;
  while (!done) {
    int Dk;
    int64_t Ck;
    if (cached) {
      if (kk >= kmax) {   // more tail batches than recorded (kmax bounds every prompt)
        if (ln == 0) set_error(err, kErrIter);
        return __builtin_nan("");
      }
      Dk = __builtin_amdgcn_readlane(fc.tD, kk);
      Ck = read_lane_i64(fc.tC, kk);
    } else {
      Dk = (int)tl.D;
      Ck = e.need_C ? tl.c0 + (int64_t)Dk * (S.g + tl.k) : 0;
    }
    if (rem > 0) {
      const int room = k.B - Dk;
      const int c2 = rem < room ? rem : room;
      E = __dadd_rn(E, batch_time(k, c2, Dk, Ck, (int64_t)c2 * cxq + (int64_t)c2 * (c2 + 1) / 2));
      rem -= c2;
      cxq += c2;
      done = reading == 1 && rem == 0;
    } else {
      E = __dadd_rn(E, batch_time(k, 0, Dk + 1, Ck + cxq, 0));
      done = true;
    }
    ++kk;
    ++it;
    if (!done && !cached) S.tail_next(e, tl);
  }
  if (it > max_iters && ln == 0) set_error(err, kErrIter);
  if (it_out) *it_out = it;
  return __dsub_rn(E, t);
}

// The summary of a state that admits a tail query in its next batch (FCache.summ),
// taken from the state itself: what the direct estimate reads of it for a query
// whose prefill fits the admission batch.
template <int KS>
__device__ __forceinline__ void take_summary(FCache& fc, const Queue<KS>& S, const QEnv& e) {
  const Coef& k = e.k;
  fc.summ = true;
  fc.g = S.g;
  fc.E = S.clock;
  fc.aP = (int)S.pre_sum;
  fc.aD = S.n_dec;
  fc.left = k.B - fc.aD - fc.aP;
  fc.aC = e.need_C ? S.c0sum + (int64_t)fc.aD * S.g : 0;
  fc.aA = e.need_A ? S.pre_attention_all(e) : 0;
  const typename Queue<KS>::Tail tl = S.tail_begin(e);
  fc.sD1 = (int)tl.D;
  fc.sC1 = e.need_C ? tl.c0 + tl.D * (int64_t)(S.g + 1) : 0;
  fc.snf = -1;   // taken when a replay on the summary first needs it
}

// The replay of a summarised state with an empty prefill list up to t, when it only
// folds quiet batches (nothing to prefill, no decode finishing: with lazy decoders
// such a batch changes only the batch counter and the clock) and stops before the
// next decode finish -- the batches Queue::quiet_run folds, with the same times in
// the same order -- or, for an empty instance, the idle jump of the clock to t.
// Returns false, changing nothing, when the replay would need more (a stepped batch,
// a new summary, the batch cap); otherwise brings the summary, the instance's scalars
// in LDS (batch counter, clock, batches replayed) and g, clk to the new state.
template <int KS>
__device__ __forceinline__ bool replay_summary(FCache& fc, const QEnv& e, LdsQueue<KS>& SL,
                                               int& g, double& clk, double t,
                                               int64_t max_iters) {
  if (fc.aD == 0) {   // nothing resident (the list is empty too): the clock jumps to t
    clk = t;
    fc.E = t;
    if (lane_id() == 0) SL.clock = t;
    __builtin_amdgcn_wave_barrier();
    return true;
  }
  if (fc.snf < 0) {   // the next decode finish of the summarised state, from its slots in LDS
    int m = 0x7fffffff;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int dl = SL.dl[s * kWave + lane_id()];
      if (dl > fc.g) m = min(m, dl);
    }
    fc.snf = wave_min(m);
  }
  const int D = fc.aD;
  double c = clk;
  int gg = g;
  int64_t n = 0;
  int64_t C = fc.aC;   // decode context sum of the next batch
  while (gg + 1 < fc.snf && c < t && n < max_iters) {
    c = __dadd_rn(c, e.need_C ? batch_time(e.k, 0, D, C, 0) : batch_time(e.k, 0, D, 0, 0));
    C += D;
    ++gg;
    ++n;
  }
  if (c < t || gg + 1 >= fc.snf) return false;
  g = gg;
  clk = c;
  fc.g = gg;
  fc.E = c;
  fc.aC = e.need_C ? C : 0;
  if (e.need_C) fc.sC1 += (int64_t)fc.sD1 * n;
  if (lane_id() == 0) {
    SL.g = gg;
    SL.clock = c;
    SL.iters += n;
  }
  __builtin_amdgcn_wave_barrier();
  return true;
}

// The direct estimate of a query of p <= left prompt tokens (its prefill completes in
// the admission batch) from the summary: the same batches, in the same order, as
// estimate_visit's direct path.
__device__ __forceinline__ double estimate_summary(const FCache& fc, const QEnv& e, int p,
                                                   double t, int reading, int64_t* it_out) {
  const Coef& k = e.k;
  double E = __dadd_rn(fc.E, batch_time(k, fc.aP + p, fc.aD, fc.aC,
                                         fc.aA + (int64_t)p * (p + 1) / 2));
  int64_t it = 1;
  if (reading != 1) {   // the decode batch after the admission batch
    E = __dadd_rn(E, batch_time(k, 0, fc.sD1 + 1, fc.sC1 + p, 0));
    ++it;
  }
  *it_out = it;
  return __dsub_rn(E, t);
}

// The whole sequential trace with each wave owning IPW instances whose states stay
// in LDS for the whole trace (one working copy in VGPRs per visit).  A scenario spans
// G workgroups of W waves; block b serves scenario z = b / G as cluster member b % G
// (consecutive blocks go to different XCDs; the members meet in device-coherent
// memory, which measured faster than keeping each scenario on one XCD).
// Iteration i (from -1): the workgroup argmax (LDS, one barrier) and the cluster
// argmax (global exchange, when G > 1) of query i, then per owned instance one visit
// (commit of query i, replay, frontier cache) and the estimate of query i + 1.
// Identical, operation for operation, to estimate + route + commit per query.
template <int KS, int W, int IPW, bool TRK>
__global__ __launch_bounds__(W * kWave) void k_trace_cl(LAR_TRACE_PARAMS, int G, uint64_t* xslot,
                                                        int tail_k, SyncCtl sc) {
  __shared__ double s_u[2][W];
  __shared__ int s_j[2][W];
  __shared__ int s_abort;
  __shared__ alignas(16) int stage[W][stage_words<TRK>()];
  __shared__ LdsQueue<KS> sst[W][IPW];   // instance states
  __shared__ LdsQueue<KS> fst[W][IPW];   // frontier states
  __shared__ LdsTags stags[TRK ? W : 1][IPW];   // instance states' tracking registers
  const int b = blockIdx.x;
  const int z = b / G;
  const int cid = b % G;
  if (z >= Z) return;
  const int wid = uni((int)(threadIdx.x / kWave));   // wave-uniform: keeps per-wave data in SGPRs
  const int nw = blockDim.x / kWave;   // waves launched (<= W)
  const int ln = lane_id();
  const double wc = w_cost[z];
  const double wl = w_lat[z];
  uint64_t* xs = xslot + (int64_t)z * 2 * kMaxCluster * 4;
  const int jbase = (cid * W + wid) * IPW;
  const int kmax = tail_k;   // <= 64, checked at launch
  const Track tk{TRK ? realized + (int64_t)z * N : nullptr, tag0, N, reading};
  if (threadIdx.x == 0) s_abort = 0;   // read after the first query's barrier
  int cols[IPW];
  FCache fc[IPW];
  QEnv env[IPW];   // per owned instance: coefficients, ring, staging (loop invariant)
  int sg[IPW];        // per owned instance: the batch counter and clock of its state
  double sclk[IPW];
#pragma unroll
  for (int r = 0; r < IPW; ++r) {
    const int j = jbase + r;
    cols[r] = j < I ? pr.col[j] : -1;
    fc[r].valid = false;
    fc[r].summ = false;
    fc[r].tD = 0;
    fc[r].tC = 0;
    fc[r].depth = 0;
    if (j < I) {
      env[r] = make_env(S, pr, z * I + j, j, stage[wid]);
      Queue<KS> q;
      q.template load<TRK>(S, env[r], z * I + j,
                           TRK ? S.r_tag + (int64_t)(z * I + j) * S.rcap : nullptr);
      q.template to_lds<TRK>(sst[wid][r], &stags[TRK ? wid : 0][r]);
      sg[r] = q.g;
      sclk[r] = q.clock;
    }
  }
  QueryBlock<IPW> cur = fetch_block<IPW>(0, N, qp, qd, qt, tau, acc, cost, n_cols, cols);
  QueryBlock<IPW> nxt = fetch_block<IPW>(kWave, N, qp, qd, qt, tau, acc, cost, n_cols, cols);
  unsigned long long wbatch = 0;   // batches of this wave's estimates
  Cand c;
  c.j = -1; c.u = 0.0; c.ttft = 0.0; c.eq2 = 0.0;
  for (int i = -1; i < N; ++i) {
    // inputs of query i (if any) and of query i + 1
    const int l = i & (kWave - 1);
    const bool last_in_block = i >= 0 && l == kWave - 1;
    int p = 1, dq = 1, m = -1;
    double tn = -__builtin_inf();
    if (i >= 0) {
      p = __builtin_amdgcn_readlane(cur.p, l);
      dq = __builtin_amdgcn_readlane(cur.d, l);
      if (i + 1 >= N) tn = t_after;
      else tn = last_in_block ? read_lane_f64(nxt.t, 0) : read_lane_f64(cur.t, l + 1);
      // workgroup argmax
      const int buf = i & 1;
      if (ln == 0) { s_u[buf][wid] = c.u; s_j[buf][wid] = c.j; }
      __syncthreads();
      double vu = 0.0;   // (read together with the abort flag: one LDS round trip)
      int vj = -1;
      if (ln < nw) { vu = s_u[buf][ln]; vj = s_j[buf][ln]; }
      if (s_abort) break;   // an exchange failed on the previous query
      // Lane v holds wave v's candidate.  The order is total, so the wave whose
      // candidate no other beats holds the workgroup's best (wave 0 when the workgroup
      // has no candidate); only it can hold the query's winner.  With several
      // workgroups that wave alone exchanges with the others and learns the winner;
      // the other waves are not chosen and go on to their visits while it runs.
      const bool any = ballot(vj >= 0) != 0;
      const bool beaten = ballot(better(vu, vj, c.u, c.j)) != 0;
      int holder = any ? (c.j >= 0 && !beaten ? 1 : 0) : (wid == 0 ? 1 : 0);
      double bu = holder && any ? c.u : 0.0;
      int bj = holder && any ? c.j : -1;
      int xok = 1;
      if (G > 1) {
        if (holder) {
          __builtin_amdgcn_s_setprio(3);   // the chain waits on this wave
          if (!cluster_exchange(bu, bj, i, G, cid, xs, err, sc)) {
            xok = 0;   // every wave leaves after the next workgroup barrier
            if (ln == 0) s_abort = 1;
          }
          __builtin_amdgcn_s_setprio(0);
        }
      }
      m = holder && xok && bj >= 0 ? key_index(bj) : -1;
      if (holder && xok) {
        if (bj == -1 && cid == 0 && wid == 0 && ln == 0)
          set_error(err, kErrArg);   // no candidate
        // the wave holding the winner (its own best) writes the outputs
        const bool mine = m >= 0 || (bj == -1 && cid == 0 && wid == 0);
        if (mine && ln == 0) {
          const int64_t o = (int64_t)z * N + i;
          choice[o] = m;
          if (chosen_ttft) chosen_ttft[o] = c.ttft;
          if (utility && m >= 0) utility[o] = c.eq2;
        }
      }
    }
    const bool more = i + 1 < N;
    int p1 = 1;
    double t1 = 0.0;
    int l1 = 0;
    bool in_nxt = false;
    if (more) {
      if (i < 0) { p1 = uni(cur.p); t1 = read_lane_f64(cur.t, 0); }
      else {
        in_nxt = last_in_block;
        l1 = last_in_block ? 0 : l + 1;
        p1 = last_in_block ? uni(nxt.p) : __builtin_amdgcn_readlane(cur.p, l + 1);
        t1 = tn;
      }
    }
    const bool p1_ok = p1 >= 1 && p1 <= max_prompt;
    if (more && !p1_ok && threadIdx.x == 0 && cid == 0) set_error(err, kErrArg);
    c.j = -1; c.u = 0.0; c.ttft = 0.0; c.eq2 = 0.0;
#pragma unroll
    for (int r = 0; r < IPW; ++r) {
      const int j = jbase + r;
      if (j < I) {
        const QEnv& e = env[r];
        Queue<KS> wk;
        // with several waves per SIMD, the chosen instance's commit, walk and next
        // estimate are the longest link of the query chain: let its wave issue first,
        // then the waves whose instances replay batches, then quiet replays, then the
        // rest (which only estimate)
        const bool hot = (W > 4) && i >= 0 && j == m;
        if (hot) __builtin_amdgcn_s_setprio(3);
        // Nothing to commit and no batch starting before tn: the visit would leave
        // the state as it is, so it is skipped while a cache or summary of that
        // state answers the estimate.
        // (not for the wide-slot shape of long-context pools, whose chosen instance's
        // walk is the chain and whose register budget the extra state would strain:
        // measured 1-2 % slower there)
        const bool idle = KS <= 4 && !(i >= 0 && j == m) && sclk[r] >= tn &&
                          (fc[r].valid || fc[r].summ);
        VisitOut vo;
        vo.direct = false;
        bool fold = false;
        if constexpr (KS <= 4 && !TRK && W > 4) {
          // a replay that only folds quiet batches, on the summary (with several waves
          // per SIMD, where the waves it relieves share the issue slots; with one, the
          // code it adds measured slower)
          if (!idle && !(i >= 0 && j == m) && fc[r].summ && fc[r].aP == 0) {
            __builtin_amdgcn_s_setprio(1);
            fold = replay_summary(fc[r], e, sst[wid][r], sg[r], sclk[r], tn, max_iters);
            if (fold) {
              vo.g = sg[r];
              vo.clock = sclk[r];
            }
          }
        }
        // the other visits that replay batches are the next longest links
        if ((W > 4) && !hot && !idle && !fold) __builtin_amdgcn_s_setprio(2);
        if (!idle && !fold) {
          wk.template from_lds<TRK>(sst[wid][r], &stags[TRK ? wid : 0][r]);
          vo = visit<KS, TRK>(wk, fc[r], e, i >= 0 && j == m, p, dq, tn, S.qcap, kmax,
                              max_iters, err, sst[wid][r], &stags[TRK ? wid : 0][r],
                              fst[wid][r],
                              TRK ? S.r_tag + (int64_t)(z * I + j) * S.rcap : nullptr,
                              tag0 + i, tk);
          sg[r] = vo.g;
          sclk[r] = vo.clock;
          fc[r].summ = false;
          if constexpr (KS <= 4)
            if (vo.direct) take_summary(fc[r], wk, e);
        } else {
          vo.g = sg[r];
          vo.clock = sclk[r];
        }
        if (more) {
          int64_t it = 0;
          double ttft;
          if (!p1_ok) {
            ttft = __builtin_nan("");
          } else if (fc[r].summ && p1 <= fc[r].left && sclk[r] >= t1) {
            ttft = estimate_summary(fc[r], e, p1, t1, reading, &it);
          } else {
            if ((idle || fold) && fc[r].summ) {   // a prompt beyond the admission batch: the state
              wk.template from_lds<TRK>(sst[wid][r], &stags[TRK ? wid : 0][r]);
              wk.refill(e);   // the whole prefill list in the window, as the visit left it
              vo.direct = true;
            }
            ttft = estimate_visit(fc[r], wk, vo, e, p1, t1, reading, kmax, max_iters, err, &it);
          }
          wbatch += it;
          const double a = read_lane_f64(in_nxt ? nxt.acc[r] : cur.acc[r], l1);
          const double co = read_lane_f64(in_nxt ? nxt.cost[r] : cur.cost[r], l1);
          const double eq2 = __dsub_rn(a, __dmul_rn(wc, co));
          const double tq = tau ? read_lane_f64(in_nxt ? nxt.tau : cur.tau, l1) : 0.0;
          int k;
          const double u = cand_value(eq2, ttft, wl, tau, tq, j, &k);
          cand_take(c, u, k, ttft, eq2);
        }
        if (W > 4) __builtin_amdgcn_s_setprio(0);
      }
    }
    if (last_in_block) {
      cur = nxt;
      nxt = fetch_block<IPW>(i + 1 + kWave, N, qp, qd, qt, tau, acc, cost, n_cols, cols);
    }
  }
  if (work && ln == 0) atomicAdd(work + z, wbatch);
#pragma unroll
  for (int r = 0; r < IPW; ++r) {
    const int j = jbase + r;
    if (j < I) {
      Queue<KS> q;
      q.template from_lds<TRK>(sst[wid][r], &stags[TRK ? wid : 0][r]);
      q.template store<TRK>(S, env[r], z * I + j);
    }
  }
}

// After a trace that reports realised TTFT, one wave per queue: the tracked queries
// still without a first token (drain() on a private copy of the stored state).  A
// kernel of its own, so the trace kernels carry none of its code.
template <int KS>
__global__ __launch_bounds__(kWave) void k_drain(DevState S, DevParams pr, int Z, int I,
                                                 double* realized, int tag0, int N, int reading,
                                                 int64_t max_iters, int32_t* err) {
  const int qid = blockIdx.x;
  if (qid >= Z * I) return;
  const int z = qid / I;
  const int j = qid % I;
  __shared__ alignas(16) int stage[stage_words<true>()];
  const QEnv e = make_env(S, pr, qid, j, stage);
  const int32_t* tags = S.r_tag + (int64_t)qid * S.rcap;
  if (S.sc[qid].ntrk <= 0) return;
  Queue<KS> w;
  w.template load<true>(S, e, qid, tags);
  const Track tk{realized + (int64_t)z * N, tag0, N, reading};
  drain(w, e, tags, tk, max_iters, err);
}

// Before a trace that reports realised TTFT: no query of it is tracked yet, no
// completed prefill is pending a first decode (earlier requests are not tracked),
// and every output entry is NaN until its first token is seen.
__global__ void k_track_begin(QScal* sc, int64_t n_queues, double* realized, int64_t n_out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n_queues) { sc[i].ntrk = 0; sc[i].pend = 0; }
  if (i < n_out) realized[i] = __builtin_nan("");
}

// After such a trace: realised TTFT = first-token time - arrival (NaN stays NaN).
__global__ void k_track_end(double* realized, const double* qt, int N, int64_t n_out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n_out) realized[i] = __dsub_rn(realized[i], qt[i % N]);
}

// Marks every ring entry untracked (when the tag counter starts over).
__global__ void k_untag(int32_t* tags, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) tags[i] = -1;
}

// ------------------------------------------------------------------ k_stats
// Orderable key of a binary64 (no NaN): larger key <=> larger value.
__device__ __forceinline__ uint64_t okey(double v) {
  uint64_t b = (uint64_t)__double_as_longlong(v);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

__device__ __forceinline__ double key_value(uint64_t k) {
  uint64_t b = (k >> 63) ? (k & 0x7fffffffffffffffull) : ~k;
  return __longlong_as_double((long long)b);
}

// Adds 1 to hist[d] for every lane of the wave with `on`, one atomic per wave when
// all of them carry the same digit (the usual case in the high digits of values of
// one magnitude, where per-lane atomics would all hit one counter).
__device__ __forceinline__ void hist_add(unsigned* hist, int d, bool on) {
  const uint64_t act = ballot(on);
  if (act == 0) return;
  const int l0 = __builtin_ctzll(act);
  const int d0 = __builtin_amdgcn_readlane(d, l0);
  if (ballot(on && d == d0) == act) {
    if (lane_id() == l0) atomicAdd(&hist[d0], (unsigned)popc(act));
  } else if (on) {
    atomicAdd(&hist[d], 1u);
  }
}

// The k0-th and k1-th smallest keys (0-based) of x[0..n) by 8-bit radix select,
// block-wide: both selections share each pass over x (one histogram each).
__device__ void block_select2(const double* x, int n, int k0, int k1, unsigned* h0,
                              unsigned* h1, uint64_t& r0, uint64_t& r1) {
  __shared__ int s_dig[2], s_rank[2];
  uint64_t p0 = 0, p1 = 0, mask = 0;
  int q0 = k0, q1 = k1;
  for (int shift = 56; shift >= 0; shift -= 8) {
    for (int b = threadIdx.x; b < 256; b += blockDim.x) { h0[b] = 0; h1[b] = 0; }
    __syncthreads();
    for (int base = 0; base < n; base += blockDim.x) {
      const int i = base + (int)threadIdx.x;
      uint64_t key = 0;
      if (i < n) key = okey(x[i]);
      const int d = (int)((key >> shift) & 0xff);
      hist_add(h0, d, i < n && (key & mask) == p0);
      hist_add(h1, d, i < n && (key & mask) == p1);
    }
    __syncthreads();
    if (threadIdx.x < 2) {   // thread 0 walks h0, thread 1 h1
      const unsigned* h = threadIdx.x == 0 ? h0 : h1;
      int r = threadIdx.x == 0 ? q0 : q1, dgt = 0;
      for (; dgt < 256; ++dgt) {
        if (r < (int)h[dgt]) break;
        r -= (int)h[dgt];
      }
      s_dig[threadIdx.x] = dgt;
      s_rank[threadIdx.x] = r;
    }
    __syncthreads();
    p0 |= (uint64_t)s_dig[0] << shift;
    p1 |= (uint64_t)s_dig[1] << shift;
    mask |= (uint64_t)0xff << shift;
    q0 = s_rank[0];
    q1 = s_rank[1];
    __syncthreads();
  }
  r0 = p0;
  r1 = p1;
}

// Per scenario z, two blocks: block 2z folds the means in query order (thread 0, the
// values staged in LDS by all threads), block 2z + 1 selects the nearest-rank p50 and
// p99 of the chosen TTFTs; the two run side by side.
__global__ __launch_bounds__(1024) void k_stats(int N, int I, const int32_t* choice,
                                               const double* chosen_ttft, const double* acc,
                                               const double* cost, int n_cols,
                                               const int32_t* col, const double* w_cost,
                                               double* out) {
  const int z = blockIdx.x >> 1;
  const int32_t* ch = choice + (int64_t)z * N;
  const double* tt = chosen_ttft + (int64_t)z * N;
  if ((blockIdx.x & 1) == 0) {
    __shared__ double s_a[1024], s_c[1024];
    const double wc = w_cost[z];
    double sa = 0.0, sc = 0.0, su = 0.0;
    for (int base = 0; base < N; base += blockDim.x) {
      const int i = base + (int)threadIdx.x;
      if (i < N) {
        const int cj = ch[i];
        if (cj >= 0 && cj < I) {
          const int c = col[cj];
          s_a[threadIdx.x] = acc[(int64_t)i * n_cols + c];
          s_c[threadIdx.x] = cost[(int64_t)i * n_cols + c];
        } else {   // not a routed instance: poison the means
          s_a[threadIdx.x] = __builtin_nan("");
          s_c[threadIdx.x] = __builtin_nan("");
        }
      }
      __syncthreads();
      if (threadIdx.x == 0) {   // left folds in query order
        const int m = N - base < (int)blockDim.x ? N - base : (int)blockDim.x;
        for (int r = 0; r < m; ++r) {
          const double a = s_a[r], co = s_c[r];
          sa = __dadd_rn(sa, a);
          sc = __dadd_rn(sc, co);
          su = __dadd_rn(su, __dsub_rn(a, __dmul_rn(wc, co)));
        }
      }
      __syncthreads();
    }
    if (threadIdx.x == 0) {
      out[z * 5 + 0] = __ddiv_rn(sa, (double)N);
      out[z * 5 + 1] = __ddiv_rn(sc, (double)N);
      out[z * 5 + 2] = __ddiv_rn(su, (double)N);
    }
    return;
  }
  __shared__ unsigned h50[256], h99[256];
  const int k50 = (int)(((int64_t)50 * N + 99) / 100 - 1);
  const int k99 = (int)(((int64_t)99 * N + 99) / 100 - 1);
  uint64_t v50, v99;
  block_select2(tt, N, k50, k99, h50, h99, v50, v99);
  if (threadIdx.x == 0) {
    out[z * 5 + 3] = key_value(v50);
    out[z * 5 + 4] = key_value(v99);
  }
}

// ------------------------------------------------------------------ targets, OnTimeUtility
// TTFT target of each query (appendix on TTFT latency assignment), in the written
// order: lin = 155 + 3.5e-3*p, raw = u + lin*v, clipped to [150, 1120] ms.
__global__ __launch_bounds__(256) void k_targets(int n, const int32_t* p, const double* u_ms,
                                                const double* v, double* tau) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const double lin = __dadd_rn(155.0, __dmul_rn(3.5e-3, (double)p[i]));
  const double raw = __dadd_rn(u_ms[i], __dmul_rn(lin, v[i]));
  const double lo = raw > 150.0 ? raw : 150.0;
  tau[i] = lo < 1120.0 ? lo : 1120.0;
}

// OnTimeUtility (Eq. 4) per scenario: the utility of Eq. 2 at the chosen instance,
// summed in query order over the queries whose realised TTFT (the replay's, as a
// trace reports it) is within the target, divided by N.
__global__ __launch_bounds__(256) void k_ontime(int N, int I, const int32_t* choice,
                                               const double* ttft_real, const double* tau,
                                               const double* acc, const double* cost, int n_cols,
                                               const int32_t* col, const double* w_cost,
                                               double* out) {
  __shared__ double s_v[256];
  __shared__ int s_on[256];
  const int z = blockIdx.x;
  const int32_t* ch = choice + (int64_t)z * N;
  const double* tt = ttft_real + (int64_t)z * N;
  const double wc = w_cost[z];
  double s = 0.0;
  for (int base = 0; base < N; base += 256) {
    const int i = base + (int)threadIdx.x;
    if (i < N) {
      const int cj = ch[i];
      const bool on = tt[i] <= tau[i];
      s_on[threadIdx.x] = on;
      if (cj >= 0 && cj < I) {
        const int c = col[cj];
        s_v[threadIdx.x] =
            __dsub_rn(acc[(int64_t)i * n_cols + c], __dmul_rn(wc, cost[(int64_t)i * n_cols + c]));
      } else {   // not a routed instance: poison the result
        s_v[threadIdx.x] = __builtin_nan("");
        s_on[threadIdx.x] = 1;
      }
    }
    __syncthreads();
    if (threadIdx.x == 0) {   // left fold in query order
      const int m = N - base < 256 ? N - base : 256;
      for (int r = 0; r < m; ++r)
        if (s_on[r]) s = __dadd_rn(s, s_v[r]);
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) out[z] = __ddiv_rn(s, (double)N);
}

// A one-thread kernel instead of a memset node, so the clear can sit in a captured graph.
__global__ void k_clear_error(int32_t* err) { *err = 0; }

// ------------------------------------------------------------------ launchers
template <int KS>
static hipError_t launch_traj_ks(const LaunchEnv& env, const double* t_ptr, double t_val) {
  if (env.no_ctx_term)
    hipLaunchKernelGGL((k_traj<KS, false>), dim3(env.Z * env.I), dim3(kWave), 0, env.stream,
                       env.S, env.P, env.T, env.Z, env.I, t_ptr, t_val, env.max_iters, env.err);
  else
    hipLaunchKernelGGL((k_traj<KS, true>), dim3(env.Z * env.I), dim3(kWave), 0, env.stream,
                       env.S, env.P, env.T, env.Z, env.I, t_ptr, t_val, env.max_iters, env.err);
  return hipGetLastError();
}

template <int KS>
static hipError_t launch_commit_ks(const LaunchEnv& env, const int32_t* choice,
                                   int64_t choice_zstride, const int32_t* qp_ptr,
                                   const int32_t* qd_ptr, int32_t qp, int32_t qd,
                                   const double* t_ptr, double t_val) {
  hipLaunchKernelGGL(k_commit<KS>, dim3(env.Z * env.I), dim3(kWave), 0, env.stream, env.S,
                     env.P, env.Z, env.I, choice, choice_zstride, qp_ptr, qd_ptr, qp, qd, t_ptr,
                     t_val, env.max_iters, env.err);
  return hipGetLastError();
}

template <int KS, int NW>
static hipError_t launch_trace_mem(const LaunchEnv& env, const TraceArgs& a) {
  const int nw = env.I < NW ? env.I : NW;
  if (a.realized)
    hipLaunchKernelGGL((k_trace_mem<KS, NW, true>), dim3(env.Z), dim3(nw * kWave), 0,
                       env.stream, LAR_TRACE_ARGS);
  else
    hipLaunchKernelGGL((k_trace_mem<KS, NW, false>), dim3(env.Z), dim3(nw * kWave), 0,
                       env.stream, LAR_TRACE_ARGS);
  return hipGetLastError();
}

template <int KS, int W, int IPW, bool TRK>
static hipError_t launch_trace_cl(const LaunchEnv& env, const TraceArgs& a) {
  const int per_wg = W * IPW;
  const int G = (env.I + per_wg - 1) / per_wg;
  if (G > kMaxCluster) return hipErrorInvalidValue;
  if ((uint64_t)a.N >= (1ull << 31)) return hipErrorInvalidValue;  // 32-bit post tags
  const int w_used = G == 1 ? (env.I + IPW - 1) / IPW : W;
  const int blocks = env.Z * G;
  if (G == 1) {   // no exchange: the workgroups never wait for each other
    hipLaunchKernelGGL((k_trace_cl<KS, W, IPW, TRK>), dim3(blocks), dim3(w_used * kWave), 0,
                       env.stream, LAR_TRACE_ARGS, G, env.xslot, env.T.K, env.sync);
    return hipGetLastError();
  }
  const int64_t n = (int64_t)env.Z * 2 * kMaxCluster * 4;
  hipLaunchKernelGGL(k_clear_exchange, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                     env.stream, env.xslot, n);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_together(k_trace_cl<KS, W, IPW, TRK>, dim3(blocks), dim3(w_used * kWave),
                         env.stream, LAR_TRACE_ARGS, G, env.xslot, env.T.K, env.sync);
}

// The clustered trace with (realised TTFT requested) or without first-token tracking.
template <int KS, int W, int IPW>
static hipError_t launch_trace_cl(const LaunchEnv& env, const TraceArgs& a) {
  return a.realized ? launch_trace_cl<KS, W, IPW, true>(env, a)
                    : launch_trace_cl<KS, W, IPW, false>(env, a);
}

template <int KS>
static hipError_t launch_trace_ks(const LaunchEnv& env, const TraceArgs& a) {
  // One instance per wave.  The whole grid must be resident at once (a cooperative
  // launch when a scenario spans several workgroups): up to 1024
  // queues get one wave per SIMD (4 per workgroup; the per-query chain is issue
  // latency bound, so a wave runs fastest alone on its SIMD), up to 4096 get 16-wave
  // workgroups (4 waves per SIMD, 128 VGPRs each).  N must fit the 31-bit post tags
  // and the decode-only tail of an estimate (at most K batches) one lane per batch.
  const int64_t queues = (int64_t)env.Z * env.I;
  auto fits = [&](int per_wg) {
    const int64_t G = (env.I + per_wg - 1) / per_wg;
    return G <= kMaxCluster && (uint64_t)a.N < (1ull << 31) && env.T.K >= 1 &&
           env.T.K <= kWave;
  };
  // A shape whose workgroups the runtime cannot make resident together reports
  // hipErrorInvalidConfiguration without running; the next one is tried, and the
  // HBM-state kernel, whose workgroups never wait for each other, takes any size.
  hipError_t e = hipErrorInvalidConfiguration;
  if constexpr (KS <= 4) {
    if (queues <= 1024 && fits(4)) e = launch_trace_cl<KS, 4, 1>(env, a);
    if (e != hipErrorInvalidConfiguration) return e;
    if (queues <= 4096 && fits(16)) e = launch_trace_cl<KS, 16, 1>(env, a);
    if (e != hipErrorInvalidConfiguration) return e;
  } else if constexpr (KS == 8) {
    if (queues <= 1024 && fits(4)) e = launch_trace_cl<8, 4, 1>(env, a);
    if (e != hipErrorInvalidConfiguration) return e;
    if (queues <= 2048 && fits(8)) e = launch_trace_cl<8, 8, 1>(env, a);
    if (e != hipErrorInvalidConfiguration) return e;
  }
  // Otherwise the states stay in HBM (L2) and are loaded per use.
  return launch_trace_mem<KS, (KS <= 4 ? 8 : (KS == 8 ? 8 : 4))>(env, a);
}

#define DRAIN_ARGS \
  env.S, env.P, env.Z, env.I, a.realized, a.tag0, a.N, env.reading, env.max_iters, env.err

hipError_t launch_trace(const LaunchEnv& env, const TraceArgs& a) {
  if (env.work) {
    hipLaunchKernelGGL(k_clear_work, dim3((env.Z + 255) / 256), dim3(256), 0, env.stream,
                       env.work, env.Z);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (a.realized) {
    const int64_t nq = (int64_t)env.Z * env.I, no = (int64_t)env.Z * a.N;
    const int64_t n = nq > no ? nq : no;
    hipLaunchKernelGGL(k_track_begin, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                       env.stream, env.S.sc, nq, a.realized, no);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipError_t e;
  if (env.limited) {
    e = launch_lim_trace(env, a);
    if (e != hipSuccess || !a.realized) return e;
    const int64_t no = (int64_t)env.Z * a.N;
    hipLaunchKernelGGL(k_track_end, dim3((unsigned)((no + 255) / 256)), dim3(256), 0,
                       env.stream, a.realized, a.qt, a.N, no);
    return hipGetLastError();
  }
  switch (env.ks) {
    case 1: e = launch_trace_ks<1>(env, a); break;
    case 2: e = launch_trace_ks<2>(env, a); break;
    case 4: e = launch_trace_ks<4>(env, a); break;
    case 8: e = launch_trace_ks<8>(env, a); break;
    case 16: e = launch_trace_ks<16>(env, a); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess || !a.realized) return e;
  const dim3 dg(env.Z * env.I), db(kWave);
  switch (env.ks) {
    case 1: hipLaunchKernelGGL(k_drain<1>, dg, db, 0, env.stream, DRAIN_ARGS); break;
    case 2: hipLaunchKernelGGL(k_drain<2>, dg, db, 0, env.stream, DRAIN_ARGS); break;
    case 4: hipLaunchKernelGGL(k_drain<4>, dg, db, 0, env.stream, DRAIN_ARGS); break;
    case 8: hipLaunchKernelGGL(k_drain<8>, dg, db, 0, env.stream, DRAIN_ARGS); break;
    default: hipLaunchKernelGGL(k_drain<16>, dg, db, 0, env.stream, DRAIN_ARGS); break;
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t no = (int64_t)env.Z * a.N;
  hipLaunchKernelGGL(k_track_end, dim3((unsigned)((no + 255) / 256)), dim3(256), 0, env.stream,
                     a.realized, a.qt, a.N, no);
  return hipGetLastError();
}

hipError_t launch_traj(const LaunchEnv& env, const double* t_ptr, double t_val) {
  if (env.limited) return hipSuccess;   // estimates under limits simulate from the state
  switch (env.ks) {
    case 1: return launch_traj_ks<1>(env, t_ptr, t_val);
    case 2: return launch_traj_ks<2>(env, t_ptr, t_val);
    case 4: return launch_traj_ks<4>(env, t_ptr, t_val);
    case 8: return launch_traj_ks<8>(env, t_ptr, t_val);
    case 16: return launch_traj_ks<16>(env, t_ptr, t_val);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_commit(const LaunchEnv& env, const int32_t* choice, int64_t choice_zstride,
                         const int32_t* qp_ptr, const int32_t* qd_ptr, int32_t qp, int32_t qd,
                         const double* t_ptr, double t_val) {
  if (env.limited)
    return launch_lim_commit(env, choice, choice_zstride, qp_ptr, qd_ptr, qp, qd, t_ptr, t_val);
  switch (env.ks) {
    case 1: return launch_commit_ks<1>(env, choice, choice_zstride, qp_ptr, qd_ptr, qp, qd, t_ptr, t_val);
    case 2: return launch_commit_ks<2>(env, choice, choice_zstride, qp_ptr, qd_ptr, qp, qd, t_ptr, t_val);
    case 4: return launch_commit_ks<4>(env, choice, choice_zstride, qp_ptr, qd_ptr, qp, qd, t_ptr, t_val);
    case 8: return launch_commit_ks<8>(env, choice, choice_zstride, qp_ptr, qd_ptr, qp, qd, t_ptr, t_val);
    case 16: return launch_commit_ks<16>(env, choice, choice_zstride, qp_ptr, qd_ptr, qp, qd, t_ptr, t_val);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_est(const LaunchEnv& env, int Q, const int32_t* q_prefill, const double* t_ptr,
                      double t_val, double* ttft, int32_t* iters) {
  if (env.limited) return launch_lim_est(env, Q, q_prefill, t_ptr, t_val, ttft, iters);
  const int64_t blocks =
      (int64_t)env.Z * ((Q + kEstChunk - 1) / kEstChunk) * ((env.I + 255) / 256);
  if (blocks == 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_est, dim3((unsigned)blocks), dim3(256), 0, env.stream, env.P, env.T,
                     env.Z, Q, env.I, q_prefill, t_ptr, t_val, env.max_prompt, env.reading,
                     env.max_iters,
                     ttft, iters, env.err);
  return hipGetLastError();
}

hipError_t launch_route(const LaunchEnv& env, int Q, const double* ttft, int64_t ttft_zstride,
                        const double* acc, const double* cost, int n_cols, const double* w_cost,
                        const double* w_lat, const double* tau, int32_t* choice,
                        double* chosen_ttft, double* utility, int64_t out_zstride, int out_q0) {
  // one wave per row, four rows per block
  const int64_t rows = (int64_t)env.Z * Q;
  if (rows == 0) return hipSuccess;
  const int waves = rows < 4 ? (int)rows : 4;
  hipLaunchKernelGGL(k_route, dim3((unsigned)((rows + waves - 1) / waves)), dim3(waves * kWave), 0,
                     env.stream, env.Z, Q, env.I, ttft,
                     ttft_zstride, acc, cost, n_cols, env.P.col, w_cost, w_lat, tau, choice,
                     chosen_ttft, utility, out_zstride, out_q0, env.err);
  return hipGetLastError();
}

hipError_t launch_targets(hipStream_t stream, int n, const int32_t* p, const double* u_ms,
                          const double* v, double* tau) {
  hipLaunchKernelGGL(k_targets, dim3((n + 255) / 256), dim3(256), 0, stream, n, p, u_ms, v, tau);
  return hipGetLastError();
}

hipError_t launch_ontime(const LaunchEnv& env, int N, const int32_t* choice,
                         const double* ttft_real, const double* tau, const double* acc,
                         const double* cost, int n_cols, const double* w_cost, double* out) {
  hipLaunchKernelGGL(k_ontime, dim3(env.Z), dim3(256), 0, env.stream, N, env.I, choice,
                     ttft_real, tau, acc, cost, n_cols, env.P.col, w_cost, out);
  return hipGetLastError();
}

hipError_t launch_untag(const LaunchEnv& env) {
  const int64_t n = (int64_t)env.Z * env.I * env.S.rcap;
  hipLaunchKernelGGL(k_untag, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, env.stream,
                     env.S.r_tag, n);
  return hipGetLastError();
}

hipError_t launch_clear_exchange(const LaunchEnv& env) {
  const int64_t n = (int64_t)env.Z * 2 * kMaxCluster * 4;
  hipLaunchKernelGGL(k_clear_exchange, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                     env.stream, env.xslot, n);
  return hipGetLastError();
}

hipError_t launch_clear_error(const LaunchEnv& env) {
  hipLaunchKernelGGL(k_clear_error, dim3(1), dim3(1), 0, env.stream, env.err);
  return hipGetLastError();
}

hipError_t launch_stats(const LaunchEnv& env, int N, const int32_t* choice,
                        const double* chosen_ttft, const double* acc, const double* cost,
                        int n_cols, const double* w_cost, double* out) {
  hipLaunchKernelGGL(k_stats, dim3(2 * env.Z), dim3(1024), 0, env.stream, N, env.I, choice, chosen_ttft,
                     acc, cost, n_cols, env.P.col, w_cost, out);
  return hipGetLastError();
}

}  // namespace lar
