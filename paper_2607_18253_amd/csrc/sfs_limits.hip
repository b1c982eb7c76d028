// sfs_limits.hip -- kernels of the SFS estimator and router under scheduler limits
// (chunk cap, context limit, KV-cache blocks with recompute preemption; the system
// appendix lists them among what the simulation follows), on the explicit-list
// wave engine of sfs_limits.h.  Every estimate simulates its (query, instance) pair
// batch by batch: from the instance state, or in the clustered trace from the
// instance's cached admission point (lim_frontier), which gives the same result.
//
//   k_lest     one wave per (scenario, query, instance): what-if estimate.
//   k_lcommit  one wave per (scenario, instance): append the routed query, replay
//              to the next arrival.
//   k_ltrace_cl  a whole sequential trace, G workgroups of 4 waves per scenario, one
//              instance per wave with its queue window in registers for the whole
//              trace; per query a workgroup argmax and the cross-workgroup exchange
//              of the default engine's clustered trace.
//   k_ltrace   the same trace, one workgroup per scenario with the states in HBM
//              (pools whose workgroups cannot all be resident at once).
//   k_ldrain   first tokens of tracked queries still waiting when a trace ends.
#include "sfs_device.h"
#include "sfs_launch.h"
#include "sfs_limits.h"
#include "sfs_route.h"

namespace lar {

// SFS estimate under limits: a private copy of the queue with the query appended at
// the tail, stepped until the query's first decode (reading 1: its prefill
// completes).  +infinity when the instance's context limit cannot hold the prompt
// (it cannot take the query); NaN with an error when the state is behind t or the
// batch cap is reached.
template <int KS>
__device__ __forceinline__ double lim_estimate(const LQueue<KS>& q, const LEnv& e, int p, int d,
                                               double t, int reading, int64_t max_iters,
                                               int32_t* err, int64_t* it_out) {
  const int ln = lane_id();
  *it_out = 0;
  if (q.clock < t) {
    if (ln == 0) set_error(err, kErrState);
    return __builtin_nan("");
  }
  if (p < 1) {
    if (ln == 0) set_error(err, kErrArg);
    return __builtin_nan("");
  }
  const int dq = entry_decode(e, p, d);
  if (dq < 1) return __builtin_inf();   // the context limit cannot hold the prompt
  LQueue<KS> w = q;
  w.template append<false>(e, p, dq, false, nullptr, -1);
  double E = w.clock;
  int64_t it = 0;
  for (;;) {
    if (it == max_iters) {
      if (ln == 0) set_error(err, kErrIter);
      *it_out = it;
      return __builtin_nan("");
    }
    const LStep o = w.template step<false>(e, nullptr, 0.0, nullptr);
    E = __dadd_rn(E, o.T);
    ++it;
    if (reading == 1 ? o.last_fill : o.last_dec) break;
  }
  *it_out = it;
  return __dsub_rn(E, t);
}

// The state of a queue just before the first batch in which a request appended at
// its tail could be admitted (whatever its prompt).  Batches before that one do not
// depend on such a request -- it waits behind requests that are not all admitted, or
// no slot, budget or KV block is left for it, or the batch preempts -- so an estimate
// from the returned state F, whose clock is the left fold of those batches' times
// from the queue's own clock, equals the estimate from the queue.  n receives their
// number.  False (and the error set) when the batch cap is reached first.
template <int KS>
__device__ __forceinline__ bool lim_frontier(const LQueue<KS>& q, const LEnv& e, LQueue<KS>& F,
                                             int64_t& n, int64_t max_iters, int32_t* err) {
  LQueue<KS> g = q;
  double E = g.clock;
  n = 0;
  while (g.n_list > 0) {
    if (n == max_iters) {
      if (lane_id() == 0) set_error(err, kErrIter);
      return false;
    }
    LQueue<KS> h = g;
    const LStep o = h.template step<false, true>(e, nullptr, 0.0, nullptr);
    if (o.tail_ok) break;
    E = __dadd_rn(E, o.T);
    ++n;
    g = h;
  }
  F = g;
  F.clock = E;
  return true;
}

// Append the query when this queue is the chosen one, then replay every batch that
// starts before t; an idle queue's clock jumps to t.  TRK: the query is tracked
// (tag) and first tokens of the replayed batches are recorded.
template <int KS, bool TRK>
__device__ __forceinline__ void lim_commit_advance(LQueue<KS>& w, const LEnv& e, bool chosen,
                                                   int p, int d, double t, int qcap,
                                                   int64_t max_iters, int32_t* err,
                                                   int32_t* tags, int tag, const LTrack& tk) {
  const int ln = lane_id();
  if (chosen) {
    const int dq = entry_decode(e, p, d);
    if (p < 1 || dq < 1) {
      if (ln == 0) set_error(err, kErrArg);
    } else if (w.waiting() + 1 > qcap) {
      if (ln == 0) set_error(err, kErrCapacity);
    } else {
      w.template append<TRK>(e, p, dq, true, tags, tag);
      if constexpr (TRK) w.ntrk += 1;
    }
  }
  double clock = w.clock;
  int64_t n = 0;
  while (w.n_list > 0 && clock < t) {
    if (n == max_iters) {
      if (ln == 0) set_error(err, kErrIter);
      break;
    }
    const LStep o = w.template step<TRK>(e, tags, clock, &tk);
    clock = __dadd_rn(clock, o.T);
    ++n;
  }
  if (w.n_list == 0 && clock < t) clock = t;
  w.clock = clock;
  w.iters += n;
}

// What-if estimates under limits: one wave per (scenario, query, instance), instance
// fastest; reads the state, changes nothing.
template <int KS>
__global__ __launch_bounds__(kWave) void k_lest(DevState S, DevParams pr, DevLimits lm, int Z,
                                               int Q, int I, const int32_t* q_prefill,
                                               const double* t_ptr, double t_val,
                                               int max_prompt, int reading, int64_t max_iters,
                                               double* ttft, int32_t* iters, int32_t* err) {
  const int64_t pair = blockIdx.x;
  if (pair >= (int64_t)Z * Q * I) return;
  const int j = (int)(pair % I);
  const int z = (int)(pair / ((int64_t)Q * I));
  const int q = (int)((pair / I) % Q);
  const int qid = z * I + j;
  const double t = t_ptr ? *t_ptr : t_val;
  __shared__ alignas(16) int lds[lim_lds_words<KS>()];
  const LEnv e = make_lenv(S, pr, lm, qid, j, lds);
  const int p = q_prefill[q];
  double v = __builtin_nan("");
  int64_t it = -1;
  if (p < 1 || p > max_prompt) {
    if (lane_id() == 0) set_error(err, kErrArg);
  } else {
    LQueue<KS> w;
    w.template load<false>(S, e, qid, nullptr);
    v = lim_estimate(w, e, p, 1, t, reading, max_iters, err, &it);
    if (v != v) it = -1;
  }
  if (lane_id() == 0) {
    ttft[pair] = v;
    if (iters) iters[pair] = (int32_t)(it < 0x7fffffff ? it : 0x7fffffff);
  }
}

template <int KS>
__global__ __launch_bounds__(kWave) void k_lcommit(DevState S, DevParams pr, DevLimits lm, int Z,
                                                  int I, const int32_t* choice,
                                                  int64_t choice_zstride, const int32_t* qp_ptr,
                                                  const int32_t* qd_ptr, int32_t qp_val,
                                                  int32_t qd_val, const double* t_ptr,
                                                  double t_val, int64_t max_iters, int32_t* err) {
  const int qid = blockIdx.x;
  if (qid >= Z * I) return;
  const int z = qid / I;
  const int j = qid % I;
  const double t = t_ptr ? *t_ptr : t_val;
  __shared__ alignas(16) int lds[lim_lds_words<KS>()];
  const LEnv e = make_lenv(S, pr, lm, qid, j, lds);
  LQueue<KS> w;
  w.template load<false>(S, e, qid, nullptr);
  const bool chosen = choice && choice[(int64_t)z * choice_zstride] == j;
  const int p = qp_ptr ? *qp_ptr : qp_val;
  const int d = qd_ptr ? *qd_ptr : qd_val;
  const LTrack off{nullptr, 0, 0, 0};
  lim_commit_advance<KS, false>(w, e, chosen, p, d, t, S.qcap, max_iters, err, nullptr, -1, off);
  w.template store<false>(S, e, qid, nullptr);
}

// A whole sequential trace under limits, one workgroup per scenario: wave w of nw
// owns instances j = w + v*nw (states in HBM, loaded per use); per query every owned
// instance is estimated, the workgroup picks the best, and every instance commits
// and replays to the next arrival.  TRK: the replay reports realised TTFT.
template <int KS, int NW, bool TRK>
__global__ __launch_bounds__(NW * kWave) void k_ltrace(LAR_TRACE_PARAMS, DevLimits lm) {
  __shared__ double s_u[2][NW], s_t[2][NW], s_q[2][NW];
  __shared__ int s_j[2][NW];
  __shared__ alignas(16) int lds[NW][lim_lds_words<KS>()];
  const int z = blockIdx.x;
  const int wid = uni((int)(threadIdx.x / kWave));   // wave-uniform: keeps per-wave data in SGPRs
  const int nw = blockDim.x / kWave;                 // waves launched (<= NW)
  const int ln = lane_id();
  const double wc = w_cost[z];
  const double wl = w_lat[z];
  const int j_l = wid + ln * nw;
  const bool own_l = j_l < I;
  const int col_l = own_l ? pr.col[j_l] : 0;
  QueryIn nx = fetch_query(0, N, qp, qd, qt, t_after, tau, acc, cost, n_cols, col_l, own_l);
  const LTrack tk{TRK ? realized + (int64_t)z * N : nullptr, tag0, N, reading};
  unsigned long long wbatch = 0;   // batches of this wave's estimates
  for (int i = 0; i < N; ++i) {
    const QueryIn q = nx;
    nx = fetch_query(i + 1, N, qp, qd, qt, t_after, tau, acc, cost, n_cols, col_l, own_l);
    const bool p_ok = q.p >= 1 && q.p <= max_prompt;
    if (!p_ok && threadIdx.x == 0) set_error(err, kErrArg);
    double bu = 0.0, bt = 0.0, bq = 0.0;
    int bj = -1;
    for (int v = 0, j = wid; j < I; ++v, j += nw) {
      const LEnv e = make_lenv(S, pr, lm, z * I + j, j, lds[wid]);
      LQueue<KS> w;
      w.template load<false>(S, e, z * I + j, nullptr);
      int64_t it = 0;
      const double ttft = p_ok ? lim_estimate(w, e, q.p, q.d, q.t, reading, max_iters, err, &it)
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
    if (m < 0 && threadIdx.x == 0) set_error(err, kErrArg);   // no instance can take it
    for (int j = wid; j < I; j += nw) {
      const LEnv e = make_lenv(S, pr, lm, z * I + j, j, lds[wid]);
      int32_t* tags = TRK ? S.r_tag + (int64_t)(z * I + j) * S.rcap : nullptr;
      LQueue<KS> w;
      w.template load<TRK>(S, e, z * I + j, tags);
      lim_commit_advance<KS, TRK>(w, e, j == m, q.p, q.d, q.tn, S.qcap, max_iters, err, tags,
                                  tag0 + i, tk);
      w.template store<TRK>(S, e, z * I + j, tags);
    }
  }
  if (work && lane_id() == 0) atomicAdd(work + z, wbatch);
}

// A whole sequential trace under limits, clustered: workgroup b serves scenario b / G
// as member b % G; wave w of member g owns instance g*W + w, whose queue window stays
// in registers for the whole trace (the ring beyond it in HBM).  Per query i: the
// workgroup's best candidate (LDS), the exchange with the other members, the outputs
// from the wave holding the winner, then every wave commits i and replays its
// instance to the next arrival and estimates query i + 1 from the instance's cached
// admission point (lim_frontier), which stays valid while the instance receives no
// query and its replay has not passed that point.  TRK: the replay reports realised
// TTFT.
template <int KS, int W, bool TRK>
__global__ __launch_bounds__(W * kWave) void k_ltrace_cl(LAR_TRACE_PARAMS, DevLimits lm, int G,
                                                        uint64_t* xslot, SyncCtl sc) {
  __shared__ double s_u[2][W];
  __shared__ int s_j[2][W];
  __shared__ int s_abort;
  __shared__ alignas(16) int lds[W][lim_lds_words<KS>()];
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
  const int j = cid * W + wid;
  const bool own = j < I;
  const int qid = z * I + (own ? j : 0);
  const LTrack tk{TRK ? realized + (int64_t)z * N : nullptr, tag0, N, reading};
  if (threadIdx.x == 0) s_abort = 0;   // read after the first query's barrier
  int cols[1] = {own ? pr.col[j] : -1};
  int32_t* tags = (TRK && own) ? S.r_tag + (int64_t)qid * S.rcap : nullptr;
  const LEnv e = make_lenv(S, pr, lm, qid, own ? j : 0, lds[wid]);
  LQueue<KS> Q;
  if (own) Q.template load<TRK>(S, e, qid, tags);
  QueryBlock<1> cur = fetch_block<1>(0, N, qp, qd, qt, tau, acc, cost, n_cols, cols);
  QueryBlock<1> nxt = fetch_block<1>(kWave, N, qp, qd, qt, tau, acc, cost, n_cols, cols);
  unsigned long long wbatch = 0;   // batches of this wave's estimates
  Cand c;
  c.j = -1; c.u = 0.0; c.ttft = 0.0; c.eq2 = 0.0;
  LQueue<KS> F;             // cached admission point of the owned instance
  bool f_ok = false;
  bool f_skip = false;      // the last search found the point at once: estimate directly
  int64_t f_iters = 0;      // the instance's replay count at F
  for (int i = -1; i < N; ++i) {
    const int l = i & (kWave - 1);
    const bool last_in_block = i >= 0 && l == kWave - 1;
    if (i >= 0) {
      const int p = __builtin_amdgcn_readlane(cur.p, l);
      const int dq = __builtin_amdgcn_readlane(cur.d, l);
      double tn;
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
      // has no candidate); only it can hold the query's winner: with several
      // workgroups it alone exchanges with the others, while the other waves (not
      // chosen) go on.
      const bool any = ballot(vj >= 0) != 0;
      const bool beaten = ballot(better(vu, vj, c.u, c.j)) != 0;
      const int holder = any ? (c.j >= 0 && !beaten ? 1 : 0) : (wid == 0 ? 1 : 0);
      double bu = holder && any ? c.u : 0.0;
      int bj = holder && any ? c.j : -1;
      int xok = 1;
      if (G > 1) {
        if (holder && !cluster_exchange(bu, bj, i, G, cid, xs, err, sc)) {
          xok = 0;   // every wave leaves after the next workgroup barrier
          if (ln == 0) s_abort = 1;
        }
      }
      const int m = holder && xok && bj >= 0 ? key_index(bj) : -1;
      if (holder && xok) {
        if (bj == -1 && cid == 0 && wid == 0 && ln == 0)
          set_error(err, kErrArg);   // no instance can take it
        // the wave holding the winner writes the outputs
        const bool mine = m >= 0 || (bj == -1 && cid == 0 && wid == 0);
        if (mine && ln == 0) {
          const int64_t o = (int64_t)z * N + i;
          choice[o] = m;
          if (chosen_ttft) chosen_ttft[o] = c.ttft;
          if (utility && m >= 0) utility[o] = c.eq2;
        }
      }
      if (own) {
        lim_commit_advance<KS, TRK>(Q, e, j == m, p, dq, tn, S.qcap, max_iters, err, tags,
                                    tag0 + i, tk);
        // F stays the admission point while the replay has not run its batch
        if (j == m || Q.iters > f_iters || (Q.iters == f_iters && Q.clock != F.clock))
          f_ok = false;
        if (j == m) f_skip = false;
      }
    }
    c.j = -1; c.u = 0.0; c.ttft = 0.0; c.eq2 = 0.0;
    if (i + 1 < N) {
      const bool in_nxt = last_in_block;
      const int l1 = i < 0 ? 0 : (last_in_block ? 0 : l + 1);
      const int p1 = in_nxt ? uni(nxt.p) : __builtin_amdgcn_readlane(cur.p, l1);
      const int d1 = in_nxt ? uni(nxt.d) : __builtin_amdgcn_readlane(cur.d, l1);
      const double t1 = read_lane_f64(in_nxt ? nxt.t : cur.t, l1);
      const bool p1_ok = p1 >= 1 && p1 <= max_prompt;
      if (!p1_ok && threadIdx.x == 0 && cid == 0) set_error(err, kErrArg);
      if (own) {
        int64_t it = 0;
        double ttft = __builtin_nan("");
        if (p1_ok && Q.clock < t1) {
          if (ln == 0) set_error(err, kErrState);
        } else if (p1_ok) {
          // a search that finds the point at once saves nothing and costs a batch: after
          // one, the instance is estimated directly until it receives a query
          if (!f_ok && !f_skip) {
            int64_t nf = 0;
            f_ok = lim_frontier(Q, e, F, nf, max_iters, err);
            f_iters = Q.iters + nf;
            if (f_ok && nf == 0) { f_ok = false; f_skip = true; }
          }
          if (f_ok) {
            const int64_t pre = f_iters - Q.iters;   // batches before F, folded in F's clock
            ttft = lim_estimate(F, e, p1, d1, t1, reading, max_iters - pre, err, &it);
            it += pre;
          } else {
            ttft = lim_estimate(Q, e, p1, d1, t1, reading, max_iters, err, &it);
          }
        }
        wbatch += it;
        const double a = read_lane_f64(in_nxt ? nxt.acc[0] : cur.acc[0], l1);
        const double co = read_lane_f64(in_nxt ? nxt.cost[0] : cur.cost[0], l1);
        const double eq2 = __dsub_rn(a, __dmul_rn(wc, co));
        const double tq = tau ? read_lane_f64(in_nxt ? nxt.tau : cur.tau, l1) : 0.0;
        int k;
        const double u = cand_value(eq2, ttft, wl, tau, tq, j, &k);
        cand_take(c, u, k, ttft, eq2);
      }
    }
    if (last_in_block) {
      cur = nxt;
      nxt = fetch_block<1>(i + 1 + kWave, N, qp, qd, qt, tau, acc, cost, n_cols, cols);
    }
  }
  if (work && ln == 0) atomicAdd(work + z, wbatch);
  if (own) Q.template store<TRK>(S, e, qid, tags);
}

// Tracked queries still without a first token when a trace under limits ends: a
// private copy of the queue runs on with no further arrivals until each has it.
template <int KS>
__global__ __launch_bounds__(kWave) void k_ldrain(DevState S, DevParams pr, DevLimits lm, int Z,
                                                 int I, double* realized, int tag0, int N,
                                                 int reading, int64_t max_iters, int32_t* err) {
  const int qid = blockIdx.x;
  if (qid >= Z * I) return;
  if (S.sc[qid].ntrk <= 0) return;
  const int z = qid / I;
  const int j = qid % I;
  __shared__ alignas(16) int lds[lim_lds_words<KS>()];
  const LEnv e = make_lenv(S, pr, lm, qid, j, lds);
  const int32_t* tags = S.r_tag + (int64_t)qid * S.rcap;
  LQueue<KS> w;
  w.template load<true>(S, e, qid, tags);
  const LTrack tk{realized + (int64_t)z * N, tag0, N, reading};
  double clock = w.clock;
  int64_t n = 0;
  while (w.ntrk > 0 && w.n_list > 0) {
    if (n == max_iters) {
      if (lane_id() == 0) set_error(err, kErrIter);
      break;
    }
    const LStep o = w.template step<true>(e, tags, clock, &tk);
    clock = __dadd_rn(clock, o.T);
    ++n;
  }
}

// Scheduler-limit paths: one switch over the slot width each.
#define LIM_SWITCH(KSV, CALL)                   \
  switch (env.ks) {                             \
    case 1: { constexpr int KSV = 1; CALL; } break;   \
    case 2: { constexpr int KSV = 2; CALL; } break;   \
    case 4: { constexpr int KSV = 4; CALL; } break;   \
    case 8: { constexpr int KSV = 8; CALL; } break;   \
    case 16: { constexpr int KSV = 16; CALL; } break; \
    default: return hipErrorInvalidValue;       \
  }

hipError_t launch_lim_est(const LaunchEnv& env, int Q, const int32_t* q_prefill,
                                 const double* t_ptr, double t_val, double* ttft,
                                 int32_t* iters) {
  const int64_t total = (int64_t)env.Z * Q * env.I;
  if (total > 0x7fffffff) return hipErrorInvalidValue;
  LIM_SWITCH(KSV, hipLaunchKernelGGL(k_lest<KSV>, dim3((unsigned)total), dim3(kWave), 0,
                                     env.stream, env.S, env.P, env.L, env.Z, Q, env.I,
                                     q_prefill, t_ptr, t_val, env.max_prompt, env.reading,
                                     env.max_iters, ttft, iters, env.err))
  return hipGetLastError();
}

hipError_t launch_lim_commit(const LaunchEnv& env, const int32_t* choice,
                                    int64_t choice_zstride, const int32_t* qp_ptr,
                                    const int32_t* qd_ptr, int32_t qp, int32_t qd,
                                    const double* t_ptr, double t_val) {
  LIM_SWITCH(KSV, hipLaunchKernelGGL(k_lcommit<KSV>, dim3(env.Z * env.I), dim3(kWave), 0,
                                     env.stream, env.S, env.P, env.L, env.Z, env.I, choice,
                                     choice_zstride, qp_ptr, qd_ptr, qp, qd, t_ptr, t_val,
                                     env.max_iters, env.err))
  return hipGetLastError();
}

// Waves per workgroup of the trace under limits: their LDS areas fill about 80 KiB.
template <int KS>
constexpr int lim_trace_waves() { return KS <= 4 ? 16 : (KS == 8 ? 8 : 4); }

template <int KS>
static hipError_t launch_lim_trace_ks(const LaunchEnv& env, const TraceArgs& a) {
  constexpr int NW = lim_trace_waves<KS>();
  const int nw = env.I < NW ? env.I : NW;
  if (a.realized)
    hipLaunchKernelGGL((k_ltrace<KS, NW, true>), dim3(env.Z), dim3(nw * kWave), 0, env.stream,
                       LAR_TRACE_ARGS, env.L);
  else
    hipLaunchKernelGGL((k_ltrace<KS, NW, false>), dim3(env.Z), dim3(nw * kWave), 0,
                       env.stream, LAR_TRACE_ARGS, env.L);
  return hipGetLastError();
}

// The clustered trace under limits (4 waves per workgroup, one per SIMD), a
// cooperative launch when a scenario spans several workgroups; reports
// hipErrorInvalidConfiguration without running when the runtime cannot make its
// workgroups resident at once.
template <int KS, bool TRK>
static hipError_t launch_lim_trace_cl(const LaunchEnv& env, const TraceArgs& a) {
  constexpr int W = 4;
  const int G = (env.I + W - 1) / W;
  if (G > kMaxCluster || (uint64_t)a.N >= (1ull << 31)) return hipErrorInvalidConfiguration;
  const int w_used = G == 1 ? env.I : W;
  if (G == 1) {   // no exchange: the workgroups never wait for each other
    hipLaunchKernelGGL((k_ltrace_cl<KS, W, TRK>), dim3(env.Z * G), dim3(w_used * kWave), 0,
                       env.stream, LAR_TRACE_ARGS, env.L, G, env.xslot, env.sync);
    return hipGetLastError();
  }
  const hipError_t e = launch_clear_exchange(env);
  if (e != hipSuccess) return e;
  return launch_together(k_ltrace_cl<KS, W, TRK>, dim3(env.Z * G), dim3(w_used * kWave),
                         env.stream, LAR_TRACE_ARGS, env.L, G, env.xslot, env.sync);
}

template <int KS>
static hipError_t launch_lim_trace_any(const LaunchEnv& env, const TraceArgs& a) {
  if constexpr (KS <= 8) {
    const hipError_t e = a.realized ? launch_lim_trace_cl<KS, true>(env, a)
                                    : launch_lim_trace_cl<KS, false>(env, a);
    if (e != hipErrorInvalidConfiguration) return e;
  }
  return launch_lim_trace_ks<KS>(env, a);
}

hipError_t launch_lim_trace(const LaunchEnv& env, const TraceArgs& a) {
  hipError_t e = hipSuccess;
  LIM_SWITCH(KSV, e = launch_lim_trace_any<KSV>(env, a))
  if (e != hipSuccess || !a.realized) return e;
  LIM_SWITCH(KSV, hipLaunchKernelGGL(k_ldrain<KSV>, dim3(env.Z * env.I), dim3(kWave), 0,
                                     env.stream, env.S, env.P, env.L, env.Z, env.I, a.realized,
                                     a.tag0, a.N, env.reading, env.max_iters, env.err))
  return hipGetLastError();
}

}  // namespace lar
