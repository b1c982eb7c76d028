// sfs_route.h -- what the trace kernels share: the candidate order of the per-query
// argmax (Sec. 3, Eq. 2 and the Lagrangian objective; Eq. 3), the trace inputs of a
// query and the workgroup argmax.
#pragma once

#include "sfs_device.h"
#include "sfs_launch.h"

namespace lar {

// Candidates of the argmax are (value, key) pairs.  The key is the instance index
// j, with bit 30 set when the candidate misses its TTFT target under the
// constrained objective (Eq. 3); a negative key means "no candidate".  The order:
// a candidate meeting its target beats one that misses it, then the larger value,
// then the lower index.  Under the Lagrangian objective every key is the bare
// index and the value is the Lagrangian utility; under Eq. 3 the value is the
// utility of Eq. 2 for a candidate meeting its target and -TTFT otherwise (so the
// empty feasible set falls back to the least estimated TTFT).  An instance whose
// estimate is +infinity (its context limit cannot hold the prompt) is no candidate,
// and neither is a NaN value.  Written without branches so a lane-wise use stays a
// few selects.
constexpr int kLateBit = 1 << 30;
__device__ __forceinline__ int key_index(int k) { return k & (kLateBit - 1); }

__device__ __forceinline__ bool better(double u1, int k1, double u2, int k2) {
  const int c1 = k1 >> 30, c2 = k2 >> 30;
  return (k1 >= 0) & (u1 == u1) &   // a NaN value is never a candidate
         ((k2 < 0) | (c1 < c2) | ((c1 == c2) & ((u1 > u2) | ((u1 == u2) & (k1 < k2)))));
}

// Value and key of instance j for one query: eq2 = acc - w_cost*cost (Eq. 2).
// tau == nullptr: Lagrangian objective, value eq2 - w_lat*ttft; else Eq. 3 with the
// query's target *tau.
__device__ __forceinline__ double cand_value(double eq2, double ttft, double wl,
                                             const double* tau, double tq, int j, int* key) {
  if (ttft == __builtin_inf()) {   // the instance cannot take the query: no candidate
    *key = -1;
    return 0.0;
  }
  if (!tau) {
    *key = j;
    return __dsub_rn(eq2, __dmul_rn(wl, ttft));
  }
  const bool ok = ttft <= tq;
  *key = ok ? j : (j | kLateBit);
  return ok ? eq2 : -ttft;
}

// One butterfly step of the lane argmax: take the partner lane's candidate (DPP
// pattern CTRL) when it is better.
template <int CTRL>
__device__ __forceinline__ void best_step_dpp(double& u, int& j) {
  const long long b = __double_as_longlong(u);
  const int lo = __builtin_amdgcn_mov_dpp((int)b, CTRL, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_mov_dpp((int)(b >> 32), CTRL, 0xf, 0xf, false);
  const double xu = __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
  const int xj = __builtin_amdgcn_mov_dpp(j, CTRL, 0xf, 0xf, false);
  const bool t = better(xu, xj, u, j);
  u = t ? xu : u;
  j = t ? xj : j;
}

// One step across 16-lane rows: the rows in ROWS take the candidate that DPP
// pattern CTRL broadcasts to them (row_bcast) when it is better; other rows keep
// their own.
template <int CTRL, int ROWS>
__device__ __forceinline__ void best_step_bcast(double& u, int& j) {
  const long long b = __double_as_longlong(u);
  const int b_lo = (int)b, b_hi = (int)(b >> 32);
  const int lo = __builtin_amdgcn_update_dpp(b_lo, b_lo, CTRL, ROWS, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(b_hi, b_hi, CTRL, ROWS, 0xf, false);
  const double xu = __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
  const int xj = __builtin_amdgcn_update_dpp(j, j, CTRL, ROWS, 0xf, false);
  const bool t = better(xu, xj, u, j);
  u = t ? xu : u;
  j = t ? xj : j;
}

// Argmax of the candidates in lanes [0, n) (every lane from n on must hold j = -1);
// the result is returned wave-uniform.  Quad permutations and the
// row mirrors combine 2, 4, 8 and 16 lanes (every lane of a row then holds the row's
// best); beyond 16, row 0's best moves into row 1 and row 2's into row 3
// (row_bcast:15), then rows 0-1's into rows 2-3 (row_bcast:31), so lane 63 holds the
// best of all.
__device__ __forceinline__ void lane_best(double& u, int& j, int n) {
  if (n > 1) best_step_dpp<0xB1>(u, j);    // quad_perm [1,0,3,2]
  if (n > 2) best_step_dpp<0x4E>(u, j);    // quad_perm [2,3,0,1]
  if (n > 4) best_step_dpp<0x141>(u, j);   // row_half_mirror
  if (n > 8) best_step_dpp<0x140>(u, j);   // row_mirror
  int src = 0;
  if (n > 16) {
    best_step_bcast<0x142, 0xa>(u, j);     // row_bcast:15 into rows 1 and 3
    best_step_bcast<0x143, 0xc>(u, j);     // row_bcast:31 into rows 2 and 3
    src = kWave - 1;
  }
  const long long b = __double_as_longlong(u);
  const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)b, src);
  const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(b >> 32), src);
  u = __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
  j = __builtin_amdgcn_readlane(j, src);
}

// Trace inputs of one query, loaded one query ahead so their memory latency hides
// behind the previous query's work.  Lane l of a wave holds acc / cost of the wave's
// l-th owned instance.
struct QueryIn {
  int p, d;
  double t, tn, tau;
  double acc_l, cost_l;   // per lane
};

__device__ __forceinline__ QueryIn fetch_query(int i, int N, const int32_t* qp, const int32_t* qd,
                                               const double* qt, double t_after,
                                               const double* tau, const double* acc,
                                               const double* cost, int n_cols, int col_l,
                                               bool own_l) {
  QueryIn q;
  q.tau = 0.0;
  if (i < N) {
    q.p = qp[i];
    q.d = qd[i];
    q.t = qt[i];
    q.tn = (i + 1 < N) ? qt[i + 1] : t_after;
    if (tau) q.tau = tau[i];
    const int64_t o = (int64_t)i * n_cols + col_l;
    q.acc_l = own_l ? acc[o] : 0.0;
    q.cost_l = own_l ? cost[o] : 0.0;
  } else {
    q.p = 1; q.d = 1; q.t = 0.0; q.tn = 0.0; q.acc_l = 0.0; q.cost_l = 0.0;
  }
  return q;
}

__device__ __forceinline__ double read_lane_f64(double v, int l) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), l);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// Candidate of the wave's l-th owned instance j for query i: lane l holds its acc /
// cost for l < 64; an instance beyond the wave's 64th reads them from memory.
__device__ __forceinline__ double utility_lane(const QueryIn& q, int l, double wc, double wl,
                                               const double* tau, double ttft, int j, int* key,
                                               double* eq2, int i, const double* acc,
                                               const double* cost, int n_cols, int col_j) {
  double a, c;
  if (l < kWave) {
    a = read_lane_f64(q.acc_l, l);
    c = read_lane_f64(q.cost_l, l);
  } else {
    const int64_t o = (int64_t)i * n_cols + col_j;
    a = acc[o];
    c = cost[o];
  }
  const double u = __dsub_rn(a, __dmul_rn(wc, c));
  *eq2 = u;
  return cand_value(u, ttft, wl, tau, q.tau, j, key);
}

// Workgroup argmax over the waves' candidates (double-buffered by query parity, so
// one barrier per query suffices); thread 0 writes the outputs.
template <int NW>
__device__ __forceinline__ int trace_pick(double bu, int bj, double bt, double bq, int i, int z,
                                          int N, int32_t* choice, double* chosen_ttft,
                                          double* utility, double (*s_u)[NW], double (*s_t)[NW],
                                          double (*s_q)[NW], int (*s_j)[NW]) {
  const int wid = uni((int)(threadIdx.x / kWave));   // wave-uniform: keeps per-wave data in SGPRs
  const int nw = blockDim.x / kWave;
  const int buf = i & 1;
  if (lane_id() == 0) { s_u[buf][wid] = bu; s_j[buf][wid] = bj; s_t[buf][wid] = bt; s_q[buf][wid] = bq; }
  __syncthreads();
  double mu = s_u[buf][0], mt = s_t[buf][0], mq = s_q[buf][0];
  int m = s_j[buf][0];
  for (int v = 1; v < nw; ++v)
    if (better(s_u[buf][v], s_j[buf][v], mu, m)) {
      mu = s_u[buf][v]; m = s_j[buf][v]; mt = s_t[buf][v]; mq = s_q[buf][v];
    }
  m = m >= 0 ? key_index(m) : -1;
  if (threadIdx.x == 0) {
    const int64_t o = (int64_t)z * N + i;
    choice[o] = m;
    if (chosen_ttft) chosen_ttft[o] = mt;
    if (utility && m >= 0) utility[o] = mq;
  }
  return m;
}

#define LAR_TRACE_PARAMS                                                                     \
  DevState S, DevParams pr, int Z, int I, int N, const int32_t *qp, const int32_t *qd,       \
      const double *qt, double t_after, const double *acc, const double *cost, int n_cols,   \
      const double *w_cost, const double *w_lat, const double *tau, int reading,             \
      int max_prompt, int64_t max_iters, int32_t *choice, double *chosen_ttft,               \
      double *utility, int32_t *err, unsigned long long *work, double *realized, int tag0

// Trace inputs of 64 consecutive queries, lane l holding query base + l; the acc /
// cost values are those of the wave's IPW owned instances.
template <int IPW>
struct QueryBlock {
  int p, d;
  double t, tau;
  double acc[IPW], cost[IPW];
};

template <int IPW>
__device__ __forceinline__ QueryBlock<IPW> fetch_block(int base, int N, const int32_t* qp,
                                                       const int32_t* qd, const double* qt,
                                                       const double* tau, const double* acc,
                                                       const double* cost, int n_cols,
                                                       const int* cols) {
  QueryBlock<IPW> b;
  const int i = base + lane_id();
  const bool in = i < N;
  b.p = in ? qp[i] : 1;
  b.d = in ? qd[i] : 1;
  b.t = in ? qt[i] : 0.0;
  b.tau = in && tau ? tau[i] : 0.0;
#pragma unroll
  for (int r = 0; r < IPW; ++r) {
    const int64_t o = (int64_t)i * n_cols + cols[r];
    b.acc[r] = in && cols[r] >= 0 ? acc[o] : 0.0;
    b.cost[r] = in && cols[r] >= 0 ? cost[o] : 0.0;
  }
  return b;
}

// Candidate of one wave for one query.
struct Cand {
  double u, ttft, eq2;
  int j;
};

__device__ __forceinline__ void cand_take(Cand& c, double u, int k, double ttft, double eq2) {
  if (better(u, k, c.u, c.j)) { c.u = u; c.j = k; c.ttft = ttft; c.eq2 = eq2; }
}

// Candidate exchange between the workgroups of one scenario, run by one wave of
// each.  Lane 0 posts the workgroup's best (utility, instance) for query i as three
// 64-bit words -- low and high half of the utility's bits, and the instance index --
// each carrying the tag i + 1 in its upper 32 bits, into slot set (i & 1).  Lane v
// polls post v until all three of its words carry the tag, so a post is taken only
// when it is whole, and the G posts arrive together with the poll: no counter, no
// fence, one round trip after the last member posts.  All accesses are relaxed
// agent-scope atomics on the same words, which the memory model keeps coherent.
// The wait is bounded in wall-clock time (s_memrealtime runs at 100 MHz; 10 s
// unless the host sets another bound): a member that never posts, or an error
// raised by another member, ends the trace with kErrSync instead of a hang.  Two slot
// sets suffice: a member posts query i + 2 only after every member has posted i + 1,
// i.e. has finished reading the posts of i.  On return j is the caller's own key if
// its post is the scenario's best, -1 if no member has a candidate, and kOtherBest
// otherwise (u is left as posted).
constexpr int kOtherBest = -2;
__device__ __forceinline__ bool cluster_exchange(double& u, int& j, int i, int G, int cid,
                                                 uint64_t* xs, int32_t* err, SyncCtl sc) {
  const int ln = lane_id();
  uint64_t* base = xs + (int64_t)(i & 1) * kMaxCluster * 4;
  const uint32_t tag = (uint32_t)(i + 1);
  if (ln == 0 && !(cid == sc.skip_cid && i == sc.skip_query)) {
    const uint64_t ub = (uint64_t)__double_as_longlong(u);
    const uint64_t hi = (uint64_t)tag << 32;
    uint64_t* sl = base + cid * 4;
    __hip_atomic_store(sl + 0, hi | (ub & 0xffffffffull), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(sl + 1, hi | (ub >> 32), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(sl + 2, hi | (uint32_t)j, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  // Two polls in flight: while one round trip is under way the other is issued, so
  // a post is seen about half a round trip sooner than with one poll at a time.
  uint64_t w0 = 0, w1 = 0, w2 = 0;
  bool ready = ln >= G;
  const uint64_t* o = base + (ln < G ? ln : 0) * 4;
  uint64_t x0 = 0, x1 = 0, x2 = 0;
  if (!ready) {
    x0 = __hip_atomic_load(o + 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    x1 = __hip_atomic_load(o + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    x2 = __hip_atomic_load(o + 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
  for (uint32_t polls = 1;; ++polls) {
    uint64_t y0 = 0, y1 = 0, y2 = 0;
    if (!ready) {   // next poll, issued before the previous one is looked at
      y0 = __hip_atomic_load(o + 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      y1 = __hip_atomic_load(o + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      y2 = __hip_atomic_load(o + 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if ((uint32_t)(x0 >> 32) == tag && (uint32_t)(x1 >> 32) == tag &&
          (uint32_t)(x2 >> 32) == tag) {
        w0 = x0; w1 = x1; w2 = x2;
        ready = true;
      }
    }
    x0 = y0; x1 = y1; x2 = y2;
    if (ballot(!ready) == 0) break;
    // the escape checks cost a round trip of their own: every 256th poll only
    if ((polls & 255u) == 0) {
      int bad = 0;
      if (ln == 0)
        bad = __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == kErrSync ||
              __builtin_amdgcn_s_memrealtime() - t0 > sc.spin_ticks;
      if (__builtin_amdgcn_readlane(bad, 0)) {
        if (ln == 0) set_error(err, kErrSync);
        return false;
      }
    }
  }
  // The order is total: the caller's post is the scenario's best when no other post
  // beats it.
  double pu = 0.0;
  int pj = -1;
  if (ln < G) {
    pu = __longlong_as_double((long long)((w0 & 0xffffffffull) | (w1 << 32)));
    pj = (int)(uint32_t)w2;
  }
  const bool any = ballot(pj >= 0) != 0;
  const bool beaten = ballot(better(pu, pj, u, j)) != 0;
  j = !any ? -1 : (j >= 0 && !beaten ? j : kOtherBest);
  return true;
}

#define LAR_TRACE_ARGS                                                                   \
  env.S, env.P, env.Z, env.I, a.N, a.qp, a.qd, a.qt, a.t_after, a.acc, a.cost, a.n_cols,     \
      a.w_cost, a.w_lat, a.tau, env.reading, env.max_prompt, env.max_iters, a.choice,        \
      a.chosen_ttft, a.utility, env.err, env.work, a.realized, a.tag0

}  // namespace lar
