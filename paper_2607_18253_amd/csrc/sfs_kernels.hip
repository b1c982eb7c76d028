// sfs_kernels.hip -- HIP kernels of the SFS estimator and router for gfx950.
//
//   k_traj   one wave per (scenario, instance): background trajectory up to the
//            batch in which a new FCFS-tail query is first served, plus the
//            decode-only batches after it.  Exact for every tail query: the query
//            is last in FCFS order and only takes budget and slots the background
//            leaves, so all batches before its admission batch are the same with or
//            without it, and after that batch the background only decodes.
//   k_est    one thread per (scenario, query, instance), instance fastest: the
//            query's own continuation from the shared trajectory (Sec. 4.1, the
//            first-output-token batch and the TTFT sum).
//   k_route  one block per (scenario, query) row: Lagrangian utility and argmax
//            with ties to the lowest instance (Sec. 3, Eq. 2).
//   k_commit one wave per (scenario, instance): append the routed query, then
//            replay batches until the clock reaches the next arrival.
//   k_stats  one block per scenario: means in query order, nearest-rank p50/p99.
#include "sfs_device.h"
#include "sfs_launch.h"

namespace lar {

// ------------------------------------------------------------------ k_traj
template <int KS>
__global__ __launch_bounds__(kWave) void k_traj(DevState S, DevParams pr, DevTraj tr, int Z, int I,
                                               const double* t_ptr, double t_val,
                                               int64_t max_iters, int32_t* err) {
  __shared__ int l_rp[KS * kWave], l_rd[KS * kWave], l_cx[KS * kWave];
  const int qid = blockIdx.x;
  if (qid >= Z * I) return;
  const int j = qid % I;
  const double t = t_ptr ? *t_ptr : t_val;
  WaveQueue<KS> w;
  w.k = load_coef(pr, j);
  w.need_C = w.k.d != 0.0;
  w.need_A = w.k.e != 0.0;
  w.l_rp = l_rp; w.l_rd = l_rd; w.l_cx = l_cx;
  w.load(S, qid);
  const int ln = lane_id();
  double E = S.clock[qid];
  int ok = 1;
  if (E < t) {
    ok = 0;
    if (ln == 0) set_error(err, kErrState);
  }
  int pre = 0;
  StepInfo adm;
  adm.f = Feat{0, 0, 0, 0};
  adm.left = w.k.B;
  bool admitted = false;
  while (ok) {
    if ((int64_t)pre >= max_iters) {   // admission batch would exceed the cap
      ok = 0;
      break;
    }
    if (w.resident() == 0) {           // empty: the query is served alone from now on
      admitted = true;
      adm.f = Feat{0, 0, 0, 0};
      adm.left = w.k.B;
      break;
    }
    StepInfo si = w.step();
    const bool reached = si.n_adm == si.n_wait0 && si.left > 0 && si.n_run0 + si.n_adm < w.k.M;
    if (reached) {
      admitted = true;
      adm = si;
      break;
    }
    E = __dadd_rn(E, batch_time(w.k, si.f.P, si.f.D, si.f.C, si.f.A));
    ++pre;
  }
  if (ln == 0) {
    tr.E[qid] = E;
    tr.pre[qid] = pre;
    tr.P[qid] = adm.f.P;
    tr.D[qid] = adm.f.D;
    tr.C[qid] = adm.f.C;
    tr.A[qid] = adm.f.A;
    tr.left[qid] = adm.left;
    tr.ok[qid] = ok && admitted ? 1 : 0;
  }
  const int ZI = Z * I;
  for (int kk = 0; kk < tr.K; ++kk) {
    int D = 0;
    int64_t C = 0;
    if (ok && w.n_run > 0) {
      StepInfo si = w.step();   // decode-only after the admission batch
      D = (int)si.f.D;
      C = si.f.C;
    }
    if (ln == 0) {
      tr.tailD[(int64_t)kk * ZI + qid] = D;
      tr.tailC[(int64_t)kk * ZI + qid] = C;
    }
  }
}

// ------------------------------------------------------------------ k_est
__global__ __launch_bounds__(256) void k_est(DevParams pr, DevTraj tr, int Z, int Q, int I,
                                            const int32_t* q_prefill, const double* t_ptr,
                                            double t_val, int max_prompt,
                                            int reading, int64_t max_iters, double* ttft,
                                            int32_t* iters, int32_t* err) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)Z * Q * I;
  if (idx >= total) return;
  const int j = (int)(idx % I);
  const int64_t zq = idx / I;
  const int q = (int)(zq % Q);
  const int z = (int)(zq / Q);
  const int qid = z * I + j;
  const int ZI = Z * I;
  const int p = q_prefill[q];
  const double t = t_ptr ? *t_ptr : t_val;
  if (p < 1 || p > max_prompt) {
    set_error(err, kErrArg);
    ttft[idx] = __builtin_nan("");
    if (iters) iters[idx] = -1;
    return;
  }
  if (!tr.ok[qid]) {
    set_error(err, kErrIter);   // a clock behind t was already reported as a state error
    ttft[idx] = __builtin_nan("");
    if (iters) iters[idx] = -1;
    return;
  }
  const Coef k = load_coef(pr, j);
  double E = tr.E[qid];
  int64_t it = (int64_t)tr.pre[qid] + 1;
  // admission batch: background features plus the query's first chunk (context 0)
  const int lft = tr.left[qid];
  const int64_t ch = p < lft ? p : lft;
  E = __dadd_rn(E, batch_time(k, tr.P[qid] + ch, tr.D[qid], tr.C[qid],
                              tr.A[qid] + ch * (ch + 1) / 2));
  int64_t rem = p - ch;
  int64_t cxq = ch;
  bool done = reading == 1 && rem == 0;
  int kk = 0;
  while (!done) {
    if (kk >= tr.K) {   // cannot happen for p <= max_prompt; guard the tail bounds
      set_error(err, kErrIter);
      E = __builtin_nan("");
      break;
    }
    const int64_t Dk = tr.tailD[(int64_t)kk * ZI + qid];
    const int64_t Ck = tr.tailC[(int64_t)kk * ZI + qid];
    if (rem > 0) {
      const int64_t room = (int64_t)k.B - Dk;
      const int64_t c2 = rem < room ? rem : room;
      E = __dadd_rn(E, batch_time(k, c2, Dk, Ck, c2 * cxq + c2 * (c2 + 1) / 2));
      rem -= c2;
      cxq += c2;
      done = reading == 1 && rem == 0;
    } else {
      E = __dadd_rn(E, batch_time(k, 0, Dk + 1, Ck + cxq, 0));
      done = true;
    }
    ++kk;
    ++it;
  }
  if (it > max_iters) set_error(err, kErrIter);
  ttft[idx] = __dsub_rn(E, t);
  if (iters) iters[idx] = (int32_t)it;
}

// ------------------------------------------------------------------ k_route
struct Best {
  double u;
  int j;   // -1 = none
};

__device__ __forceinline__ bool better(double u1, int j1, double u2, int j2) {
  if (j2 < 0) return j1 >= 0;
  if (j1 < 0) return false;
  return u1 > u2 || (u1 == u2 && j1 < j2);
}

__global__ __launch_bounds__(256) void k_route(int Z, int Q, int I, const double* ttft,
                                              int64_t ttft_zstride, const double* acc,
                                              const double* cost, int n_cols, const int32_t* col,
                                              const double* w_cost, const double* w_lat,
                                              int32_t* choice, double* chosen_ttft,
                                              double* utility, int64_t out_zstride, int out_q0) {
  __shared__ double s_u[256 / kWave];
  __shared__ int s_j[256 / kWave];
  const int row = blockIdx.x;   // z * Q + q
  const int z = row / Q;
  const int q = row % Q;
  const double wc = w_cost[z];
  const double wl = w_lat[z];
  const double* trow = ttft + (int64_t)z * ttft_zstride + (int64_t)q * I;
  const double* arow = acc + (int64_t)q * n_cols;
  const double* crow = cost + (int64_t)q * n_cols;
  double bu = 0.0;
  int bj = -1;
  for (int j = threadIdx.x; j < I; j += blockDim.x) {
    const int c = col[j];
    const double pen = __dmul_rn(wc, crow[c]);
    double u = __dsub_rn(arow[c], pen);
    u = __dsub_rn(u, __dmul_rn(wl, trow[j]));
    if (bj < 0 || u > bu) { bu = u; bj = j; }
  }
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) {
    const double u2 = __shfl_xor(bu, o, kWave);
    const int j2 = __shfl_xor(bj, o, kWave);
    if (better(u2, j2, bu, bj)) { bu = u2; bj = j2; }
  }
  const int wid = threadIdx.x / kWave;
  if (lane_id() == 0) { s_u[wid] = bu; s_j[wid] = bj; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < (int)(blockDim.x / kWave); ++w)
      if (better(s_u[w], s_j[w], bu, bj)) { bu = s_u[w]; bj = s_j[w]; }
    const int64_t o = (int64_t)z * out_zstride + out_q0 + q;
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
template <int KS>
__global__ __launch_bounds__(kWave) void k_commit(DevState S, DevParams pr, int Z, int I,
                                                 const int32_t* choice, int64_t choice_zstride,
                                                 const int32_t* qp_ptr, const int32_t* qd_ptr,
                                                 int32_t qp_val, int32_t qd_val,
                                                 const double* t_ptr, double t_val,
                                                 int64_t max_iters, int32_t* err) {
  __shared__ int l_rp[KS * kWave], l_rd[KS * kWave], l_cx[KS * kWave];
  const int qid = blockIdx.x;
  if (qid >= Z * I) return;
  const int z = qid / I;
  const int j = qid % I;
  const int ln = lane_id();
  const double t = t_ptr ? *t_ptr : t_val;
  WaveQueue<KS> w;
  w.k = load_coef(pr, j);
  w.need_C = w.k.d != 0.0;
  w.need_A = w.k.e != 0.0;
  w.l_rp = l_rp; w.l_rd = l_rd; w.l_cx = l_cx;
  w.load(S, qid);
  if (choice && choice[(int64_t)z * choice_zstride] == j) {
    const int p = qp_ptr ? *qp_ptr : qp_val;
    int d = qd_ptr ? *qd_ptr : qd_val;
    d = d < 1 ? 1 : d;
    if (p < 1) {
      if (ln == 0) set_error(err, kErrArg);
    } else if (w.n_wait + 1 > w.qcap) {
      if (ln == 0) set_error(err, kErrCapacity);
    } else {
      int pos = w.head + w.n_wait;
      if (pos >= w.qcap) pos -= w.qcap;
      if (ln == 0) {
        S.wait_p[(int64_t)qid * S.qcap + pos] = p;
        S.wait_rd[(int64_t)qid * S.qcap + pos] = d;
      }
      w.n_wait += 1;
      // make lane 0's store visible to the loads of the replay below
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
      __syncthreads();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
  }
  double clock = S.clock[qid];
  int64_t n = 0;
  while (w.resident() > 0 && clock < t) {
    if (n == max_iters) {
      if (ln == 0) set_error(err, kErrIter);
      break;
    }
    StepInfo si = w.step();
    clock = __dadd_rn(clock, batch_time(w.k, si.f.P, si.f.D, si.f.C, si.f.A));
    ++n;
  }
  if (w.resident() == 0 && clock < t) clock = t;
  w.store(S, qid);
  if (ln == 0) {
    S.clock[qid] = clock;
    S.iters[qid] += n;
  }
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

// k-th smallest key (0-based) of x[0..n) by 8-bit radix select, block-wide.
__device__ uint64_t block_select(const double* x, int n, int kth, unsigned* hist) {
  uint64_t prefix = 0, mask = 0;
  int rank = kth;
  for (int shift = 56; shift >= 0; shift -= 8) {
    for (int b = threadIdx.x; b < 256; b += blockDim.x) hist[b] = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
      const uint64_t key = okey(x[i]);
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 0xff], 1u);
    }
    __syncthreads();
    __shared__ int s_digit, s_rank;
    if (threadIdx.x == 0) {
      int r = rank, dgt = 0;
      for (; dgt < 256; ++dgt) {
        if (r < (int)hist[dgt]) break;
        r -= (int)hist[dgt];
      }
      s_digit = dgt;
      s_rank = r;
    }
    __syncthreads();
    prefix |= (uint64_t)s_digit << shift;
    mask |= (uint64_t)0xff << shift;
    rank = s_rank;
    __syncthreads();
  }
  return prefix;
}

__global__ __launch_bounds__(256) void k_stats(int N, int I, const int32_t* choice,
                                              const double* chosen_ttft, const double* acc,
                                              const double* cost, int n_cols,
                                              const int32_t* col, const double* w_cost,
                                              double* out) {
  __shared__ unsigned hist[256];
  const int z = blockIdx.x;
  const int32_t* ch = choice + (int64_t)z * N;
  const double* tt = chosen_ttft + (int64_t)z * N;
  __shared__ double s_a[256], s_c[256];
  const double wc = w_cost[z];
  double sa = 0.0, sc = 0.0, su = 0.0;
  for (int base = 0; base < N; base += 256) {
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
      const int m = N - base < 256 ? N - base : 256;
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
  const int k50 = (int)(((int64_t)50 * N + 99) / 100 - 1);
  const int k99 = (int)(((int64_t)99 * N + 99) / 100 - 1);
  const uint64_t v50 = block_select(tt, N, k50, hist);
  const uint64_t v99 = block_select(tt, N, k99, hist);
  if (threadIdx.x == 0) {
    out[z * 5 + 3] = key_value(v50);
    out[z * 5 + 4] = key_value(v99);
  }
}

// A one-thread kernel instead of a memset node, so the clear can sit in a captured graph.
__global__ void k_clear_error(int32_t* err) { *err = 0; }

// ------------------------------------------------------------------ launchers
template <int KS>
static hipError_t launch_traj_ks(const LaunchEnv& env, const double* t_ptr, double t_val) {
  hipLaunchKernelGGL(k_traj<KS>, dim3(env.Z * env.I), dim3(kWave), 0, env.stream, env.S,
                     env.P, env.T, env.Z, env.I, t_ptr, t_val, env.max_iters, env.err);
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

hipError_t launch_traj(const LaunchEnv& env, const double* t_ptr, double t_val) {
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
  const int64_t total = (int64_t)env.Z * Q * env.I;
  const int64_t blocks = (total + 255) / 256;
  hipLaunchKernelGGL(k_est, dim3((unsigned)blocks), dim3(256), 0, env.stream, env.P, env.T,
                     env.Z, Q, env.I, q_prefill, t_ptr, t_val, env.max_prompt, env.reading,
                     env.max_iters,
                     ttft, iters, env.err);
  return hipGetLastError();
}

hipError_t launch_route(const LaunchEnv& env, int Q, const double* ttft, int64_t ttft_zstride,
                        const double* acc, const double* cost, int n_cols, const double* w_cost,
                        const double* w_lat, int32_t* choice, double* chosen_ttft,
                        double* utility, int64_t out_zstride, int out_q0) {
  hipLaunchKernelGGL(k_route, dim3(env.Z * Q), dim3(256), 0, env.stream, env.Z, Q, env.I, ttft,
                     ttft_zstride, acc, cost, n_cols, env.P.col, w_cost, w_lat, choice,
                     chosen_ttft, utility, out_zstride, out_q0);
  return hipGetLastError();
}

hipError_t launch_clear_error(const LaunchEnv& env) {
  hipLaunchKernelGGL(k_clear_error, dim3(1), dim3(1), 0, env.stream, env.err);
  return hipGetLastError();
}

hipError_t launch_stats(const LaunchEnv& env, int N, const int32_t* choice,
                        const double* chosen_ttft, const double* acc, const double* cost,
                        int n_cols, const double* w_cost, double* out) {
  hipLaunchKernelGGL(k_stats, dim3(env.Z), dim3(256), 0, env.stream, N, env.I, choice, chosen_ttft,
                     acc, cost, n_cols, env.P.col, w_cost, out);
  return hipGetLastError();
}

}  // namespace lar
