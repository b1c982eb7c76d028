// sfs_lps.hip -- the average-case TTFT estimator for routing without real-time
// workload information (Sec. 4.2, Eqs. 10 and 11; the appendix on the limited
// processor sharing abstraction, Eqs. 12 and 13).
//
//   k_lps_wait  one thread per (scenario, instance): the expected queueing delay W of
//               an LPS server of capacity mu shared by at most k active queries under
//               arrivals at rate alpha --
//                 Poisson arrivals, memoryless work:  rho = alpha/mu,
//                   W = rho^k / (mu - alpha);
//                 variability-corrected (Eq. 13): E[Q] = 1/mu, rho = alpha*E[Q],
//                   W = ((ca2 + cs2)/2) * ((rho^k * E[Q]) / (1 - rho));
//               rho^k is the product of k factors taken left to right.
//   k_lps_est   one thread per (scenario, query, instance), instance fastest:
//               L = (W + p/theta) + t_dec (Eq. 11).  Bound by the 8-byte write of
//               each estimate.
// Every operation is one binary64 round-to-nearest-even operation in the order
// written; parameters outside the model give NaN and the sticky LAR_E_ARG.
#include "../../include/lar.h"
#include "sfs_device.h"
#include "sfs_launch.h"

namespace lar {

constexpr int kLpsMaxK = 65536;

// rho^k, the product of k factors taken left to right (rho >= 0); once it is 0 it
// stays 0, so the loop may stop there.
__device__ __forceinline__ double pow_left(double rho, int k) {
  double r = rho;
  for (int m = 1; m < k && r != 0.0; ++m) r = __dmul_rn(r, rho);
  return r;
}

__device__ __forceinline__ bool lps_ok(const lar_lps_params& q, int mode) {
  const bool base = __builtin_isfinite(q.arrival_rate) && __builtin_isfinite(q.service_rate) &&
                    q.arrival_rate >= 0.0 && q.arrival_rate < q.service_rate && q.k >= 1 &&
                    q.k <= kLpsMaxK &&
                    __builtin_isfinite(q.prefill_rate) && q.prefill_rate > 0.0 &&
                    __builtin_isfinite(q.decode_ms) && q.decode_ms >= 0.0 && q.reserved == 0;
  if (mode == LAR_LPS_POISSON) return base;
  return base && __builtin_isfinite(q.ca2) && __builtin_isfinite(q.cs2) && q.ca2 >= 0.0 &&
         q.cs2 >= 0.0;
}

__global__ __launch_bounds__(256) void k_lps_wait(const lar_lps_params* prm, int n, int mode,
                                                 double* wait, int32_t* err) {
  const int x = blockIdx.x * blockDim.x + threadIdx.x;
  if (x >= n) return;
  const lar_lps_params q = prm[x];
  double w = __builtin_nan("");
  if (lps_ok(q, mode)) {
    const double alpha = q.arrival_rate, mu = q.service_rate;
    if (mode == LAR_LPS_POISSON) {
      const double rho = __ddiv_rn(alpha, mu);
      w = __ddiv_rn(pow_left(rho, q.k), __dsub_rn(mu, alpha));
    } else {
      const double eq = __ddiv_rn(1.0, mu);
      const double rho = __dmul_rn(alpha, eq);
      if (rho < 1.0) {
        const double h = __ddiv_rn(__dadd_rn(q.ca2, q.cs2), 2.0);
        const double t = __ddiv_rn(__dmul_rn(pow_left(rho, q.k), eq), __dsub_rn(1.0, rho));
        w = __dmul_rn(h, t);
      }
    }
  }
  if (w != w) set_error(err, kErrArg);
  wait[x] = w;
}

// One block per (row, 256 instances): row = z * Q + q; the instances of a row are
// consecutive in the output, so each block writes 256 consecutive estimates.
__global__ __launch_bounds__(256) void k_lps_est(const lar_lps_params* prm, const double* wait,
                                                int Q, int I, int col_blocks,
                                                const int32_t* q_prefill, double* ttft,
                                                int32_t* err) {
  const int64_t row = blockIdx.x / (unsigned)col_blocks;   // z * Q + q
  const int j = (int)(blockIdx.x - row * col_blocks) * blockDim.x + threadIdx.x;
  if (j >= I) return;
  const int z = (int)(row / Q);
  const int q = (int)(row - (int64_t)z * Q);
  const int p = q_prefill[q];
  const int64_t zj = (int64_t)z * I + j;
  double l = __builtin_nan("");
  if (p >= 1) {
    const double theta = prm[zj].prefill_rate, t_dec = prm[zj].decode_ms;
    l = __dadd_rn(__dadd_rn(wait[zj], __ddiv_rn((double)p, theta)), t_dec);
  } else if (j == 0) {
    set_error(err, kErrArg);
  }
  ttft[row * I + j] = l;
}

hipError_t launch_lps(const LaunchEnv& env, const lar_lps_params* prm, int mode, double* wait,
                      int Q, const int32_t* q_prefill, double* ttft) {
  const int n = env.Z * env.I;
  hipLaunchKernelGGL(k_lps_wait, dim3((n + 255) / 256), dim3(256), 0, env.stream, prm, n, mode,
                     wait, env.err);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int col_blocks = (env.I + 255) / 256;
  const int64_t blocks = (int64_t)env.Z * Q * col_blocks;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;   // checked on the host first
  hipLaunchKernelGGL(k_lps_est, dim3((unsigned)blocks), dim3(256), 0, env.stream, prm, wait, Q,
                     env.I, col_blocks, q_prefill, ttft, env.err);
  return hipGetLastError();
}

}  // namespace lar
