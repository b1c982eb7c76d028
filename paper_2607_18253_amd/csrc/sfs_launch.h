// sfs_launch.h -- host-side launch environment shared by the C ABI and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <tuple>

#include "../../include/lar.h"
#include "sfs_device.h"
#include "sfs_limits.h"

namespace lar {

// Bound of the cross-workgroup wait of the clustered trace (s_memrealtime ticks,
// 100 MHz) and a post that a member leaves out on purpose (skip_cid = -1: none).
// The host sets skip_* only in tests of the timeout path.
struct SyncCtl {
  uint64_t spin_ticks;
  int skip_cid, skip_query;
};

struct LaunchEnv {
  DevState S;
  DevParams P;
  DevTraj T;
  int Z, I;
  int ks;             // running slots per lane (1, 2, 4, 8, 16)
  int64_t max_iters;
  int max_prompt;
  bool no_ctx_term;   // every instance has d == 0 (the trajectory walk keeps no context sums)
  int reading;        // 0: first decode batch, 1: batch completing the prefill
  int32_t* err;       // sticky device error
  hipStream_t stream;
  // cross-workgroup candidate exchange of the clustered trace kernel
  uint64_t* xslot;    // [Z][2][kMaxCluster][4] tagged candidate posts
  SyncCtl sync;
  unsigned long long* work;   // [Z] batches simulated by the estimates of the last trace
  // scheduler limits: when set, estimates, commits and traces run the explicit-list
  // engine of sfs_limits.h on the state laid out for it
  bool limited;
  DevLimits L;
};

constexpr int kMaxCluster = 64;

struct TraceArgs {
  int N;
  const int32_t *qp, *qd;
  const double* qt;
  double t_after;
  const double *acc, *cost;
  int n_cols;
  const double *w_cost, *w_lat;
  const double* tau;   // per-query TTFT targets (constrained objective) or nullptr
  int32_t* choice;
  double *chosen_ttft, *utility;
  double* realized;    // [Z][N] realised TTFT of each query, or nullptr (no tracking)
  int tag0;            // tag of query 0 in the ring (queries tag0 .. tag0 + N - 1)
};

hipError_t launch_trace(const LaunchEnv& env, const TraceArgs& a);
hipError_t launch_traj(const LaunchEnv& env, const double* t_ptr, double t_val);
hipError_t launch_est(const LaunchEnv& env, int Q, const int32_t* q_prefill, const double* t_ptr,
                      double t_val, double* ttft, int32_t* iters);
hipError_t launch_route(const LaunchEnv& env, int Q, const double* ttft, int64_t ttft_zstride,
                        const double* acc, const double* cost, int n_cols, const double* w_cost,
                        const double* w_lat, const double* tau, int32_t* choice,
                        double* chosen_ttft, double* utility, int64_t out_zstride, int out_q0);
hipError_t launch_targets(hipStream_t stream, int n, const int32_t* p, const double* u_ms,
                          const double* v, double* tau);
hipError_t launch_ontime(const LaunchEnv& env, int N, const int32_t* choice,
                         const double* ttft_real, const double* tau, const double* acc,
                         const double* cost, int n_cols, const double* w_cost, double* out);
hipError_t launch_commit(const LaunchEnv& env, const int32_t* choice, int64_t choice_zstride,
                         const int32_t* qp_ptr, const int32_t* qd_ptr, int32_t qp, int32_t qd,
                         const double* t_ptr, double t_val);
hipError_t launch_clear_error(const LaunchEnv& env);
hipError_t launch_clear_exchange(const LaunchEnv& env);   // clears every scenario's posts
// the same calls under scheduler limits (sfs_limits.hip)
hipError_t launch_lim_est(const LaunchEnv& env, int Q, const int32_t* q_prefill,
                          const double* t_ptr, double t_val, double* ttft, int32_t* iters);
hipError_t launch_lim_commit(const LaunchEnv& env, const int32_t* choice, int64_t choice_zstride,
                             const int32_t* qp_ptr, const int32_t* qd_ptr, int32_t qp, int32_t qd,
                             const double* t_ptr, double t_val);
hipError_t launch_lim_trace(const LaunchEnv& env, const TraceArgs& a);
hipError_t launch_untag(const LaunchEnv& env);
hipError_t launch_lps(const LaunchEnv& env, const lar_lps_params* prm, int mode, double* wait,
                      int Q, const int32_t* q_prefill, double* ttft);
hipError_t launch_stats(const LaunchEnv& env, int N, const int32_t* choice,
                        const double* chosen_ttft, const double* acc, const double* cost,
                        int n_cols, const double* w_cost, double* out);

// Launch a grid whose workgroups wait for each other (the clustered traces: the
// members of a scenario exchange candidates every query) as a cooperative launch,
// so that the runtime either makes every workgroup resident at once or refuses the
// launch.  A refusal is reported as hipErrorInvalidConfiguration, on which the
// callers fall through to a launch shape that needs no co-residency.  The kernel's
// bounded wait stays as a backstop.
template <typename... KArgs, typename... Args>
inline hipError_t launch_together(void (*kernel)(KArgs...), dim3 grid, dim3 block,
                                  hipStream_t stream, Args... args) {
  static_assert(sizeof...(KArgs) == sizeof...(Args), "one value per kernel parameter");
  std::tuple<KArgs...> vals(static_cast<KArgs>(args)...);
  void* ptrs[sizeof...(KArgs)];
  std::apply([&ptrs](auto&... v) {
    int k = 0;
    ((ptrs[k++] = static_cast<void*>(&v)), ...);
  }, vals);
  const hipError_t e =
      hipLaunchCooperativeKernel(reinterpret_cast<const void*>(kernel), grid, block, ptrs, 0,
                                 stream);
  if (e == hipErrorCooperativeLaunchTooLarge) {
    (void)hipGetLastError();   // clear it: the caller tries another shape
    return hipErrorInvalidConfiguration;
  }
  return e;
}

}  // namespace lar
