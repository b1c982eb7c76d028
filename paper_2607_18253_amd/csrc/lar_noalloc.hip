// lar_noalloc.hip -- the what-if estimate and route (lar_estimate_ttft followed by
// lar_route, one scenario) for callers that cannot allocate device memory: code
// under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
// It needs no context.  The snapshot comes in device memory; every intermediate
// buffer -- the queues' device layout, the per-instance coefficients, the background
// trajectories and their decode-only tails -- lives in one file-scope device array,
// `scratch`, of which each GPU holds its own copy until the process ends.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>

#include "../../include/lar.h"
#include "sfs_launch.h"

namespace {

constexpr size_t kScratchBytes = size_t(32) << 20;   // per GPU
constexpr int kNoAllocTail = 64;   // decode-only batches recorded after an admission batch
constexpr int kMaxDevices = 64;

}  // namespace

// The whole working memory of lar_whatif_noalloc on one GPU.  Host code never uses
// this name as an address: it takes the device address from hipGetSymbolAddress
// (once per device) and passes that to the kernels.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

using namespace lar;

std::mutex g_mu;
void* g_scratch[kMaxDevices];   // device address of `scratch` per device, once looked up

thread_local char g_msg[256];   // detail of this thread's last failed call

lar_status fail(lar_status code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_msg, sizeof g_msg, fmt, ap);
  va_end(ap);
  return code;
}

// Device address of the current device's `scratch`, looked up on the first call on
// that device.
lar_status scratch_address(unsigned char** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return fail(LAR_E_HIP, "no current device");
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(LAR_E_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch[dev] = p;
  }
  *out = static_cast<unsigned char*>(g_scratch[dev]);
  return LAR_OK;
}

// Byte offsets of the arrays inside `scratch`, each 256-byte aligned.
struct Layout {
  size_t sc, pa, pi, d_last, d_cx0, d_seq, r_rp, r_rd, r_cx, r_seq;
  size_t E, pre, P, D, C, A, left, ok, tailD, tailC, K, end;
};

Layout layout_for(size_t I, size_t mcap, size_t rcap) {
  Layout L{};
  size_t at = 0;
  auto take = [&at](size_t bytes) {
    const size_t o = at;
    at += (bytes + 255) / 256 * 256;
    return o;
  };
  L.sc = take(I * sizeof(QScal));
  L.pa = take(5 * I * sizeof(double));
  L.pi = take(3 * I * sizeof(int32_t));
  L.d_last = take(I * mcap * 4);
  L.d_cx0 = take(I * mcap * 4);
  L.d_seq = take(I * mcap * 4);
  L.r_rp = take(I * rcap * 4);
  L.r_rd = take(I * rcap * 4);
  L.r_cx = take(I * rcap * 4);
  L.r_seq = take(I * rcap * 4);
  L.E = take(I * 8);
  L.pre = take(I * 4);
  L.P = take(I * 8);
  L.D = take(I * 8);
  L.C = take(I * 8);
  L.A = take(I * 8);
  L.left = take(I * 4);
  L.ok = take(I * 4);
  L.tailD = take(kNoAllocTail * I * 4);
  L.tailC = take(kNoAllocTail * I * 8);
  L.K = take(4);
  L.end = at;
  return L;
}

// Zeroes the error word and the tail count before a call: a kernel, not a memset
// node, so the call can be captured in a graph.
__global__ void k_noalloc_begin(int32_t* status, int32_t* K) {
  *status = 0;
  *K = 0;
}

// One wave per instance: checks instance j of the device snapshot and lays it out as
// the device state of one queue (decoding requests in slots, the prefill list --
// partially prefilled, then waiting requests -- in the ring, each with its FCFS
// position), its coefficients as arrays, and the number of decode-only tail batches
// the longest prompt can need after its admission batch (it gets >= 1 token there
// and >= B - M + 1 in every later batch, then one decode batch).  An instance that
// fails a check gets an empty state and sets the error word, so that the kernels
// after this one only ever see a valid state.
__global__ __launch_bounds__(kWave) void k_noalloc_layout(
    int I, int mcap, int rcap, int max_resident, int max_prompt, int n_cols,
    const lar_instance_params* prm, const int32_t* offsets, const int32_t* rp_in,
    const int32_t* rd_in, const int32_t* cx_in, const double* clock_in, DevState S, double* pa,
    int32_t* pi, int32_t* K, int32_t* err) {
  const int j = blockIdx.x;
  if (j >= I) return;
  const int ln = lane_id();
  const lar_instance_params p = prm[j];
  const double clk = clock_in[j];
  const int lo = offsets[j], hi = offsets[j + 1];
  const bool coef_ok = __builtin_isfinite(p.a) && __builtin_isfinite(p.b) && __builtin_isfinite(p.c) &&
                       __builtin_isfinite(p.d) && __builtin_isfinite(p.e);
  const bool prm_ok = coef_ok && p.max_seqs >= 1 && p.max_seqs <= mcap &&
                      p.token_budget >= p.max_seqs && p.token_budget <= (1 << 30) - 1 &&
                      p.col >= 0 && p.col < n_cols && p.reserved == 0 && __builtin_isfinite(clk);
  const int n = hi - lo;
  bool ok = prm_ok && n >= 0 && n <= max_resident && lo >= 0 && (j > 0 || lo == 0);
  int code = prm_ok ? kErrState : kErrArg;
  int nd = 0, np = 0, npart = 0, nrun = 0;
  bool seen_waiting = false;
  int64_t c0 = 0, ps = 0;
  const int64_t db = (int64_t)j * mcap, rb = (int64_t)j * rcap;
  for (int base = 0; ok && base < n; base += kWave) {
    const int idx = base + ln;
    const bool in = idx < n;
    int rp = 0, rd = 1, cx = 1;
    if (in) { rp = rp_in[lo + idx]; rd = rd_in[lo + idx]; cx = cx_in[lo + idx]; }
    const bool bad = in && (rp < 0 || rd < 1 || cx < 0 || (rp == 0 && cx == 0));
    const uint64_t run = ballot(in && cx > 0), wait = ballot(in && cx == 0);
    // running requests precede waiting ones, at most M of them run
    const bool order_bad = run != 0 && (seen_waiting || (wait != 0 && __builtin_ctzll(wait) <
                                                                      63 - __builtin_clzll(run)));
    nrun += popc(run);
    if (ballot(bad) != 0 || order_bad || nrun > p.max_seqs) { ok = false; break; }
    seen_waiting = seen_waiting || wait != 0;
    const bool dec = in && rp == 0;
    const uint64_t dm = ballot(dec), pm = ballot(in && rp > 0);
    if (dec) {
      const int s = nd + mbcnt(dm);
      S.d_last[db + s] = rd;   // batch counter starts at 0: the last batch is rd
      S.d_cx0[db + s] = cx;
      S.d_seq[db + s] = idx;
    } else if (in) {
      const int r = np + mbcnt(pm);
      S.r_rp[rb + r] = rp;
      S.r_rd[rb + r] = rd;
      S.r_cx[rb + r] = cx;
      S.r_seq[rb + r] = idx;
    }
    c0 += wave_sum64(dec ? (int64_t)cx : 0);
    ps += wave_sum64(dec || !in ? 0 : (int64_t)rp);
    npart += popc(ballot(in && rp > 0 && cx > 0));
    nd += popc(dm);
    np += popc(pm);
  }
  // tail batches of the longest prompt
  int64_t k = 1;
  if (prm_ok) {
    const int64_t room = (int64_t)p.token_budget - p.max_seqs + 1;
    k = ((int64_t)max_prompt - 1 + room - 1) / room + 1;
    if (k > kNoAllocTail) {
      ok = false;
      code = kErrArg;
      k = kNoAllocTail;
    }
  }
  if (ln != 0) return;
  if (!ok) {
    set_error(err, code);
    nd = np = npart = 0;
    c0 = ps = 0;
  }
  QScal q{};
  q.n_dec = nd;
  q.n_part = npart;
  q.n_pre = np;
  q.next_seq = ok ? n : 0;
  q.c0sum = c0;
  q.pre_sum = ps;
  q.clock = ok ? clk : 0.0;
  S.sc[j] = q;
  pa[j] = ok ? p.a : 0.0;
  pa[I + j] = ok ? p.b : 0.0;
  pa[2 * I + j] = ok ? p.c : 0.0;
  pa[3 * I + j] = ok ? p.d : 0.0;
  pa[4 * I + j] = ok ? p.e : 0.0;
  pi[j] = ok ? p.token_budget : 1;
  pi[I + j] = ok ? p.max_seqs : 1;
  pi[2 * I + j] = ok ? p.col : 0;
  atomicMax(K, (int32_t)k);
}

}  // namespace

extern "C" {

lar_status lar_whatif_noalloc(const lar_whatif_config* cfg, const lar_instance_params* params,
                              const int32_t* offsets, const int32_t* rem_prefill,
                              const int32_t* rem_decode, const int32_t* context,
                              const double* clock_ms, int32_t n_q, const int32_t* q_prefill,
                              double t_ms, const double* acc, const double* cost,
                              const double* w_cost, const double* w_lat, double* ttft_ms,
                              int32_t* iters, int32_t* choice, double* chosen_ttft,
                              double* utility, int32_t* status) {
  if (!cfg) return fail(LAR_E_ARG, "null config");
  const int I = cfg->n_inst, mcap = cfg->max_seqs_cap;
  if (I < 1 || mcap < 1 || mcap > 1024 || cfg->max_resident < 0 || cfg->max_prompt < 1 ||
      cfg->n_cols < 1 || cfg->max_iters < 1 || (cfg->flags & ~1) != 0)
    return fail(LAR_E_ARG, "config out of range");
  if (n_q < 0) return fail(LAR_E_ARG, "n_q < 0");
  if (!std::isfinite(t_ms)) return fail(LAR_E_ARG, "t_ms not finite");
  if (!params || !offsets || !clock_ms || !rem_prefill || !rem_decode || !context || !w_cost ||
      !w_lat || !status || (n_q > 0 && (!q_prefill || !acc || !cost || !ttft_ms || !choice)))
    return fail(LAR_E_ARG, "null argument");
  if ((int64_t)n_q * I > ((int64_t)1 << 40)) return fail(LAR_E_ARG, "output too large");
  if (n_q == 0) return LAR_OK;
  const int rcap = cfg->max_resident + mcap;
  const Layout L = layout_for((size_t)I, (size_t)mcap, (size_t)rcap);
  if (L.end > kScratchBytes)
    return fail(LAR_E_CAPACITY, "working memory of %zu bytes exceeds the %zu-byte scratch "
                "(n_inst %d, max_seqs_cap %d, max_resident %d)", L.end, kScratchBytes, I, mcap,
                cfg->max_resident);
  unsigned char* base = nullptr;
  const lar_status st = scratch_address(&base);
  if (st != LAR_OK) return st;
  auto at = [base](size_t off) { return static_cast<void*>(base + off); };

  LaunchEnv env{};
  env.S.sc = static_cast<QScal*>(at(L.sc));
  env.S.d_last = static_cast<int32_t*>(at(L.d_last));
  env.S.d_cx0 = static_cast<int32_t*>(at(L.d_cx0));
  env.S.d_seq = static_cast<int32_t*>(at(L.d_seq));
  env.S.r_rp = static_cast<int32_t*>(at(L.r_rp));
  env.S.r_rd = static_cast<int32_t*>(at(L.r_rd));
  env.S.r_cx = static_cast<int32_t*>(at(L.r_cx));
  env.S.r_seq = static_cast<int32_t*>(at(L.r_seq));
  env.S.r_tag = nullptr;   // no first-token tracking on this path
  env.S.mcap = mcap;
  env.S.rcap = rcap;
  env.S.qcap = cfg->max_resident;
  double* pa = static_cast<double*>(at(L.pa));
  int32_t* pi = static_cast<int32_t*>(at(L.pi));
  env.P.a = pa;
  env.P.b = pa + I;
  env.P.c = pa + 2 * I;
  env.P.d = pa + 3 * I;
  env.P.e = pa + 4 * I;
  env.P.B = pi;
  env.P.M = pi + I;
  env.P.col = pi + 2 * I;
  env.T.E = static_cast<double*>(at(L.E));
  env.T.pre = static_cast<int32_t*>(at(L.pre));
  env.T.P = static_cast<int64_t*>(at(L.P));
  env.T.D = static_cast<int64_t*>(at(L.D));
  env.T.C = static_cast<int64_t*>(at(L.C));
  env.T.A = static_cast<int64_t*>(at(L.A));
  env.T.left = static_cast<int32_t*>(at(L.left));
  env.T.ok = static_cast<int32_t*>(at(L.ok));
  env.T.tailD = static_cast<int32_t*>(at(L.tailD));
  env.T.tailC = static_cast<int64_t*>(at(L.tailC));
  env.T.K = 0;
  int32_t* Kword = static_cast<int32_t*>(at(L.K));
  env.T.Kdev = Kword;
  env.Z = 1;
  env.I = I;
  env.ks = 1;
  while (env.ks * kWave < mcap) env.ks *= 2;
  env.max_iters = cfg->max_iters;
  env.max_prompt = cfg->max_prompt;
  env.reading = cfg->flags & 1;
  env.err = status;
  env.stream = static_cast<hipStream_t>(cfg->stream);
  env.xslot = nullptr;
  env.work = nullptr;
  env.limited = false;

  hipLaunchKernelGGL(k_noalloc_begin, dim3(1), dim3(1), 0, env.stream, status, Kword);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess) {
    hipLaunchKernelGGL(k_noalloc_layout, dim3(I), dim3(kWave), 0, env.stream, I, mcap, rcap,
                       cfg->max_resident, cfg->max_prompt, cfg->n_cols, params, offsets,
                       rem_prefill, rem_decode, context, clock_ms, env.S, pa, pi, Kword, status);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = launch_traj(env, nullptr, t_ms);
  if (e == hipSuccess) e = launch_est(env, n_q, q_prefill, nullptr, t_ms, ttft_ms, iters);
  if (e == hipSuccess)
    e = launch_route(env, n_q, ttft_ms, (int64_t)n_q * I, acc, cost, cfg->n_cols, w_cost, w_lat,
                     nullptr, choice, chosen_ttft, utility, n_q, 0);
  if (e != hipSuccess) return fail(LAR_E_HIP, "launch: %s", hipGetErrorString(e));
  return LAR_OK;
}

const char* lar_noalloc_error_string(void) { return g_msg; }

}  // extern "C"
