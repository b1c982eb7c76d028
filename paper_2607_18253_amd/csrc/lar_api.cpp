// lar_api.cpp -- host implementation of the C ABI declared in include/lar.h.
//
// Owns the device state of a context (structure-of-arrays in HBM, one slice per
// (scenario, instance) queue), validates snapshots on the host, and enqueues the
// kernels of sfs_kernels.hip on the caller's stream.  Hot calls (estimate, route,
// commit, trace, stats) allocate nothing and never synchronise.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <algorithm>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/lar.h"
#include "sfs_launch.h"

using lar::LaunchEnv;

struct lar_ctx {
  lar_config cfg{};
  int Z = 0, I = 0, mcap = 0, qcap = 0, ks = 0;
  hipStream_t stream = nullptr;
  lar::DevState S{};
  lar::DevTraj T{};
  // parameters on device
  double* pa = nullptr;   // [5][I]: a, b, c, d, e
  int32_t* pi = nullptr;  // [3][I]: B, M, col
  double* row_ttft = nullptr;  // [Z][I] TTFT row of lar_route_step
  uint64_t* xslot = nullptr;   // [Z][2][kMaxCluster][4] candidate posts of the clustered trace
  lar::SyncCtl sync{1000000000ull, -1, -1};   // 10 s wait bound; no post left out
  unsigned long long* work = nullptr;          // [Z] estimate batches of the last trace
  double* lps_wait = nullptr;                  // [Z][I] LPS queueing delays (lar_estimate_lps)
  int32_t tag_next = 0;        // ring tag of the next query tracked for its realised TTFT
  int32_t tag_start = 0;       // tag_next after a (re)load
  lar::DevState snap{};        // one scenario's copy of the last loaded snapshot
  // scheduler limits (lar_set_scheduler): host copy and device [4][I] (chunk cap, KV
  // blocks, log2 block size, context limit)
  bool limited = false;
  std::vector<lar_sched_limits> lim;
  int32_t* plim = nullptr;
  int32_t* err = nullptr;
  size_t tail_elems = 0;  // allocated K * Z * I
  bool loaded = false;
  int max_col = 0;
  bool no_ctx_term = false;   // every instance of the loaded pool has d == 0
  lar_status sticky = LAR_OK;
  std::string msg;
  std::vector<void*> allocs;
};

namespace {

lar_status fail(lar_ctx* ctx, lar_status code, const char* fmt, ...) {
  if (ctx) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    ctx->msg = buf;
  }
  return code;
}

#define HIP_TRY(ctx, expr)                                                             \
  do {                                                                                 \
    hipError_t e_ = (expr);                                                            \
    if (e_ != hipSuccess)                                                              \
      return fail(ctx, LAR_E_HIP, "%s: %s", #expr, hipGetErrorString(e_));             \
  } while (0)

template <class T>
lar_status dev_alloc(lar_ctx* ctx, T** p, size_t n) {
  void* q = nullptr;
  hipError_t e = hipMalloc(&q, n ? n * sizeof(T) : 16);
  if (e != hipSuccess) return fail(ctx, LAR_E_HIP, "hipMalloc(%zu): %s", n * sizeof(T),
                                   hipGetErrorString(e));
  ctx->allocs.push_back(q);
  *p = static_cast<T*>(q);
  return LAR_OK;
}

void dev_free(lar_ctx* ctx, void* p) {
  if (!p) return;
  for (auto& a : ctx->allocs)
    if (a == p) { (void)hipFree(p); a = nullptr; }
}

LaunchEnv env_of(const lar_ctx* ctx) {
  LaunchEnv e;
  e.S = ctx->S;
  e.P.a = ctx->pa;
  e.P.b = ctx->pa + ctx->I;
  e.P.c = ctx->pa + 2 * ctx->I;
  e.P.d = ctx->pa + 3 * ctx->I;
  e.P.e = ctx->pa + 4 * ctx->I;
  e.P.B = ctx->pi;
  e.P.M = ctx->pi + ctx->I;
  e.P.col = ctx->pi + 2 * ctx->I;
  e.T = ctx->T;
  e.Z = ctx->Z;
  e.I = ctx->I;
  e.ks = ctx->ks;
  e.max_iters = ctx->cfg.max_iters;
  e.max_prompt = ctx->cfg.max_prompt;
  e.no_ctx_term = ctx->no_ctx_term;
  e.reading = ctx->cfg.flags & 1;
  e.err = ctx->err;
  e.stream = ctx->stream;
  e.xslot = ctx->xslot;
  e.sync = ctx->sync;
  e.work = ctx->work;
  e.limited = ctx->limited;
  e.L.H = ctx->plim;
  e.L.K = ctx->plim + ctx->I;
  e.L.sh = ctx->plim + 2 * ctx->I;
  e.L.X = ctx->plim + 3 * ctx->I;
  return e;
}

lar_status ready(lar_ctx* ctx) {
  if (!ctx) return LAR_E_ARG;
  if (ctx->sticky != LAR_OK) return ctx->sticky;
  if (!ctx->loaded) return fail(ctx, LAR_E_STATE, "no state loaded (call lar_load_state)");
  return LAR_OK;
}

// Largest token budget: the saturating prefix sums of the batch composition add two
// values of at most B each in 32-bit lanes, so 2B must stay below 2^31.
const int64_t kMaxBudget = (int64_t(1) << 30) - 1;

}  // namespace

extern "C" {

lar_status lar_create(lar_ctx** out, const lar_config* cfg) {
  if (!out) return LAR_E_ARG;
  *out = nullptr;
  if (!cfg) return LAR_E_ARG;
  if (cfg->n_scen < 1 || cfg->n_inst < 1 || cfg->max_seqs_cap < 1 || cfg->max_seqs_cap > 1024 ||
      cfg->queue_cap < 1 || cfg->max_prompt < 1 || cfg->max_iters < 1 ||
      (cfg->flags & ~1) != 0)
    return LAR_E_ARG;
  if ((int64_t)cfg->n_scen * cfg->n_inst > (int64_t)1 << 24) return LAR_E_ARG;
  lar_ctx* ctx = new lar_ctx;
  ctx->cfg = *cfg;
  // Test hooks of the cross-workgroup wait, from the environment: LAR_SYNC_TIMEOUT_MS
  // bounds the wait (default 10 s); LAR_TEST_SKIP_POST="member:query" makes one
  // workgroup leave out its post for one query, so the others reach the bound.
  if (const char* v = std::getenv("LAR_SYNC_TIMEOUT_MS")) {
    const long long ms = std::atoll(v);
    if (ms > 0) ctx->sync.spin_ticks = (uint64_t)ms * 100000ull;
  }
  if (const char* v = std::getenv("LAR_TEST_SKIP_POST")) {
    int m = -1, q = -1;
    if (std::sscanf(v, "%d:%d", &m, &q) == 2 && m >= 0 && q >= 0) {
      ctx->sync.skip_cid = m;
      ctx->sync.skip_query = q;
    }
  }
  // Test hook of the realised-TTFT tags: LAR_TEST_TAG_START starts the tag counter
  // near its end, so that a test reaches the wrap (every slot untagged, restart at 0).
  if (const char* v = std::getenv("LAR_TEST_TAG_START")) {
    const long long t0 = std::atoll(v);
    if (t0 > 0 && t0 <= INT32_MAX) ctx->tag_start = (int32_t)t0;
  }
  ctx->Z = cfg->n_scen;
  ctx->I = cfg->n_inst;
  ctx->mcap = cfg->max_seqs_cap;
  ctx->qcap = cfg->queue_cap;
  ctx->ks = 1;
  while (ctx->ks * 64 < ctx->mcap) ctx->ks *= 2;
  ctx->stream = static_cast<hipStream_t>(cfg->stream);
  const size_t ZI = (size_t)ctx->Z * ctx->I;
  lar_status st = LAR_OK;
  auto chk = [&](lar_status s) { if (st == LAR_OK) st = s; };
  const int rcap = ctx->qcap + ctx->mcap;
  auto alloc_state = [&](lar::DevState& D, size_t nq) {
    chk(dev_alloc(ctx, &D.sc, nq));
    chk(dev_alloc(ctx, &D.d_last, nq * ctx->mcap));
    chk(dev_alloc(ctx, &D.d_cx0, nq * ctx->mcap));
    chk(dev_alloc(ctx, &D.d_seq, nq * ctx->mcap));
    chk(dev_alloc(ctx, &D.r_rp, nq * rcap));
    chk(dev_alloc(ctx, &D.r_rd, nq * rcap));
    chk(dev_alloc(ctx, &D.r_cx, nq * rcap));
    chk(dev_alloc(ctx, &D.r_seq, nq * rcap));
    chk(dev_alloc(ctx, &D.r_tag, nq * rcap));
    D.mcap = ctx->mcap;
    D.rcap = rcap;
    D.qcap = ctx->qcap;
  };
  alloc_state(ctx->S, ZI);
  alloc_state(ctx->snap, (size_t)ctx->I);
  chk(dev_alloc(ctx, &ctx->pa, 5 * (size_t)ctx->I));
  chk(dev_alloc(ctx, &ctx->pi, 3 * (size_t)ctx->I));
  chk(dev_alloc(ctx, &ctx->T.E, ZI));
  chk(dev_alloc(ctx, &ctx->T.pre, ZI));
  chk(dev_alloc(ctx, &ctx->T.P, ZI));
  chk(dev_alloc(ctx, &ctx->T.D, ZI));
  chk(dev_alloc(ctx, &ctx->T.C, ZI));
  chk(dev_alloc(ctx, &ctx->T.A, ZI));
  chk(dev_alloc(ctx, &ctx->T.left, ZI));
  chk(dev_alloc(ctx, &ctx->T.ok, ZI));
  chk(dev_alloc(ctx, &ctx->row_ttft, ZI));
  chk(dev_alloc(ctx, &ctx->err, 1));
  chk(dev_alloc(ctx, &ctx->xslot, (size_t)ctx->Z * 2 * lar::kMaxCluster * 4));
  chk(dev_alloc(ctx, &ctx->work, (size_t)ctx->Z));
  chk(dev_alloc(ctx, &ctx->plim, 4 * (size_t)ctx->I));
  chk(dev_alloc(ctx, &ctx->lps_wait, ZI));
  if (st == LAR_OK && hipMemset(ctx->err, 0, sizeof(int32_t)) != hipSuccess)
    st = fail(ctx, LAR_E_HIP, "hipMemset of the error word failed");
  if (st == LAR_OK && hipMemset(ctx->work, 0, sizeof(unsigned long long) * ctx->Z) != hipSuccess)
    st = fail(ctx, LAR_E_HIP, "hipMemset of the work counters failed");
  if (st != LAR_OK) {
    lar_destroy(ctx);
    return st;
  }
  ctx->T.K = 0;
  *out = ctx;
  return LAR_OK;
}

lar_status lar_destroy(lar_ctx* ctx) {
  if (!ctx) return LAR_OK;
  (void)hipStreamSynchronize(ctx->stream);
  for (void* p : ctx->allocs)
    if (p) (void)hipFree(p);
  delete ctx;
  return LAR_OK;
}

const char* lar_error_string(const lar_ctx* ctx) {
  if (!ctx) return "null context";
  return ctx->msg.c_str();
}

lar_status lar_load_state(lar_ctx* ctx, const lar_instance_params* params, const int32_t* offsets,
                          const int32_t* rem_prefill, const int32_t* rem_decode,
                          const int32_t* context, const double* clock_ms) {
  if (!ctx) return LAR_E_ARG;
  if (!params || !offsets || !clock_ms) return fail(ctx, LAR_E_ARG, "null argument");
  const int I = ctx->I, Z = ctx->Z, mcap = ctx->mcap, qcap = ctx->qcap;
  if (offsets[0] != 0) return fail(ctx, LAR_E_ARG, "offsets[0] must be 0");
  for (int j = 0; j < I; ++j)
    if (offsets[j + 1] < offsets[j]) return fail(ctx, LAR_E_ARG, "offsets decrease at %d", j);
  if (offsets[I] > 0 && (!rem_prefill || !rem_decode || !context))
    return fail(ctx, LAR_E_ARG, "null request arrays");
  int max_col = 0;
  int64_t K = 1;
  for (int j = 0; j < I; ++j) {
    const lar_instance_params& p = params[j];
    const double co[5] = {p.a, p.b, p.c, p.d, p.e};
    for (double v : co)
      if (!std::isfinite(v)) return fail(ctx, LAR_E_ARG, "instance %d: non-finite coefficient", j);
    if (p.max_seqs < 1 || p.max_seqs > mcap)
      return fail(ctx, LAR_E_ARG, "instance %d: max_seqs %d outside [1, %d]", j, p.max_seqs, mcap);
    if (p.token_budget < p.max_seqs || p.token_budget > kMaxBudget)
      return fail(ctx, LAR_E_ARG, "instance %d: token_budget %d outside [max_seqs, 2^30 - 1]", j,
                  p.token_budget);
    if (p.col < 0 || p.reserved != 0)
      return fail(ctx, LAR_E_ARG, "instance %d: bad col/reserved", j);
    if (!std::isfinite(clock_ms[j])) return fail(ctx, LAR_E_ARG, "instance %d: bad clock", j);
    if (p.col > max_col) max_col = p.col;
    // decode-only batches the longest query can need after its admission batch:
    // it gets >= 1 token there and >= B - M + 1 per later batch, then one decode batch
    const int64_t room = (int64_t)p.token_budget - p.max_seqs + 1;
    const int64_t k = ((int64_t)ctx->cfg.max_prompt - 1 + room - 1) / room + 1;
    if (k > K) K = k;
  }
  // validate the snapshot and lay it out as the device state of one scenario:
  // decoding requests in slots, the rest (partially prefilled, then waiting) in the
  // prefill ring, every request tagged with its FCFS position
  const int rcap = qcap + mcap;
  std::vector<int32_t> d_last((size_t)I * mcap, 0), d_cx0((size_t)I * mcap, 0),
      d_seq((size_t)I * mcap, 0), r_rp((size_t)I * rcap, 0), r_rd((size_t)I * rcap, 0),
      r_cx((size_t)I * rcap, 0), r_seq((size_t)I * rcap, 0), r_tag((size_t)I * rcap, -1);
  std::vector<lar::QScal> sc(I);
  if (ctx->limited) {
    // under scheduler limits every request stays in the ring, in FCFS order, with
    // its predicted decode cut to the context limit
    for (int j = 0; j < I; ++j) {
      const lar_sched_limits& L = ctx->lim[j];
      int nr = 0, nw = 0, n = 0;
      int64_t held = 0, ps = 0;
      for (int r = offsets[j]; r < offsets[j + 1]; ++r) {
        const int32_t rp = rem_prefill[r], cx = context[r];
        int32_t rd = rem_decode[r];
        if (rp < 0 || rd < 1 || cx < 0 || (rp == 0 && cx == 0))
          return fail(ctx, LAR_E_STATE, "instance %d request %d: invalid (rp %d, rd %d, cx %d)", j,
                      n, rp, rd, cx);
        const int64_t total = (int64_t)cx + rp;
        if (L.max_ctx > 0) {
          if (total >= L.max_ctx)
            return fail(ctx, LAR_E_STATE, "instance %d request %d: context %lld >= max_ctx %d",
                        j, n, (long long)total, L.max_ctx);
          if (rd > L.max_ctx - total) rd = (int32_t)(L.max_ctx - total);
        }
        if (cx > 0) {
          if (nw > 0)
            return fail(ctx, LAR_E_STATE, "instance %d: running request after a waiting one", j);
          if (nr >= params[j].max_seqs)
            return fail(ctx, LAR_E_STATE, "instance %d: more than max_seqs running", j);
          ++nr;
          if (L.kv_blocks > 0) held += (cx + (int64_t)L.block_size - 1) / L.block_size;
        } else {
          if (nw >= qcap)
            return fail(ctx, LAR_E_CAPACITY, "instance %d: more than queue_cap waiting", j);
          ++nw;
        }
        const size_t x = (size_t)j * rcap + n;
        r_rp[x] = rp; r_rd[x] = rd; r_cx[x] = cx; r_seq[x] = n;
        ps += rp;
        ++n;
      }
      if (L.kv_blocks > 0 && held > L.kv_blocks)
        return fail(ctx, LAR_E_STATE, "instance %d: running requests hold %lld > %d KV blocks", j,
                    (long long)held, L.kv_blocks);
      lar::QScal q{};
      q.n_dec = 0;
      q.n_part = nr;
      q.n_pre = n;
      q.head = 0;
      q.next_seq = n;
      q.pre_sum = ps;
      q.clock = clock_ms[j];
      sc[j] = q;
    }
  }
  for (int j = 0; j < I && !ctx->limited; ++j) {
    int nr = 0, nw = 0, nd = 0, np = 0, npart = 0;
    int64_t c0 = 0, ps = 0;
    for (int r = offsets[j]; r < offsets[j + 1]; ++r) {
      const int32_t rp = rem_prefill[r], rd = rem_decode[r], cx = context[r];
      const int seq = r - offsets[j];
      if (rp < 0 || rd < 1 || cx < 0 || (rp == 0 && cx == 0))
        return fail(ctx, LAR_E_STATE, "instance %d request %d: invalid (rp %d, rd %d, cx %d)", j,
                    seq, rp, rd, cx);
      if (cx > 0) {
        if (nw > 0)
          return fail(ctx, LAR_E_STATE, "instance %d: running request after a waiting one", j);
        if (nr >= params[j].max_seqs)
          return fail(ctx, LAR_E_STATE, "instance %d: more than max_seqs running", j);
        ++nr;
      } else {
        if (nw >= qcap)
          return fail(ctx, LAR_E_CAPACITY, "instance %d: more than queue_cap waiting", j);
        ++nw;
      }
      if (rp == 0) {   // decoding: last batch = rd (batch counter starts at 0)
        d_last[(size_t)j * mcap + nd] = rd;
        d_cx0[(size_t)j * mcap + nd] = cx;
        d_seq[(size_t)j * mcap + nd] = seq;
        c0 += cx;
        ++nd;
      } else {
        r_rp[(size_t)j * rcap + np] = rp;
        r_rd[(size_t)j * rcap + np] = rd;
        r_cx[(size_t)j * rcap + np] = cx;
        r_seq[(size_t)j * rcap + np] = seq;
        ps += rp;
        if (cx > 0) ++npart;
        ++np;
      }
    }
    lar::QScal q{};
    q.g = 0;
    q.n_dec = nd;
    q.n_part = npart;
    q.n_pre = np;
    q.head = 0;
    q.next_seq = offsets[j + 1] - offsets[j];
    q.c0sum = c0;
    q.pre_sum = ps;
    q.clock = clock_ms[j];
    q.iters = 0;
    sc[j] = q;
  }
  // trajectory tail buffers (grow only)
  const size_t ZI = (size_t)Z * I;
  if ((size_t)K * ZI > ctx->tail_elems) {
    dev_free(ctx, ctx->T.tailD);
    dev_free(ctx, ctx->T.tailC);
    ctx->T.tailD = nullptr;
    ctx->T.tailC = nullptr;
    ctx->tail_elems = 0;
    lar_status s = dev_alloc(ctx, &ctx->T.tailD, (size_t)K * ZI);
    if (s == LAR_OK) s = dev_alloc(ctx, &ctx->T.tailC, (size_t)K * ZI);
    if (s != LAR_OK) return s;
    ctx->tail_elems = (size_t)K * ZI;
  }
  ctx->T.K = (int32_t)K;
  // parameters
  std::vector<double> pa(5 * (size_t)I);
  std::vector<int32_t> pi(3 * (size_t)I);
  for (int j = 0; j < I; ++j) {
    pa[j] = params[j].a;
    pa[I + j] = params[j].b;
    pa[2 * I + j] = params[j].c;
    pa[3 * I + j] = params[j].d;
    pa[4 * I + j] = params[j].e;
    pi[j] = params[j].token_budget;
    pi[I + j] = params[j].max_seqs;
    pi[2 * I + j] = params[j].col;
  }
  ctx->no_ctx_term = true;
  for (int j = 0; j < I; ++j)
    if (params[j].d != 0.0) ctx->no_ctx_term = false;
  hipStream_t s = ctx->stream;
  HIP_TRY(ctx, hipStreamSynchronize(s));
  HIP_TRY(ctx, hipMemcpy(ctx->pa, pa.data(), pa.size() * sizeof(double), hipMemcpyHostToDevice));
  HIP_TRY(ctx, hipMemcpy(ctx->pi, pi.data(), pi.size() * sizeof(int32_t), hipMemcpyHostToDevice));
  lar::DevState& sn = ctx->snap;
  HIP_TRY(ctx, hipMemcpy(sn.sc, sc.data(), sc.size() * sizeof(lar::QScal), hipMemcpyHostToDevice));
  HIP_TRY(ctx, hipMemcpy(sn.d_last, d_last.data(), d_last.size() * 4, hipMemcpyHostToDevice));
  HIP_TRY(ctx, hipMemcpy(sn.d_cx0, d_cx0.data(), d_cx0.size() * 4, hipMemcpyHostToDevice));
  HIP_TRY(ctx, hipMemcpy(sn.d_seq, d_seq.data(), d_seq.size() * 4, hipMemcpyHostToDevice));
  HIP_TRY(ctx, hipMemcpy(sn.r_rp, r_rp.data(), r_rp.size() * 4, hipMemcpyHostToDevice));
  HIP_TRY(ctx, hipMemcpy(sn.r_rd, r_rd.data(), r_rd.size() * 4, hipMemcpyHostToDevice));
  HIP_TRY(ctx, hipMemcpy(sn.r_cx, r_cx.data(), r_cx.size() * 4, hipMemcpyHostToDevice));
  HIP_TRY(ctx, hipMemcpy(sn.r_seq, r_seq.data(), r_seq.size() * 4, hipMemcpyHostToDevice));
  HIP_TRY(ctx, hipMemcpy(sn.r_tag, r_tag.data(), r_tag.size() * 4, hipMemcpyHostToDevice));
  ctx->loaded = true;
  ctx->sticky = LAR_OK;
  {
    lar_status rs = lar_reload_state(ctx);
    if (rs != LAR_OK) { ctx->loaded = false; return rs; }
  }
  HIP_TRY(ctx, hipStreamSynchronize(s));
  ctx->max_col = max_col;
  ctx->msg.clear();
  return LAR_OK;
}

lar_status lar_set_scheduler(lar_ctx* ctx, const lar_sched_limits* limits) {
  if (!ctx) return LAR_E_ARG;
  const int I = ctx->I;
  std::vector<int32_t> dev(4 * (size_t)I, 0);
  if (limits) {
    for (int j = 0; j < I; ++j) {
      const lar_sched_limits& L = limits[j];
      if (L.chunk_cap < 0 || L.kv_blocks < 0 || L.max_ctx < 0)
        return fail(ctx, LAR_E_ARG, "instance %d: negative limit", j);
      int sh = 0;
      if (L.kv_blocks > 0) {
        if (L.block_size < 1 || L.block_size > 65536 || (L.block_size & (L.block_size - 1)))
          return fail(ctx, LAR_E_ARG, "instance %d: block_size %d not a power of two in "
                      "[1, 65536]", j, L.block_size);
        if (L.max_ctx < 1 || (int64_t)L.kv_blocks * L.block_size < L.max_ctx)
          return fail(ctx, LAR_E_ARG, "instance %d: a KV cache needs max_ctx > 0 and "
                      "kv_blocks * block_size >= max_ctx", j);
        while ((1 << sh) < L.block_size) ++sh;
      }
      dev[j] = L.chunk_cap;
      dev[I + j] = L.kv_blocks;
      dev[2 * I + j] = sh;
      dev[3 * I + j] = L.max_ctx;
    }
  }
  HIP_TRY(ctx, hipStreamSynchronize(ctx->stream));
  HIP_TRY(ctx, hipMemcpy(ctx->plim, dev.data(), dev.size() * sizeof(int32_t),
                         hipMemcpyHostToDevice));
  ctx->limited = limits != nullptr;
  ctx->lim.assign(limits ? limits : nullptr, limits ? limits + I : nullptr);
  ctx->loaded = false;   // the state layout depends on the scheduler: load again
  ctx->msg.clear();
  return LAR_OK;
}

// Z copies of one scenario's array of n 32-bit words, dst[z * n + i] = src[i]: the
// snapshot re-installed for every scenario in one launch per array.
__global__ void k_replicate(uint32_t* dst, const uint32_t* src, int64_t n, int64_t total) {
  for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < total;
       x += (int64_t)gridDim.x * blockDim.x)
    dst[x] = src[x % n];
}

static hipError_t replicate(void* dst, const void* src, size_t bytes, int Z, hipStream_t s) {
  const int64_t n = (int64_t)(bytes / 4), total = n * Z;
  if (total == 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(k_replicate, dim3((unsigned)blocks), dim3(256), 0, s, (uint32_t*)dst,
                     (const uint32_t*)src, n, total);
  return hipGetLastError();
}

lar_status lar_reload_state(lar_ctx* ctx) {
  if (!ctx) return LAR_E_ARG;
  if (!ctx->loaded) return fail(ctx, LAR_E_STATE, "no state loaded (call lar_load_state)");
  const size_t I = ctx->I, mcap = ctx->mcap, rcap = ctx->snap.rcap;
  const lar::DevState& sn = ctx->snap;
  const lar::DevState& S = ctx->S;
  hipStream_t s = ctx->stream;
  const int Z = ctx->Z;
  static_assert(sizeof(lar::QScal) % 4 == 0, "QScal is copied in 32-bit words");
  HIP_TRY(ctx, replicate(S.sc, sn.sc, I * sizeof(lar::QScal), Z, s));
  HIP_TRY(ctx, replicate(S.d_last, sn.d_last, I * mcap * 4, Z, s));
  HIP_TRY(ctx, replicate(S.d_cx0, sn.d_cx0, I * mcap * 4, Z, s));
  HIP_TRY(ctx, replicate(S.d_seq, sn.d_seq, I * mcap * 4, Z, s));
  HIP_TRY(ctx, replicate(S.r_rp, sn.r_rp, I * rcap * 4, Z, s));
  HIP_TRY(ctx, replicate(S.r_rd, sn.r_rd, I * rcap * 4, Z, s));
  HIP_TRY(ctx, replicate(S.r_cx, sn.r_cx, I * rcap * 4, Z, s));
  HIP_TRY(ctx, replicate(S.r_seq, sn.r_seq, I * rcap * 4, Z, s));
  HIP_TRY(ctx, replicate(S.r_tag, sn.r_tag, I * rcap * 4, Z, s));
  ctx->tag_next = ctx->tag_start;   // every ring entry is untracked again
  HIP_TRY(ctx, lar::launch_clear_error(env_of(ctx)));
  ctx->sticky = LAR_OK;
  return LAR_OK;
}

lar_status lar_estimate_ttft(lar_ctx* ctx, int32_t n_q, const int32_t* q_prefill, double t_ms,
                             double* ttft_ms, int32_t* iters) {
  lar_status st = ready(ctx);
  if (st != LAR_OK) return st;
  if (n_q < 0) return fail(ctx, LAR_E_ARG, "n_q < 0");
  if (n_q == 0) return LAR_OK;
  if (!q_prefill || !ttft_ms) return fail(ctx, LAR_E_ARG, "null argument");
  if (!std::isfinite(t_ms)) return fail(ctx, LAR_E_ARG, "t_ms not finite");
  if ((int64_t)ctx->Z * n_q * ctx->I > ((int64_t)1 << 40))
    return fail(ctx, LAR_E_ARG, "output too large");
  const LaunchEnv env = env_of(ctx);
  HIP_TRY(ctx, lar::launch_traj(env, nullptr, t_ms));
  HIP_TRY(ctx, lar::launch_est(env, n_q, q_prefill, nullptr, t_ms, ttft_ms, iters));
  return LAR_OK;
}

// Row argmax, Lagrangian (tau == nullptr, w_lat given) or constrained (tau given).
static lar_status route_rows(lar_ctx* ctx, int32_t n_q, const double* ttft_ms,
                             const double* tau_ms, const double* acc, const double* cost,
                             int32_t n_cols, const double* w_cost, const double* w_lat,
                             int32_t* choice, double* chosen_ttft, double* utility) {
  lar_status st = ready(ctx);
  if (st != LAR_OK) return st;
  if (n_q < 0) return fail(ctx, LAR_E_ARG, "n_q < 0");
  if (n_q == 0) return LAR_OK;
  if (!ttft_ms || !acc || !cost || !w_cost || !choice || (!tau_ms && !w_lat))
    return fail(ctx, LAR_E_ARG, "null argument");
  if (n_cols <= ctx->max_col)
    return fail(ctx, LAR_E_ARG, "n_cols %d does not cover instance column %d", n_cols, ctx->max_col);
  if ((int64_t)ctx->Z * n_q > INT32_MAX) return fail(ctx, LAR_E_ARG, "too many rows");
  const LaunchEnv env = env_of(ctx);
  HIP_TRY(ctx, lar::launch_route(env, n_q, ttft_ms, (int64_t)n_q * ctx->I, acc, cost, n_cols,
                                 w_cost, tau_ms ? w_cost : w_lat, tau_ms, choice, chosen_ttft,
                                 utility, n_q, 0));
  return LAR_OK;
}

lar_status lar_route(lar_ctx* ctx, int32_t n_q, const double* ttft_ms, const double* acc,
                     const double* cost, int32_t n_cols, const double* w_cost,
                     const double* w_lat, int32_t* choice, double* chosen_ttft,
                     double* utility) {
  return route_rows(ctx, n_q, ttft_ms, nullptr, acc, cost, n_cols, w_cost, w_lat, choice,
                    chosen_ttft, utility);
}

lar_status lar_route_constrained(lar_ctx* ctx, int32_t n_q, const double* ttft_ms,
                                 const double* tau_ms, const double* acc, const double* cost,
                                 int32_t n_cols, const double* w_cost, int32_t* choice,
                                 double* chosen_ttft, double* utility) {
  return route_rows(ctx, n_q, ttft_ms, tau_ms, acc, cost, n_cols, w_cost, nullptr, choice,
                    chosen_ttft, utility);
}

lar_status lar_ttft_targets(lar_ctx* ctx, int32_t n, const int32_t* q_prefill,
                            const double* u_ms, const double* v, double* tau_ms) {
  if (!ctx) return LAR_E_ARG;
  if (n < 0) return fail(ctx, LAR_E_ARG, "n < 0");
  if (n == 0) return LAR_OK;
  if (!q_prefill || !u_ms || !v || !tau_ms) return fail(ctx, LAR_E_ARG, "null argument");
  HIP_TRY(ctx, lar::launch_targets(ctx->stream, n, q_prefill, u_ms, v, tau_ms));
  return LAR_OK;
}

lar_status lar_commit(lar_ctx* ctx, const int32_t* choice, int32_t q_prefill, int32_t q_decode,
                      double t_next_ms) {
  lar_status st = ready(ctx);
  if (st != LAR_OK) return st;
  if (choice && q_prefill < 1) return fail(ctx, LAR_E_ARG, "q_prefill < 1");
  if (!std::isfinite(t_next_ms)) return fail(ctx, LAR_E_ARG, "t_next_ms not finite");
  const LaunchEnv env = env_of(ctx);
  HIP_TRY(ctx, lar::launch_commit(env, choice, 1, nullptr, nullptr, q_prefill, q_decode, nullptr,
                                  t_next_ms));
  return LAR_OK;
}

lar_status lar_route_step(lar_ctx* ctx, const int32_t* q_prefill, const int32_t* q_decode,
                          const double* t_ms, const double* t_next_ms, const double* acc,
                          const double* cost, int32_t n_cols, const double* w_cost,
                          const double* w_lat, const double* tau_ms, int32_t* choice,
                          double* chosen_ttft, double* utility) {
  lar_status st = ready(ctx);
  if (st != LAR_OK) return st;
  if (!q_prefill || !q_decode || !t_ms || !t_next_ms || !acc || !cost || !w_cost || !choice ||
      (!tau_ms && !w_lat))
    return fail(ctx, LAR_E_ARG, "null argument");
  if (n_cols <= ctx->max_col)
    return fail(ctx, LAR_E_ARG, "n_cols %d does not cover instance column %d", n_cols, ctx->max_col);
  // the four calls of one routing step, every query value read from device memory
  const LaunchEnv env = env_of(ctx);
  HIP_TRY(ctx, lar::launch_traj(env, t_ms, 0.0));
  HIP_TRY(ctx, lar::launch_est(env, 1, q_prefill, t_ms, 0.0, ctx->row_ttft, nullptr));
  HIP_TRY(ctx, lar::launch_route(env, 1, ctx->row_ttft, (int64_t)ctx->I, acc, cost, n_cols,
                                 w_cost, tau_ms ? w_cost : w_lat, tau_ms, choice, chosen_ttft,
                                 utility, 1, 0));
  HIP_TRY(ctx, lar::launch_commit(env, choice, 1, q_prefill, q_decode, 0, 0, t_next_ms, 0.0));
  return LAR_OK;
}

static lar_status trace_rows(lar_ctx* ctx, int32_t n_q, const int32_t* q_prefill,
                             const int32_t* q_decode, const double* q_t_ms, double t_after_ms,
                             const double* tau_ms, const double* acc, const double* cost,
                             int32_t n_cols, const double* w_cost, const double* w_lat,
                             int32_t* choice, double* chosen_ttft, double* utility,
                             double* realized) {
  lar_status st = ready(ctx);
  if (st != LAR_OK) return st;
  if (n_q < 0) return fail(ctx, LAR_E_ARG, "n_q < 0");
  if (n_q == 0) return LAR_OK;
  if (!q_prefill || !q_decode || !q_t_ms || !acc || !cost || !w_cost || !choice ||
      (!tau_ms && !w_lat))
    return fail(ctx, LAR_E_ARG, "null argument");
  if (n_cols <= ctx->max_col)
    return fail(ctx, LAR_E_ARG, "n_cols %d does not cover instance column %d", n_cols, ctx->max_col);
  if (!std::isfinite(t_after_ms)) return fail(ctx, LAR_E_ARG, "t_after_ms not finite");
  const LaunchEnv env = env_of(ctx);
  lar::TraceArgs ta;
  ta.N = n_q;
  ta.qp = q_prefill;
  ta.qd = q_decode;
  ta.qt = q_t_ms;
  ta.t_after = t_after_ms;
  ta.acc = acc;
  ta.cost = cost;
  ta.n_cols = n_cols;
  ta.w_cost = w_cost;
  ta.w_lat = tau_ms ? w_cost : w_lat;   // unused under the constrained objective
  ta.tau = tau_ms;
  ta.choice = choice;
  ta.chosen_ttft = chosen_ttft;
  ta.utility = utility;
  ta.realized = realized;
  ta.tag0 = 0;
  if (realized) {
    // tags tag0 .. tag0 + N - 1 must stay positive int32; when the counter would run
    // past that, every ring entry is marked untracked and the counter starts over
    if (ctx->tag_next > INT32_MAX - n_q) {
      HIP_TRY(ctx, lar::launch_untag(env));
      ctx->tag_next = 0;
    }
    ta.tag0 = ctx->tag_next;
    ctx->tag_next += n_q;
  }
  HIP_TRY(ctx, lar::launch_trace(env, ta));
  return LAR_OK;
}

lar_status lar_route_trace(lar_ctx* ctx, int32_t n_q, const int32_t* q_prefill,
                           const int32_t* q_decode, const double* q_t_ms, double t_after_ms,
                           const double* acc, const double* cost, int32_t n_cols,
                           const double* w_cost, const double* w_lat, int32_t* choice,
                           double* chosen_ttft, double* utility, double* realized_ttft) {
  return trace_rows(ctx, n_q, q_prefill, q_decode, q_t_ms, t_after_ms, nullptr, acc, cost, n_cols,
                    w_cost, w_lat, choice, chosen_ttft, utility, realized_ttft);
}

lar_status lar_route_trace_constrained(lar_ctx* ctx, int32_t n_q, const int32_t* q_prefill,
                                       const int32_t* q_decode, const double* q_t_ms,
                                       double t_after_ms, const double* tau_ms, const double* acc,
                                       const double* cost, int32_t n_cols, const double* w_cost,
                                       int32_t* choice, double* chosen_ttft, double* utility,
                                       double* realized_ttft) {
  return trace_rows(ctx, n_q, q_prefill, q_decode, q_t_ms, t_after_ms, tau_ms, acc, cost, n_cols,
                    w_cost, nullptr, choice, chosen_ttft, utility, realized_ttft);
}

lar_status lar_stats(lar_ctx* ctx, int32_t n_q, const int32_t* choice, const double* chosen_ttft,
                     const double* acc, const double* cost, int32_t n_cols,
                     const double* w_cost, double* stats) {
  lar_status st = ready(ctx);
  if (st != LAR_OK) return st;
  if (n_q < 1) return fail(ctx, LAR_E_ARG, "n_q < 1");
  if (!choice || !chosen_ttft || !acc || !cost || !w_cost || !stats)
    return fail(ctx, LAR_E_ARG, "null argument");
  if (n_cols <= ctx->max_col)
    return fail(ctx, LAR_E_ARG, "n_cols %d does not cover instance column %d", n_cols, ctx->max_col);
  const LaunchEnv env = env_of(ctx);
  HIP_TRY(ctx, lar::launch_stats(env, n_q, choice, chosen_ttft, acc, cost, n_cols, w_cost, stats));
  return LAR_OK;
}

lar_status lar_ontime_utility(lar_ctx* ctx, int32_t n_q, const int32_t* choice,
                              const double* realized_ttft, const double* tau_ms, const double* acc,
                              const double* cost, int32_t n_cols, const double* w_cost,
                              double* out) {
  lar_status st = ready(ctx);
  if (st != LAR_OK) return st;
  if (n_q < 1) return fail(ctx, LAR_E_ARG, "n_q < 1");
  if (!choice || !realized_ttft || !tau_ms || !acc || !cost || !w_cost || !out)
    return fail(ctx, LAR_E_ARG, "null argument");
  if (n_cols <= ctx->max_col)
    return fail(ctx, LAR_E_ARG, "n_cols %d does not cover instance column %d", n_cols, ctx->max_col);
  const LaunchEnv env = env_of(ctx);
  HIP_TRY(ctx, lar::launch_ontime(env, n_q, choice, realized_ttft, tau_ms, acc, cost, n_cols,
                                  w_cost, out));
  return LAR_OK;
}

lar_status lar_estimate_lps(lar_ctx* ctx, const lar_lps_params* params, int32_t mode,
                            int32_t n_q, const int32_t* q_prefill, double* ttft_ms) {
  if (!ctx) return LAR_E_ARG;
  if (ctx->sticky != LAR_OK) return ctx->sticky;
  if (n_q < 0) return fail(ctx, LAR_E_ARG, "n_q < 0");
  if (mode != LAR_LPS_POISSON && mode != LAR_LPS_VARIABILITY)
    return fail(ctx, LAR_E_ARG, "unknown LPS mode %d", mode);
  if (n_q == 0) return LAR_OK;
  if (!params || !q_prefill || !ttft_ms) return fail(ctx, LAR_E_ARG, "null argument");
  if ((int64_t)ctx->Z * n_q * ((ctx->I + 255) / 256) > 0x7fffffff)
    return fail(ctx, LAR_E_ARG, "output too large");
  HIP_TRY(ctx, lar::launch_lps(env_of(ctx), params, mode, ctx->lps_wait, n_q, q_prefill, ttft_ms));
  return LAR_OK;
}

lar_status lar_trace_work(lar_ctx* ctx, int64_t* estimate_batches) {
  if (!ctx || !estimate_batches) return LAR_E_ARG;
  HIP_TRY(ctx, hipStreamSynchronize(ctx->stream));
  HIP_TRY(ctx, hipMemcpy(estimate_batches, ctx->work, sizeof(int64_t) * ctx->Z,
                         hipMemcpyDeviceToHost));
  return LAR_OK;
}

lar_status lar_sync(lar_ctx* ctx) {
  if (!ctx) return LAR_E_ARG;
  HIP_TRY(ctx, hipStreamSynchronize(ctx->stream));
  if (ctx->sticky == LAR_OK) {
    int32_t e = 0;
    HIP_TRY(ctx, hipMemcpy(&e, ctx->err, sizeof e, hipMemcpyDeviceToHost));
    if (e != 0) {
      ctx->sticky = e;
      fail(ctx, e, "device error %d (sticky until lar_load_state)", e);
    }
  }
  return ctx->sticky;
}

lar_status lar_read_state(lar_ctx* ctx, int32_t scen, int32_t* offsets, int32_t* rem_prefill,
                          int32_t* rem_decode, int32_t* context, double* clock_ms,
                          int64_t* iterations_run, int64_t out_cap, int64_t* n_total) {
  if (!ctx) return LAR_E_ARG;
  if (!ctx->loaded) return fail(ctx, LAR_E_STATE, "no state loaded");
  if (scen < 0 || scen >= ctx->Z) return fail(ctx, LAR_E_ARG, "scenario out of range");
  if (!offsets || !clock_ms || !iterations_run || !n_total || out_cap < 0)
    return fail(ctx, LAR_E_ARG, "null argument");
  lar_status st = lar_sync(ctx);
  if (st == LAR_E_HIP) return st;
  const int I = ctx->I, mcap = ctx->mcap, rcap = ctx->S.rcap;
  const size_t o = (size_t)scen * I;
  std::vector<lar::QScal> sc(I);
  std::vector<int32_t> d_last((size_t)I * mcap), d_cx0((size_t)I * mcap), d_seq((size_t)I * mcap),
      r_rp((size_t)I * rcap), r_rd((size_t)I * rcap), r_cx((size_t)I * rcap), r_seq((size_t)I * rcap);
  const lar::DevState& S = ctx->S;
  const hipMemcpyKind k = hipMemcpyDeviceToHost;
  HIP_TRY(ctx, hipMemcpy(sc.data(), S.sc + o, I * sizeof(lar::QScal), k));
  HIP_TRY(ctx, hipMemcpy(d_last.data(), S.d_last + o * mcap, d_last.size() * 4, k));
  HIP_TRY(ctx, hipMemcpy(d_cx0.data(), S.d_cx0 + o * mcap, d_cx0.size() * 4, k));
  HIP_TRY(ctx, hipMemcpy(d_seq.data(), S.d_seq + o * mcap, d_seq.size() * 4, k));
  HIP_TRY(ctx, hipMemcpy(r_rp.data(), S.r_rp + o * rcap, r_rp.size() * 4, k));
  HIP_TRY(ctx, hipMemcpy(r_rd.data(), S.r_rd + o * rcap, r_rd.size() * 4, k));
  HIP_TRY(ctx, hipMemcpy(r_cx.data(), S.r_cx + o * rcap, r_cx.size() * 4, k));
  HIP_TRY(ctx, hipMemcpy(r_seq.data(), S.r_seq + o * rcap, r_seq.size() * 4, k));
  int64_t total = 0;
  for (int j = 0; j < I; ++j) {
    clock_ms[j] = sc[j].clock;
    iterations_run[j] = sc[j].iters;
    total += sc[j].n_dec + sc[j].n_pre;
  }
  *n_total = total;
  if (total > out_cap) return fail(ctx, LAR_E_CAPACITY, "output arrays hold %lld < %lld",
                                   (long long)out_cap, (long long)total);
  if (total > 0 && (!rem_prefill || !rem_decode || !context))
    return fail(ctx, LAR_E_ARG, "null request arrays");
  // merge decoding requests and the prefill list back into arrival order
  struct Req { int32_t seq, rp, rd, cx; };
  std::vector<Req> reqs;
  int64_t pos = 0;
  offsets[0] = 0;
  for (int j = 0; j < I; ++j) {
    const lar::QScal& q = sc[j];
    reqs.clear();
    for (int s2 = 0; s2 < q.n_dec; ++s2) {
      const size_t x = (size_t)j * mcap + s2;
      reqs.push_back({d_seq[x], 0, d_last[x] - q.g, d_cx0[x] + q.g});
    }
    for (int e = 0; e < q.n_pre; ++e) {
      const size_t x = (size_t)j * rcap + (q.head + e) % rcap;
      reqs.push_back({r_seq[x], r_rp[x], r_rd[x], r_cx[x]});
    }
    std::sort(reqs.begin(), reqs.end(), [](const Req& a, const Req& b) { return a.seq < b.seq; });
    for (const Req& r : reqs) {
      rem_prefill[pos] = r.rp;
      rem_decode[pos] = r.rd;
      context[pos] = r.cx;
      ++pos;
    }
    offsets[j + 1] = (int32_t)pos;
  }
  return ctx->sticky;
}

}  // extern "C"
