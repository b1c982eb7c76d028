// sfs_device.h -- device-side state layout and the event-driven wave batch engine
// for gfx950.
//
// One wavefront owns one (scenario, instance) queue.  The resident set (Sec. 4,
// setup) is split by what a token batch does with each request (Sec. 4.1):
//   * decoding requests (prefill done): one decode token per batch, nothing else,
//     so they are kept lazily as (last, cx0) -- `last` = index of the batch that
//     produces their final predicted token, context = cx0 + g at batch counter g --
//     in unordered VGPR slots (slot s = k*64 + lane).  A batch only has to find the
//     slots whose `last` is due; D and the decode-context sum C are running totals.
//   * the prefill list: running partially prefilled requests, then waiting
//     requests, in arrival (FCFS) order, in an HBM ring.  Its head sits in a
//     64-lane register window; one saturating wave prefix sum of the remaining
//     prefill gives every chunk of the batch.  Fully served entries are always a
//     prefix of the window and move to the decode slots.
// Every request carries its arrival sequence number, so the FCFS list can be
// rebuilt on read-out.  A routed query also carries a tag in the ring (its index
// in a trace, -1 if untracked), read back when the query gets its first token.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lar {

constexpr int kWave = 64;

// Error codes shared with the C ABI (lar.h); kept numerically identical.
constexpr int kErrArg = -1, kErrState = -2, kErrCapacity = -3, kErrIter = -4, kErrSync = -6;

// Per-queue scalars, one 64-byte record per (scenario, instance).
struct alignas(64) QScal {
  int32_t g;         // batches completed since the snapshot (batch counter)
  int32_t n_dec;     // decoding requests
  int32_t n_part;    // running partially prefilled requests (head of the prefill list)
  int32_t n_pre;     // prefill list length (partials + waiting)
  int32_t head;      // ring index of the prefill list head
  int32_t next_seq;  // arrival number of the next appended request
  int64_t c0sum;     // sum of cx0 over decoding requests
  int64_t pre_sum;   // sum of remaining prefill over the prefill list
  double clock;      // instance clock, ms
  int64_t iters;     // batches replayed since the load
  // first-token tracking, kept up to date only by a trace that reports realised
  // TTFT (it zeroes both first)
  int32_t pend;      // prefills completed by the last batch (they decode next batch)
  int32_t ntrk;      // tracked queries of the running trace without a first token
};
static_assert(sizeof(QScal) == 64, "QScal is one 64-byte record");

// Device state of Z*I queues.  Decode slots are compacted (first n_dec valid) in
// HBM; the prefill list is a ring of rcap entries per queue.
struct DevState {
  QScal* sc;                          // [ZI]
  int32_t *d_last, *d_cx0, *d_seq;    // [ZI][mcap]
  int32_t *r_rp, *r_rd, *r_cx, *r_seq;  // [ZI][rcap]
  int32_t* r_tag;                     // [ZI][rcap] query tag of each ring entry
  int32_t mcap, rcap, qcap;           // rcap = qcap + mcap
};

struct DevParams {
  const double *a, *b, *c, *d, *e;    // [I]
  const int32_t *B, *M, *col;         // [I]
};

// Background trajectory of one queue up to the batch in which a new tail query
// would first receive prefill tokens (its admission batch), plus the decode-only
// batches that follow it.
struct DevTraj {
  double* E;            // [ZI] clock folded over the batches before the admission batch
  int32_t* pre;         // [ZI] number of those batches
  int64_t *P, *D, *C, *A;  // [ZI] background features of the admission batch
  int32_t* left;        // [ZI] budget the background leaves in that batch (>= 1)
  int32_t* ok;          // [ZI] 1 = valid; 0 = iteration cap or clock behind t
  int32_t* tailD;       // [K][ZI] decode tokens of the k-th batch after admission
  int64_t* tailC;       // [K][ZI] their context sum
  int32_t K;
  const int32_t* Kdev;  // when set, K is read from device memory (worked out there)
};

__device__ __forceinline__ int tail_count(const DevTraj& tr) { return tr.Kdev ? *tr.Kdev : tr.K; }

struct Coef {
  double a, b, c, d, e;
  int B, M;
};

__device__ __forceinline__ Coef load_coef(const DevParams& pr, int j) {
  Coef k;
  k.a = pr.a[j]; k.b = pr.b[j]; k.c = pr.c[j]; k.d = pr.d[j]; k.e = pr.e[j];
  k.B = pr.B[j]; k.M = pr.M[j];
  return k;
}

// Batch time (Sec. 4.1): ((((a + b*P) + c*D) + d*C) + e*A), one rounding per op.
// P <= B and D <= M fit in 32 bits.  C and A are converted only when their
// coefficient is non-zero; otherwise the term is computed as coef * 0.0, which has
// the same bits as coef * C for every finite C >= 0.
__device__ __forceinline__ double batch_time(const Coef& k, int P, int D, int64_t C, int64_t A) {
  double t = k.a;
  t = __dadd_rn(t, __dmul_rn(k.b, (double)P));
  t = __dadd_rn(t, __dmul_rn(k.c, (double)D));
  t = __dadd_rn(t, __dmul_rn(k.d, k.d != 0.0 ? (double)C : 0.0));
  t = __dadd_rn(t, __dmul_rn(k.e, k.e != 0.0 ? (double)A : 0.0));
  return t;
}

__device__ __forceinline__ void set_error(int32_t* err, int code) { atomicCAS(err, 0, code); }

// ------------------------------------------------------------------ wave primitives
__device__ __forceinline__ int lane_id() { return (int)__lane_id(); }
__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ int popc(uint64_t m) { return __popcll(m); }
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ int lane_last(int x) { return __builtin_amdgcn_readlane(x, kWave - 1); }
__device__ __forceinline__ int lane_read(int x, int l) { return __builtin_amdgcn_readlane(x, l); }

// Number of set bits of m below this lane.
__device__ __forceinline__ int mbcnt(uint64_t m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Inclusive prefix sum over the wave, saturating at cap, with DPP lane moves
// (row_shr within 16-lane rows, then row_bcast:15 / row_bcast:31 across rows).
// Inputs in [0, cap] with cap < 2^30 (the token budget's bound), so a sum of two
// saturated values stays below 2^31: no intermediate overflows;
// min(sat(x), L) == min(x, L) for every L <= cap.
__device__ __forceinline__ int scan_sat(int x, int cap) {
  x = min(x + __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, true), cap);  // row_shr:1
  x = min(x + __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, true), cap);  // row_shr:2
  x = min(x + __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, true), cap);  // row_shr:4
  x = min(x + __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, true), cap);  // row_shr:8
  x = min(x + __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false), cap); // row_bcast:15
  x = min(x + __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false), cap); // row_bcast:31
  return x;
}

// Minimum over the wave (DPP row_shr within rows, then row_bcast across rows; lanes
// without a source keep INT_MAX).
__device__ __forceinline__ int wave_min(int x) {
  const int big = 0x7fffffff;
  x = min(x, __builtin_amdgcn_update_dpp(big, x, 0x111, 0xf, 0xf, false));  // row_shr:1
  x = min(x, __builtin_amdgcn_update_dpp(big, x, 0x112, 0xf, 0xf, false));  // row_shr:2
  x = min(x, __builtin_amdgcn_update_dpp(big, x, 0x114, 0xf, 0xf, false));  // row_shr:4
  x = min(x, __builtin_amdgcn_update_dpp(big, x, 0x118, 0xf, 0xf, false));  // row_shr:8
  x = min(x, __builtin_amdgcn_update_dpp(big, x, 0x142, 0xa, 0xf, false));  // row_bcast:15
  x = min(x, __builtin_amdgcn_update_dpp(big, x, 0x143, 0xc, 0xf, false));  // row_bcast:31
  return uni(__builtin_amdgcn_readlane(x, kWave - 1));
}

// Value of the previous lane (0 in lane 0): DPP wave_shr:1.
__device__ __forceinline__ int prev_lane(int x) {
  return __builtin_amdgcn_update_dpp(0, x, 0x138, 0xf, 0xf, true);
}

// Sum of a 64-bit per-lane value over the lanes set in m (few lanes expected).
__device__ __forceinline__ int64_t sum_lanes64(int64_t v, uint64_t m) {
  int64_t s = 0;
  const int lo = (int)(uint32_t)(uint64_t)v;
  const int hi = (int)(uint32_t)((uint64_t)v >> 32);
  while (m) {
    const int l = __builtin_ctzll(m);
    m &= m - 1;
    s += (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane(hi, l) << 32) |
                   (uint64_t)(uint32_t)__builtin_amdgcn_readlane(lo, l));
  }
  return s;
}

__device__ __forceinline__ int64_t uni64(int64_t x) {
  int lo = uni((int)(uint32_t)(uint64_t)x);
  int hi = uni((int)(uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint64_t)(uint32_t)lo);
}

// Inclusive prefix sums over the wave with DPP lane moves (row_shr within 16-lane
// rows, then row_bcast:15 / row_bcast:31 across rows; lanes without a source add 0).
__device__ __forceinline__ int scan_add32(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, true);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, true);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, true);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, true);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false); // row_bcast:15
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false); // row_bcast:31
  return x;
}

// The same in 64 bits: both halves move together, the carry of the low half goes
// into the high one.
__device__ __forceinline__ int64_t scan_add64(int64_t v) {
  uint32_t lo = (uint32_t)(uint64_t)v, hi = (uint32_t)((uint64_t)v >> 32);
#define LAR_SCAN64_STEP(ctrl, rows, bc)                                                    \
  {                                                                                        \
    const uint32_t l2 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)lo, ctrl, rows, 0xf, bc); \
    const uint32_t h2 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)hi, ctrl, rows, 0xf, bc); \
    const uint32_t nl = lo + l2;                                                           \
    hi = hi + h2 + (nl < lo ? 1u : 0u);                                                    \
    lo = nl;                                                                               \
  }
  LAR_SCAN64_STEP(0x111, 0xf, true)
  LAR_SCAN64_STEP(0x112, 0xf, true)
  LAR_SCAN64_STEP(0x114, 0xf, true)
  LAR_SCAN64_STEP(0x118, 0xf, true)
  LAR_SCAN64_STEP(0x142, 0xa, false)
  LAR_SCAN64_STEP(0x143, 0xc, false)
#undef LAR_SCAN64_STEP
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ int64_t wave_sum64(int64_t x) {
  const int64_t s = scan_add64(x);
  const uint32_t hi = (uint32_t)lane_last((int)(uint32_t)((uint64_t)s >> 32));
  const uint32_t lo = (uint32_t)lane_last((int)(uint32_t)(uint64_t)s);
  return uni64((int64_t)(((uint64_t)hi << 32) | lo));
}

__device__ __forceinline__ int wave_sum32(int x) { return uni(lane_last(scan_add32(x))); }

// ------------------------------------------------------------------ LDS copies of queues
// A queue's state kept in LDS by a persistent kernel: decode slots in the register
// layout (slot s = k*64 + lane), the prefill window, and the scalars.
template <int KS>
struct LdsQueue {
  int dl[KS * kWave], dc[KS * kWave], ds[KS * kWave];
  int wrp[kWave], wrd[kWave], wcx[kWave], wseq[kWave];
  int g, n_dec, n_part, n_pre, head, next_seq, woff, nwin, pend, ntrk, ptag_ok;
  int64_t c0sum, pre_sum, iters;
  double clock;
};

// The per-lane tracking registers of a queue (see Queue), kept beside its LDS copy
// by kernels that track first tokens.
struct LdsTags {
  int wtag[kWave], ptag[kWave];
};

// LDS words per wave of the staging area that step() uses to move completed
// prefills into decode slots (one more row when it also moves their tags).
template <bool TRK>
constexpr int stage_words() { return (TRK ? 4 : 3) * kWave; }

// ------------------------------------------------------------------ the batch engine
struct StepOut {
  int P, D;
  int64_t C, A;
  int h0;    // ring head before the batch
  int pn;    // prefills completed by the batch before (first decode in this one)
  int nd;    // prefills completed by this batch: ring entries h0 .. h0 + nd - 1
  int pt;    // lane x < 64: tag of the x-th prefill completed by the batch before
  bool pt_ok;   // pt holds them (else they are read from the ring)
};

// What a wave needs besides the state to work on one queue: the batch-time
// coefficients, the queue's prefill ring in HBM, and the wave's LDS staging area
// (3 or 4 x 64 ints, 16-byte aligned).  Rebuilt from the parameters whenever a wave picks the queue up.
struct QEnv {
  Coef k;
  bool need_C, need_A;   // d != 0, e != 0: only then are C / A accumulated
  int32_t *r_rp, *r_rd, *r_cx, *r_seq;
  int rcap;
  int* stg;
};

__device__ __forceinline__ QEnv make_env(const DevState& S, const DevParams& pr, int qid, int j,
                                         int* stage) {
  QEnv e;
  e.k = load_coef(pr, j);
  e.need_C = e.k.d != 0.0;
  e.need_A = e.k.e != 0.0;
  e.rcap = S.rcap;
  const int64_t rb = (int64_t)qid * S.rcap;
  e.r_rp = S.r_rp + rb; e.r_rd = S.r_rd + rb; e.r_cx = S.r_cx + rb; e.r_seq = S.r_seq + rb;
  e.stg = stage;
  return e;
}

template <int KS>
struct Queue {
  // decode slots (slot s = k*64 + lane); a slot is free iff dl <= g
  int dl[KS], dc[KS], ds[KS];
  // prefill-list window: lane woff + i holds entry i of the list, i < nwin
  int wrp, wrd, wcx, wseq;
  // first-token tracking (TRK paths only): tag of the window entry, and in lane
  // x < 64 the tag of the x-th prefill completed by the last batch (valid while
  // ptag_ok; a queue loaded from HBM reads them from the ring instead)
  int wtag, ptag;
  bool ptag_ok;
  int woff, nwin;
  // scalars (wave-uniform)
  int g, n_dec, n_part, n_pre, head, next_seq;
  int pend, ntrk;   // first-token tracking (TRK: copied in and out; else unused)
  int64_t c0sum, pre_sum;
  double clock;
  int64_t iters;
  template <bool TRK = false>
  __device__ void load(const DevState& S, const QEnv& e, int qid, const int32_t* tags = nullptr) {
    const int ln = lane_id();
    const QScal* q = S.sc + qid;
    g = uni(q->g); n_dec = uni(q->n_dec); n_part = uni(q->n_part); n_pre = uni(q->n_pre);
    head = uni(q->head); next_seq = uni(q->next_seq);
    if constexpr (TRK) { pend = uni(q->pend); ntrk = uni(q->ntrk); }
    else { pend = 0; ntrk = 0; }
    c0sum = uni64(q->c0sum); pre_sum = uni64(q->pre_sum);
    clock = q->clock;
    iters = uni64(q->iters);
    const int64_t db = (int64_t)qid * S.mcap;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int slot = s * kWave + ln;
      if (slot < n_dec) {
        dl[s] = S.d_last[db + slot]; dc[s] = S.d_cx0[db + slot]; ds[s] = S.d_seq[db + slot];
      } else {
        dl[s] = 0; dc[s] = 0; ds[s] = 0;
      }
    }
    woff = 0;
    nwin = 0;
    wrp = 0; wrd = 0; wcx = 0; wseq = 0;
    if constexpr (TRK) { wtag = -1; ptag = -1; ptag_ok = false; }
    refill<TRK>(e, tags);
  }

  // Copy to / from an LDS copy (same layout as the registers); TRK: the tracking
  // state too, the per-lane part in Tg.
  template <bool TRK = false>
  __device__ void to_lds(LdsQueue<KS>& L, LdsTags* Tg = nullptr) const {
    const int ln = lane_id();
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      L.dl[s * kWave + ln] = dl[s]; L.dc[s * kWave + ln] = dc[s]; L.ds[s * kWave + ln] = ds[s];
    }
    L.wrp[ln] = wrp; L.wrd[ln] = wrd; L.wcx[ln] = wcx; L.wseq[ln] = wseq;
    if constexpr (TRK) { Tg->wtag[ln] = wtag; Tg->ptag[ln] = ptag; }
    if (ln == 0) {
      L.g = g; L.n_dec = n_dec; L.n_part = n_part; L.n_pre = n_pre; L.head = head;
      L.next_seq = next_seq; L.woff = woff; L.nwin = nwin; L.c0sum = c0sum;
      if constexpr (TRK) { L.pend = pend; L.ntrk = ntrk; L.ptag_ok = ptag_ok; }
      L.pre_sum = pre_sum; L.iters = iters; L.clock = clock;
    }
    __builtin_amdgcn_wave_barrier();
  }

  template <bool TRK = false>
  __device__ void from_lds(const LdsQueue<KS>& L, const LdsTags* Tg = nullptr) {
    const int ln = lane_id();
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      dl[s] = L.dl[s * kWave + ln]; dc[s] = L.dc[s * kWave + ln]; ds[s] = L.ds[s * kWave + ln];
    }
    wrp = L.wrp[ln]; wrd = L.wrd[ln]; wcx = L.wcx[ln]; wseq = L.wseq[ln];
    if constexpr (TRK) { wtag = Tg->wtag[ln]; ptag = Tg->ptag[ln]; }
    g = uni(L.g); n_dec = uni(L.n_dec); n_part = uni(L.n_part); n_pre = uni(L.n_pre);
    head = uni(L.head); next_seq = uni(L.next_seq); woff = uni(L.woff); nwin = uni(L.nwin);
    if constexpr (TRK) { pend = uni(L.pend); ntrk = uni(L.ntrk); ptag_ok = uni(L.ptag_ok) != 0; }
    c0sum = uni64(L.c0sum); pre_sum = uni64(L.pre_sum); iters = uni64(L.iters);
    clock = L.clock;
  }

  // Write the queue back: decode slots compacted, window entries into the ring.
  template <bool TRK = false>
  __device__ void store(const DevState& S, const QEnv& e, int qid) const {
    const int ln = lane_id();
    const int64_t db = (int64_t)qid * S.mcap;
    int base = 0;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const bool live = dl[s] > g;
      const uint64_t m = ballot(live);
      if (live) {
        const int dst = base + mbcnt(m);
        S.d_last[db + dst] = dl[s]; S.d_cx0[db + dst] = dc[s]; S.d_seq[db + dst] = ds[s];
      }
      base += popc(m);
    }
    const int idx = ln - woff;
    if (idx >= 0 && idx < nwin) {
      int pos = head + idx;
      if (pos >= e.rcap) pos -= e.rcap;
      e.r_rp[pos] = wrp; e.r_rd[pos] = wrd; e.r_cx[pos] = wcx; e.r_seq[pos] = wseq;
    }
    if (ln == 0) {
      QScal* q = S.sc + qid;
      q->g = g; q->n_dec = n_dec; q->n_part = n_part; q->n_pre = n_pre; q->head = head;
      q->next_seq = next_seq; q->c0sum = c0sum; q->pre_sum = pre_sum; q->clock = clock;
      q->iters = iters;
      if constexpr (TRK) { q->pend = pend; q->ntrk = ntrk; }
    }
    // the same wave loads this queue again later in a persistent kernel
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  }

  // Move the window down to lane 0.
  template <bool TRK = false>
  __device__ void compact() {
    if (woff == 0) return;
    const int src = min(lane_id() + woff, kWave - 1);
    wrp = __shfl(wrp, src, kWave);
    wrd = __shfl(wrd, src, kWave);
    wcx = __shfl(wcx, src, kWave);
    wseq = __shfl(wseq, src, kWave);
    if constexpr (TRK) wtag = __shfl(wtag, src, kWave);
    woff = 0;
  }

  // Make min(n_pre, 64) list entries visible in the window (TRK: with their tags
  // from the queue's tag ring).
  template <bool TRK = false>
  __device__ void refill(const QEnv& e, const int32_t* tags = nullptr) {
    const int want = min(n_pre, kWave);
    if (nwin >= want) return;
    if (woff + want > kWave) compact<TRK>();
    const int idx = lane_id() - woff;
    if (idx >= nwin && idx < want) {
      int pos = head + idx;
      if (pos >= e.rcap) pos -= e.rcap;
      wrp = e.r_rp[pos]; wrd = e.r_rd[pos]; wcx = e.r_cx[pos]; wseq = e.r_seq[pos];
      if constexpr (TRK) wtag = tags[pos];
    }
    nwin = want;
  }

  __device__ int resident() const { return n_dec + n_pre; }

  // A new query at the FCFS tail gets prefill tokens in the next batch iff every
  // request of the prefill list is served in full with budget to spare and a
  // sequence slot is left for the query.
  __device__ bool tail_admitted_next(const QEnv& e) const {
    return n_dec + n_pre < e.k.M && (int64_t)n_dec + pre_sum < (int64_t)e.k.B;
  }

  // No prefill token can be scheduled in the next batch (empty prefill list, budget
  // used up by decodes, or no running partial and no free sequence slot).  Nothing
  // then changes until the next decode finishes: D, P = A = 0 stay fixed and C grows
  // by D per batch.
  __device__ bool quiet(const QEnv& e) const {
    return !(n_pre > 0 && e.k.B - n_dec > 0 && (n_part > 0 || e.k.M - n_dec - n_part > 0));
  }

  // Index of the next batch in which a decoding request finishes (INT_MAX if none).
  __device__ int next_finish() const {
    int m = 0x7fffffff;
#pragma unroll
    for (int s = 0; s < KS; ++s)
      if (dl[s] > g) m = min(m, dl[s]);
    return wave_min(m);
  }

  // Append a waiting request at the FCFS tail (the caller checked the capacity).
  // A tracked query (tags: the queue's tag ring, non-null) leaves its tag in its
  // ring slot, where it is looked up at its first token.  An untracked append
  // leaves an older tag in the slot: tags only grow between the resets that clear
  // every slot, so an older tag is below the running trace's first tag and ignored.
  __device__ void append(const QEnv& e, int p, int d, int32_t* tags = nullptr, int tag = -1) {
    const int ln = lane_id();
    const int idx = n_pre;
    int pos = head + idx;
    if (pos >= e.rcap) pos -= e.rcap;
    if (nwin == n_pre && idx < kWave) {     // the window holds the whole list: extend it
      if (woff + idx >= kWave) {
        if (tags) compact<true>(); else compact<false>();
      }
      if (ln == woff + idx) { wrp = p; wrd = d; wcx = 0; wseq = next_seq; }
      if (tags) {
        if (ln == woff + idx) wtag = tag;
        if (ln == 0) tags[pos] = tag;
        // other lanes of this wave read the tag back at the first token
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
      }
      nwin = idx + 1;
    } else {                                // beyond the window: the ring, read on refill
      if (ln == 0) {
        e.r_rp[pos] = p; e.r_rd[pos] = d; e.r_cx[pos] = 0; e.r_seq[pos] = next_seq;
        if (tags) tags[pos] = tag;
      }
      // other lanes of this wave read the entry back on refill
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    }
    n_pre += 1;
    pre_sum += p;
    next_seq += 1;
  }

  // Sum over the prefill list of rp*cx + rp*(rp+1)/2: the prefill-attention feature
  // of a batch that serves the whole list.  Entries beyond the window have not been
  // served since they were written to the ring, so the ring holds their values.
  __device__ int64_t pre_attention_all(const QEnv& e) const {
    const int ln = lane_id();
    const int idx = ln - woff;
    int64_t a = 0;
    if (idx >= 0 && idx < nwin) a = (int64_t)wrp * wcx + (int64_t)wrp * (wrp + 1) / 2;
    for (int base = nwin; base < n_pre; base += kWave) {
      const int x = base + ln;
      if (x < n_pre) {
        int pos = head + x;
        if (pos >= e.rcap) pos -= e.rcap;
        const int64_t r = e.r_rp[pos];
        a += r * e.r_cx[pos] + r * (r + 1) / 2;
      }
    }
    return wave_sum64(a);
  }

  // Build the next token batch, apply it, return its features (TRK: and keep the
  // completed prefills' count and tags for first-token tracking; tags is the queue's
  // tag ring).
  template <bool TRK = false>
  __device__ StepOut step(const QEnv& e, const int32_t* tags = nullptr) {
    const int ln = lane_id();
    const Coef& k = e.k;
    const bool need_C = e.need_C, need_A = e.need_A;
    int* stg = e.stg;
    const int B = k.B;
    const int gn = g + 1;   // index of this batch
    StepOut o;
    int nd = 0, pt_new = -1;
    if constexpr (TRK) { o.h0 = head; o.pn = pend; o.pt = ptag; o.pt_ok = ptag_ok; }
    o.D = n_dec;
    o.C = need_C ? c0sum + (int64_t)n_dec * g : 0;
    int left = B - n_dec;

    // decoding requests whose last token is in this batch leave after it
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const uint64_t fm = ballot(dl[s] == gn);
      if (fm) {
        n_dec -= popc(fm);
        if (need_C) c0sum -= sum_lanes64(dc[s], fm);
      }
    }

    // prefill chunks in FCFS order over the window (and further windows)
    int64_t P = 0, A = 0;
    int free_slots = k.M - (int)o.D - n_part;   // slots for waiting admissions
    bool more = true;
    // The usual batch: only the window's first entry can take tokens (it is the one
    // eligible entry, or it takes the whole budget).  Its chunk, and its move to a
    // decode slot when it completes, need no scan and no staging; the result is that
    // of the loop below.
    if (n_pre > 0 && left > 0 && (n_part > 0 || free_slots > 0) && nwin > 0 && n_part <= 1) {
      const int r0 = lane_read(wrp, woff);
      const int n_elig = n_part + max(0, min(free_slots, nwin - n_part));
      if (r0 >= left || n_elig == 1) {
        const int nw0 = nwin;
        const int cx0 = lane_read(wcx, woff);
        const int ch = min(r0, left);
        P += ch;
        left -= ch;
        pre_sum -= ch;
        if (need_A) A += (int64_t)ch * cx0 + (int64_t)ch * (ch + 1) / 2;
        if (ln == woff) {
          wrp -= ch;
          wcx += ch;
        }
        if (n_part == 0) free_slots -= 1;   // a waiting entry was admitted
        const bool full = ch == r0;
        if (full) {
          // completed prefill: decoding from the next batch, last = g + 1 + rd
          const int nl = gn + lane_read(wrd, woff);
          const int nc = cx0 + ch - gn;
          const int sq = lane_read(wseq, woff);
          if (need_C) c0sum += nc;
          if constexpr (TRK) {
            const int tg = lane_read(wtag, woff);
            if (ln == nd) pt_new = tg;
          }
          bool placed = false;
#pragma unroll
          for (int s = 0; s < KS; ++s) {
            const uint64_t fm = ballot(dl[s] <= gn);
            if (!placed && fm) {
              if (ln == __builtin_ctzll(fm)) { dl[s] = nl; dc[s] = nc; ds[s] = sq; }
              placed = true;
            }
          }
          n_dec += 1;
          if constexpr (TRK) nd += 1;
          woff += 1;
          nwin -= 1;
          head += 1;
          if (head >= e.rcap) head -= e.rcap;
          n_pre -= 1;
          if (n_part == 1) n_part = 0;
        } else if (n_part == 0) {
          n_part = 1;   // the waiting entry got a chunk and stays partial
        }
        // the loop below goes on only when the whole window was served
        more = full && nw0 == 1;
        if (more) refill<TRK>(e, tags);
      }
    }
    while (more && n_pre > 0 && left > 0 && (n_part > 0 || free_slots > 0)) {
      if (nwin == 0) refill<TRK>(e, tags);
      const int nw0 = nwin;
      const int idx = ln - woff;
      const bool valid = idx >= 0 && idx < nw0;
      const bool part = idx < n_part;
      const bool elig = valid && (part || (idx - n_part) < free_slots);
      const int x = elig ? min(wrp, B) : 0;
      const int incl = scan_sat(x, B);
      const int excl = prev_lane(incl);
      const int ch = min(incl, left) - min(excl, left);
      const int served = min(uni(lane_last(incl)), left);
      P += served;
      left -= served;
      pre_sum -= served;
      const uint64_t chm = ballot(ch > 0);
      const uint64_t fullm = ballot(ch > 0 && ch == wrp);
      const int n_full = popc(fullm);
      const int n_adm_w = popc(chm & ~ballot(part));
      // the first entry not served in full was waiting and got a chunk
      const bool part_waiting = n_full < nw0 && n_full >= n_part &&
                                ((chm >> (woff + n_full)) & 1ull) != 0;
      if (need_A && chm) {
        const int64_t av = (int64_t)ch * wcx + (int64_t)ch * (ch + 1) / 2;
        A += sum_lanes64(av, chm);
      }
      if (ch > 0) {
        wrp -= ch;
        wcx += ch;
      }
      free_slots -= n_adm_w;
      if (n_full > 0) {
        // completed prefills start decoding next batch: last = g + 1 + rd
        const int nl = gn + wrd;
        const int nc = wcx - gn;
        if (need_C) c0sum += sum_lanes64(nc, fullm);
        const bool full = ((fullm >> ln) & 1ull) != 0;
        if (full) {
          stg[idx] = nl; stg[kWave + idx] = nc; stg[2 * kWave + idx] = wseq;
          if constexpr (TRK) stg[3 * kWave + idx] = wtag;
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        if constexpr (TRK) {   // lanes nd .. nd + n_full - 1 (below 64) take their tags
          const int x = ln - nd;
          if (x >= 0 && x < n_full) pt_new = stg[3 * kWave + x];
        }
        int placed = 0;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          if (placed < n_full) {
            const bool fr = dl[s] <= gn;
            const uint64_t fm = ballot(fr);
            const int r = placed + mbcnt(fm);
            if (fr && r < n_full) { dl[s] = stg[r]; dc[s] = stg[kWave + r]; ds[s] = stg[2 * kWave + r]; }
            placed += popc(fm);
          }
        }
        __builtin_amdgcn_wave_barrier();
        n_dec += n_full;
        if constexpr (TRK) nd += n_full;
        woff += n_full;
        nwin -= n_full;
        head += n_full;
        if (head >= e.rcap) head -= e.rcap;
        n_pre -= n_full;
      }
      n_part = n_part - min(n_full, n_part) + (part_waiting ? 1 : 0);
      // continue only if the whole window was served (more entries may wait in the ring)
      if (n_full < nw0) break;
      refill<TRK>(e, tags);
    }
    if (nwin < n_pre && nwin < kWave / 2) refill<TRK>(e, tags);
    o.P = (int)P;
    o.A = need_A ? A : 0;
    if constexpr (TRK) { o.nd = nd; pend = nd; ptag = pt_new; ptag_ok = true; }
    g = gn;
    return o;
  }

  // Realised TTFT of the tracked queries whose first token came in the batch just
  // stepped (o, from step<true>), which ended at clk: the batch completing their prefill (reading 1)
  // or the next one, their first decode (reading 0).  Those entries have left the
  // prefill list (the ring slots just before the head), but their slots still hold
  // their tags: appends fill the slots after the list, and the completed entries
  // (running, so at most M minus the running partials) plus the list (at most qcap
  // waiting entries plus the running partials) never exceed the ring's qcap + mcap
  // slots.  Tags tag0 .. tag0 + N - 1 are the queries of the running trace;
  // out[i] = clk, the first-token time (the arrival is subtracted after the trace).
  __device__ void realize(const QEnv& e, const int32_t* tags, const StepOut& o, int reading,
                          double clk, double* out, int tag0, int N) {
    const int n = reading == 1 ? o.nd : o.pn;
    if (n == 0) return;
    const int ln = lane_id();
    int hit = 0;
    // the first 64 tags from registers (captured by step), the rest from the ring
    const bool regs = reading == 1 || o.pt_ok;
    if (regs && ln < n) {
      const int tag = reading == 1 ? ptag : o.pt;
      const int q = tag - tag0;
      if (tag >= 0 && q >= 0 && q < N) {
        out[q] = clk;
        ++hit;
      }
    }
    int lo = reading == 1 ? o.h0 : o.h0 - o.pn;
    if (lo < 0) lo += e.rcap;
    for (int x = regs ? kWave + ln : ln; x < n; x += kWave) {
      int pos = lo + x;
      if (pos >= e.rcap) pos -= e.rcap;
      const int tag = tags[pos];
      const int q = tag - tag0;
      if (tag >= 0 && q >= 0 && q < N) {
        out[q] = clk;
        ++hit;
      }
    }
    ntrk -= wave_sum32(hit);
  }

  // The decode-only batches that follow the admission batch of a tail query, read
  // from the current state without changing it.  Valid when tail_admitted_next()
  // holds and the whole prefill list is in the window: the admission batch serves
  // every list entry in full (entry e then decodes until batch g + 1 + rd_e) and
  // keeps the decoding requests with last > g + 1.  Batch k after it (k >= 1) has
  //   D_k = #{dl >= g + 1 + k} + #{list entries: rd >= k},
  //   C_k = (sum of cx0 over those) + D_k * (g + k).
  // tail_begin() sets up k = 1; tail_next() moves to k + 1.
  struct Tail {
    int k;
    int64_t D, c0;   // count and cx0 sum of the requests alive in batch k
  };

  __device__ Tail tail_begin(const QEnv& e) const {
    const bool need_C = e.need_C;
    const int ln = lane_id();
    Tail t;
    t.k = 1;
    // decoding requests surviving the admission batch, plus every list entry
    // (all have rd >= 1); the cx0 sum is c0sum minus the leavers plus the entries
    int64_t D = 0, c0 = c0sum;
    const int gn = g + 1;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      D += popc(ballot(dl[s] > gn));
      if (need_C) {
        const uint64_t fm = ballot(dl[s] == gn);
        if (fm) c0 -= sum_lanes64(dc[s], fm);
      }
    }
    const int idx = ln - woff;
    const bool ent = idx >= 0 && idx < nwin;
    const uint64_t em = ballot(ent);
    D += popc(em);
    if (need_C) c0 += sum_lanes64((int64_t)(wcx + wrp) - gn, em);
    t.D = D;
    t.c0 = c0;
    return t;
  }

  __device__ void tail_next(const QEnv& e, Tail& t) const {
    const bool need_C = e.need_C;
    const int ln = lane_id();
    // requests whose last decode is batch k leave: old slots with dl == g + 1 + k,
    // list entries with rd == k
    const int due = g + 1 + t.k;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const uint64_t m = ballot(dl[s] == due);
      if (m) {
        t.D -= popc(m);
        if (need_C) t.c0 -= sum_lanes64(dc[s], m);
      }
    }
    const int idx = ln - woff;
    const bool ent = idx >= 0 && idx < nwin;
    const uint64_t em = ballot(ent && wrd == t.k);
    if (em) {
      t.D -= popc(em);
      if (need_C) t.c0 -= sum_lanes64((int64_t)(wcx + wrp) - (g + 1), em);
    }
    t.k += 1;
  }

  // Fold the quiet batches that precede the next decode finish into clk (one add
  // per batch, in batch order), stopping early once clk >= t_stop or n reaches
  // max_iters.  Call only when quiet(e) holds; returns the batches folded.
  __device__ int64_t quiet_run(const QEnv& e, double& clk, double t_stop, int64_t n,
                               int64_t max_iters) {
    const int nf = next_finish();
    const int D = n_dec;
    int64_t done = 0;
    if (!e.need_C) {
      const double T = batch_time(e.k, 0, D, 0, 0);
      while (g + 1 < nf && clk < t_stop && n + done < max_iters) {
        clk = __dadd_rn(clk, T);
        ++g;
        ++done;
      }
    } else {
      int64_t C = c0sum + (int64_t)D * g;
      while (g + 1 < nf && clk < t_stop && n + done < max_iters) {
        clk = __dadd_rn(clk, batch_time(e.k, 0, D, C, 0));
        C += D;
        ++g;
        ++done;
      }
    }
    // (a tracked replay folds quiet batches only with pend == 0, which they keep)
    return done;
  }
};

}  // namespace lar
