// sfs_device.h -- device-side layout and the wave-level SFS batch engine (gfx950).
//
// One wavefront owns one (scenario, instance) queue.  Its running requests live in
// VGPRs, slot s = k*64 + lane (k < KS), compacted in FCFS order; the waiting
// requests stay in an HBM ring that is only read, a window of 64 at a time.  One
// token batch (Sec. 4.1: one decode token per decoding sequence, then prefill
// chunks in arrival order under the token budget and the running-sequence cap)
// costs a few ballots, saturating wave prefix sums and, when requests finish or
// are admitted, one order-preserving compaction through LDS.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lar {

constexpr int kWave = 64;

// Error codes shared with the C ABI (lar.h); kept numerically identical.
constexpr int kErrArg = -1, kErrState = -2, kErrCapacity = -3, kErrIter = -4;

struct DevState {
  int32_t *run_rp, *run_rd, *run_cx;  // [ZI][mcap] running requests, FCFS, compacted
  int32_t *wait_p, *wait_rd;          // [ZI][qcap] ring of waiting requests (FCFS)
  int32_t *n_run, *w_head, *n_wait;   // [ZI]
  double *clock;                      // [ZI] instance clock, ms
  int64_t *iters;                     // [ZI] batches replayed since the load
  int32_t mcap, qcap;
};

struct DevParams {
  const double *a, *b, *c, *d, *e;    // [I]
  const int32_t *B, *M, *col;         // [I]
};

// Background trajectory of one queue up to the batch in which a new tail query
// would first receive prefill tokens (its admission batch), plus the decode-only
// batches that follow it.  Written by k_traj, read by k_est.
struct DevTraj {
  double *E;            // [ZI] clock folded over the batches before the admission batch
  int32_t *pre;         // [ZI] number of those batches
  int64_t *P, *D, *C, *A;  // [ZI] background features of the admission batch
  int32_t *left;        // [ZI] budget the background leaves in that batch (>= 1)
  int32_t *ok;          // [ZI] 1 = valid; 0 = iteration cap or clock behind t
  int32_t *tailD;       // [K][ZI] decode tokens of the k-th batch after admission
  int64_t *tailC;       // [K][ZI] their context sum
  int32_t K;
};

struct Coef {
  double a, b, c, d, e;
  int B, M;
};

struct Feat {
  int64_t P, D, C, A;
};

__device__ __forceinline__ Coef load_coef(const DevParams& pr, int j) {
  Coef k;
  k.a = pr.a[j]; k.b = pr.b[j]; k.c = pr.c[j]; k.d = pr.d[j]; k.e = pr.e[j];
  k.B = pr.B[j]; k.M = pr.M[j];
  return k;
}

// Batch time (Sec. 4.1): ((((a + b*P) + c*D) + d*C) + e*A), one rounding per op.
__device__ __forceinline__ double batch_time(const Coef& k, int64_t P, int64_t D, int64_t C,
                                             int64_t A) {
  double t = k.a;
  t = __dadd_rn(t, __dmul_rn(k.b, (double)P));
  t = __dadd_rn(t, __dmul_rn(k.c, (double)D));
  t = __dadd_rn(t, __dmul_rn(k.d, (double)C));
  t = __dadd_rn(t, __dmul_rn(k.e, (double)A));
  return t;
}

__device__ __forceinline__ void set_error(int32_t* err, int code) {
  atomicCAS(err, 0, code);
}

// ------------------------------------------------------------------ wave primitives
__device__ __forceinline__ int lane_id() { return (int)__lane_id(); }
__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ int popc(uint64_t m) { return __popcll(m); }
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ int lane_last(int x) { return __builtin_amdgcn_readlane(x, kWave - 1); }

// Inclusive prefix sum over the wave, saturating at cap.  Inputs in [0, cap] with
// cap <= 2^30, so no intermediate overflows; min(sat(x), L) == min(x, L) for L <= cap.
__device__ __forceinline__ int scan_sat(int x, int cap) {
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    int y = __shfl_up(x, o, kWave);
    if (lane_id() >= o) x = min(x + y, cap);
  }
  return x;
}

__device__ __forceinline__ int64_t shfl_xor64(int64_t x, int m) {
  int lo = (int)(uint32_t)(uint64_t)x;
  int hi = (int)(uint32_t)((uint64_t)x >> 32);
  lo = __shfl_xor(lo, m, kWave);
  hi = __shfl_xor(hi, m, kWave);
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint64_t)(uint32_t)lo);
}

__device__ __forceinline__ int64_t uni64(int64_t x) {
  int lo = uni((int)(uint32_t)(uint64_t)x);
  int hi = uni((int)(uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint64_t)(uint32_t)lo);
}

__device__ __forceinline__ int64_t wave_sum64(int64_t x) {
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) x += shfl_xor64(x, o);
  return uni64(x);
}

__device__ __forceinline__ int wave_sum32(int x) {
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) x += __shfl_xor(x, o, kWave);
  return uni(x);
}

// ------------------------------------------------------------------ the batch engine
struct StepInfo {
  Feat f;
  int left;      // budget left after the batch
  int n_adm;     // waiting requests admitted in the batch
  int n_wait0;   // waiting requests before the batch
  int n_run0;    // running requests before the batch
};

template <int KS>
struct WaveQueue {
  int rp[KS], rd[KS], cx[KS];  // slot s = k*64 + lane
  int n_run, head, n_wait;     // wave-uniform
  int qcap;
  const int32_t* wp;           // waiting ring of this queue
  const int32_t* wr;
  int* l_rp;                   // LDS staging, KS*64 ints each
  int* l_rd;
  int* l_cx;
  Coef k;
  bool need_C, need_A;         // d != 0, e != 0: only then are C / A needed

  __device__ void load(const DevState& S, int qid) {
    const int ln = lane_id();
    n_run = uni(S.n_run[qid]);
    head = uni(S.w_head[qid]);
    n_wait = uni(S.n_wait[qid]);
    qcap = S.qcap;
    wp = S.wait_p + (int64_t)qid * S.qcap;
    wr = S.wait_rd + (int64_t)qid * S.qcap;
    const int64_t base = (int64_t)qid * S.mcap;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int slot = s * kWave + ln;
      if (slot < n_run) {
        rp[s] = S.run_rp[base + slot];
        rd[s] = S.run_rd[base + slot];
        cx[s] = S.run_cx[base + slot];
      } else {
        rp[s] = 0; rd[s] = 0; cx[s] = 0;
      }
    }
  }

  __device__ void store(const DevState& S, int qid) const {
    const int ln = lane_id();
    const int64_t base = (int64_t)qid * S.mcap;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int slot = s * kWave + ln;
      if (slot < S.mcap) {
        S.run_rp[base + slot] = rp[s];
        S.run_rd[base + slot] = rd[s];
        S.run_cx[base + slot] = cx[s];
      }
    }
    if (ln == 0) {
      S.n_run[qid] = n_run;
      S.w_head[qid] = head;
      S.n_wait[qid] = n_wait;
    }
  }

  __device__ int resident() const { return n_run + n_wait; }

  // Build the next token batch, apply it, and return its features.
  __device__ StepInfo step() {
    const int ln = lane_id();
    const int B = k.B;
    StepInfo info;
    info.n_wait0 = n_wait;
    info.n_run0 = n_run;

    // 1. one decode token for every running request whose prefill is complete
    bool valid[KS], dec[KS];
    int D = 0;
    int64_t c_lane = 0;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      valid[s] = (s * kWave + ln) < n_run;
      dec[s] = valid[s] && rp[s] == 0;
      D += popc(ballot(dec[s]));
      if (dec[s]) c_lane += cx[s];
    }
    int left = B - D;

    // 2a. prefill chunks for running requests with prefill left, in slot (FCFS) order
    int chunk[KS];
    int64_t p_lane = 0, a_lane = 0;
    uint64_t any_part = 0;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      chunk[s] = 0;
      any_part |= ballot(valid[s] && rp[s] > 0);
    }
    if (any_part) {
      int carry = 0;   // saturating prefix of the earlier passes
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const int x = (valid[s] && rp[s] > 0) ? min(rp[s], B) : 0;
        int incl = scan_sat(x, B);
        int excl = __shfl_up(incl, 1, kWave);
        if (ln == 0) excl = 0;
        incl = min(incl + carry, B);
        excl = min(excl + carry, B);
        chunk[s] = min(incl, left) - min(excl, left);
        carry = uni(lane_last(incl));
      }
      left -= min(carry, left);
    }

    // apply decode tokens and running chunks; find the requests that stay
    bool keep[KS];
    int n_keep = 0;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int ch = chunk[s];
      if (ch > 0) {
        p_lane += ch;
        a_lane += (int64_t)ch * cx[s] + (int64_t)ch * (ch + 1) / 2;
        cx[s] += ch;
        rp[s] -= ch;
      }
      if (dec[s]) {
        cx[s] += 1;
        rd[s] -= 1;
      }
      keep[s] = valid[s] && rd[s] > 0;
      n_keep += popc(ballot(keep[s]));
    }

    // 2b. admit waiting requests in FCFS order while budget and sequence slots last
    int n_adm = 0;
    const bool admit = left > 0 && n_run < k.M && n_wait > 0;
    const bool relayout = admit || n_keep != n_run;
    if (relayout) {
      // order-preserving compaction of the running slots into LDS
      int before = 0;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const uint64_t m = ballot(keep[s]);
        if (keep[s]) {
          const int dst = before + (int)__builtin_amdgcn_mbcnt_hi(
              (uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
          l_rp[dst] = rp[s];
          l_rd[dst] = rd[s];
          l_cx[dst] = cx[s];
        }
        before += popc(m);
      }
    }
    if (admit) {
      const int lim = min(n_wait, k.M - n_run);
      for (;;) {
        const int w = n_adm + ln;
        const bool v = w < lim;
        int p = 0, r = 0;
        if (v) {
          int pos = head + w;
          if (pos >= qcap) pos -= qcap;
          p = wp[pos];
          r = wr[pos];
        }
        const int x = v ? min(p, B) : 0;
        const int incl = scan_sat(x, B);
        int excl = __shfl_up(incl, 1, kWave);
        if (ln == 0) excl = 0;
        const int ch = min(incl, left) - min(excl, left);
        const uint64_t am = ballot(ch > 0);
        if (ch > 0) {
          const int dst = n_keep + n_adm + ln;
          l_rp[dst] = p - ch;
          l_rd[dst] = r;
          l_cx[dst] = ch;
          p_lane += ch;
          a_lane += (int64_t)ch * (ch + 1) / 2;
        }
        const int na = popc(am);
        left -= min(uni(lane_last(incl)), left);
        n_adm += na;
        if (na < kWave || left == 0 || n_adm >= lim) break;
      }
      head += n_adm;
      if (head >= qcap) head -= qcap;
      n_wait -= n_adm;
    }
    if (relayout) {
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      n_run = n_keep + n_adm;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const int slot = s * kWave + ln;
        if (slot < n_run) {
          rp[s] = l_rp[slot];
          rd[s] = l_rd[slot];
          cx[s] = l_cx[slot];
        } else {
          rp[s] = 0; rd[s] = 0; cx[s] = 0;
        }
      }
      __builtin_amdgcn_wave_barrier();
    }

    info.f.P = wave_sum64(p_lane);
    info.f.D = D;
    info.f.C = need_C ? wave_sum64(c_lane) : 0;
    info.f.A = need_A ? wave_sum64(a_lane) : 0;
    info.left = left;
    info.n_adm = n_adm;
    return info;
  }
};

}  // namespace lar
