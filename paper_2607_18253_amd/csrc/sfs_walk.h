// sfs_walk.h -- the background trajectory of one queue (Sec. 4.1) for the batched
// what-if estimate, walked without changing the queue's state.
//
// The batch engine of sfs_device.h keeps every decoding request in a register slot
// so that a trace can write the queue back.  The trajectory only reads the state, and
// of the decoding requests a batch only needs how many there are, how many leave
// after it and (when d != 0) the sums of their context offsets.  So here they are
// counts per batch index of their last token:
//   * a ring of kWalkBins bins in LDS, bin (last mod kWalkBins), for requests whose
//     last token is at most kWalkNear batches ahead of the batch that created them;
//   * the 64 bins of the current batch window [hb, hb + 64) in one register (lane x
//     = batch hb + x), updated in place; the ring holds zeros there;
//   * requests further ahead in a short list in LDS (far list).
// The prefill list is read in FCFS order from the queue's ring with scalar loads;
// its head entry, the only one that can be partially served, is kept in scalars.
// Every batch is then a few scalar operations per served entry.
//
// Batch composition, times and the stopping rule are those of Queue::step and
// Queue::quiet_run, operation for operation (same roundings, same order), so the
// trajectory's clock, features and decode tail are bit-identical to the engine's.
// walk_traj returns false, before writing anything, when the queue is outside what
// this walk covers (more than one partially served request, more far requests than
// the far list holds, or context sums without their bins); the caller then runs the
// engine.
#pragma once

#include "sfs_device.h"

namespace lar {

constexpr int kWalkBins = 2048;                 // ring of per-batch counts (power of two)
constexpr int kWalkNear = kWalkBins - kWave;    // farthest last-token offset kept in the ring
constexpr int kWalkFar = 256;                   // far list capacity

template <bool NC>
struct WalkLds {
  int cnt[kWalkBins];                  // decoding requests per last-token batch
  int64_t c0[NC ? kWalkBins : 1];      // NC: sum of their context offsets
  int flast[kWalkFar], fc0[kWalkFar];  // far list: last-token batch, context offset
};

// Orders this wave's earlier LDS accesses (any lane) before its later ones.
__device__ __forceinline__ void walk_lds_sync() {
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ int64_t lane_read64(int64_t v, int l) {
  const int lo = __builtin_amdgcn_readlane((int)(uint32_t)(uint64_t)v, l);
  const int hi = __builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), l);
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint64_t)(uint32_t)lo);
}

// One lane's add to an LDS word (32 or 64 bits), issued as a single ds_add: the
// compiler's atomic lowering would first count the active lanes, and here exactly one
// lane is active.  A wave's LDS operations complete in order, so a later read by any
// lane sees the sum; the memory clobber keeps the compiler from moving LDS accesses
// across it.
__device__ __forceinline__ void lds_add_one(int* p, int v) {
  const uint32_t a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) int*)p;
  asm volatile("ds_add_u32 %0, %1" : : "v"(a), "v"(v) : "memory");
}
__device__ __forceinline__ void lds_add_one(int64_t* p, int64_t v) {
  const uint32_t a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) int64_t*)p;
  asm volatile("ds_add_u64 %0, %1" : : "v"(a), "v"(v) : "memory");
}

// Wave-uniform read of a ring field.  Nothing writes the rings while a trajectory is
// walked, so the read may go through the scalar cache (constant address space).
typedef const __attribute__((address_space(4))) int32_t walk_cint;
__device__ __forceinline__ int ring_s(const int32_t* base, int pos) {
  const uint32_t off = (uint32_t)pos * 4u;   // pos < rcap: a 32-bit byte offset
  return *(walk_cint*)((const char*)base + off);
}

// Decoding requests of one queue as per-batch counts (see the top of this file).
// NCL: the LDS has context-sum bins; QC: this queue keeps context sums (d != 0).
template <bool NCL, bool QC>
struct WalkBins {
  WalkLds<NCL>& L;
  int hb;          // batch of lane 0 of the register window (multiple of 64)
  int hv;          // lane x: requests whose last token is batch hb + x
  int64_t hvc;     // QC: their context-offset sum
  int n_far, far_next;

  // Record a request whose last token is batch nl, context offset nc; near: nl is at
  // most kWalkNear batches after the batch that creates it.  Far requests go to the
  // far list (counted past its capacity, which makes the walk give up); far_next
  // takes them in at far_update(), which must come before batch nl - kWalkNear.
  __device__ __forceinline__ void place(int nl, int nc, int near) {
    const int ln = lane_id();
    const int x = nl - hb;
    // in the window: that lane's bin (no lane matches a bin past the window)
    hv += ln == x ? 1 : 0;
    if constexpr (QC) hvc += ln == x ? (int64_t)nc : 0;
    if (__builtin_expect(!near, 0)) {   // far: the list
      if (ln == 0 && n_far < kWalkFar) { L.flast[n_far] = nl; L.fc0[n_far] = nc; }
      n_far += 1;
    } else if (ln == 0 && x >= kWave) {   // past the window: the ring bin
      lds_add_one(&L.cnt[nl & (kWalkBins - 1)], 1);
      if constexpr (QC) lds_add_one(&L.c0[nl & (kWalkBins - 1)], (int64_t)nc);
    }
  }

  // Take far list entries from .. n_far - 1 into far_next.
  __device__ void far_update(int from) {
    walk_lds_sync();
    int m = 0x7fffffff;
    for (int base = from; base < n_far; base += kWave) {
      const int x = base + lane_id();
      m = min(m, wave_min(x < n_far ? L.flast[x] : 0x7fffffff));
    }
    far_next = min(far_next, m);
  }

  // Move the register window to the 64 bins starting at batch nb (a multiple of 64).
  // The bins passed over hold no requests; the ring keeps zeros under the window.
  __device__ void roll(int nb) {
    walk_lds_sync();
    const int x = (nb + lane_id()) & (kWalkBins - 1);
    hb = nb;
    hv = L.cnt[x];
    L.cnt[x] = 0;
    if constexpr (QC) {
      hvc = L.c0[x];
      L.c0[x] = 0;
    }
  }

  // Far requests whose last token is batch b: add their count and offsets to fin,
  // finc, and find the next far last-token batch after b.
  __device__ void far_finish(int b, int& fin, int64_t& finc) {
    walk_lds_sync();
    int nxt = 0x7fffffff;
    for (int base = 0; base < n_far; base += kWave) {
      const int x = base + lane_id();
      int l = 0, c = 0;
      if (x < n_far) { l = L.flast[x]; c = L.fc0[x]; }
      const uint64_t m = ballot(x < n_far && l == b);
      if (m) {
        fin += popc(m);
        if constexpr (QC) finc += sum_lanes64(c, m);
      }
      nxt = min(nxt, wave_min(x < n_far && l > b ? l : 0x7fffffff));
    }
    far_next = nxt;
  }

  // First batch after g in which a decoding request finishes (INT_MAX if none).
  __device__ int next_finish(int g) {
    int nf = 0x7fffffff;
    const int ln = lane_id();
    const uint64_t m = ballot(hv != 0 && hb + ln > g);
    if (m) {
      nf = hb + __builtin_ctzll(m);
    } else {
      walk_lds_sync();
      for (int b = hb + kWave; b <= g + kWalkNear; b += kWave) {
        const int v = L.cnt[(b + ln) & (kWalkBins - 1)];
        const uint64_t m2 = ballot(v != 0 && b + ln > g);
        if (m2) {
          nf = b + __builtin_ctzll(m2);
          break;
        }
      }
    }
    return min(nf, far_next);
  }
};

// The trajectory of k_traj for queue qid: clock and features of the batches up to
// the admission batch of a new FCFS-tail query, then the decode tail (K batches).
// QC, QA: the queue's d and e are non-zero (context sums and prefill attention are
// accumulated); NCL: the LDS has context-sum bins (needed for QC).
template <int KS, bool NCL, bool QC, bool QA>
__device__ bool walk_traj(const DevState& S, const QEnv& e, int qid, const DevTraj& tr, int ZI,
                          double t, int64_t max_iters, int32_t* err, WalkLds<NCL>& lds) {
  static_assert(NCL || !QC, "context sums need their bins");
  const int ln = lane_id();
  const Coef& k = e.k;
  constexpr bool need_C = QC;
  constexpr bool need_A = QA;
  const QScal* q = S.sc + qid;
  int g = uni(q->g);
  int n_dec = uni(q->n_dec);
  int n_part = uni(q->n_part);
  int n_pre = uni(q->n_pre);
  const int head = uni(q->head);
  int64_t c0sum = uni64(q->c0sum);
  int64_t pre_sum = uni64(q->pre_sum);
  if (n_part > 1 || n_dec > KS * kWave) return false;
  // batches are counted in 32 bits; a cap beyond that leaves the rare longer
  // trajectory to the engine
  const int cap = max_iters < 0x7fffffff ? (int)max_iters : 0x7fffffff;

  // decoding requests into the bins (or the far list)
  WalkBins<NCL, QC> w{lds, 0, 0, 0, 0, 0x7fffffff};
  for (int x = ln; x < kWalkBins; x += kWave) {
    lds.cnt[x] = 0;
    if constexpr (QC) lds.c0[x] = 0;
  }
  walk_lds_sync();
  const int64_t db = (int64_t)qid * S.mcap;
  for (int base = 0; base < n_dec; base += kWave) {
    const int slot = base + ln;
    const bool v = slot < n_dec;
    int dl = 0, dc = 0;
    if (v) {
      dl = S.d_last[db + slot];
      if (need_C) dc = S.d_cx0[db + slot];
    }
    const bool far = v && dl - g > kWalkNear;
    const uint64_t fm = ballot(far);
    if (v && !far) {
      atomicAdd(&lds.cnt[dl & (kWalkBins - 1)], 1);
      if constexpr (QC)
        atomicAdd((unsigned long long*)&lds.c0[dl & (kWalkBins - 1)],
                  (unsigned long long)(int64_t)dc);
    }
    if (fm) {
      const int nf = popc(fm);
      if (w.n_far + nf > kWalkFar) return false;
      if (far) {
        const int x = w.n_far + mbcnt(fm);
        lds.flast[x] = dl;
        lds.fc0[x] = dc;
      }
      w.n_far += nf;
      w.far_next = min(w.far_next, wave_min(far ? dl : 0x7fffffff));
    }
  }
  w.roll((g + 1) & ~(kWave - 1));

  // the prefill list: head entry (list index li, ring slot pos) as it stands
  const int rcap = e.rcap;
  const int n_list = n_pre;
  int pos = head;
  int h_rp = 0, h_rd = 0, h_cx = 0;
  if (n_pre > 0) {
    h_rp = ring_s(e.r_rp, pos);
    h_rd = ring_s(e.r_rd, pos);
    h_cx = ring_s(e.r_cx, pos);
  }

  double E = q->clock;
  int ok = 1;
  if (E < t) {
    ok = 0;
    if (ln == 0) set_error(err, kErrState);
  }
  int pre = 0;
  const int B = k.B, M = k.M;
  int far_seen = w.n_far;
  // Outer loop: the events the batch loop below leaves to it (the admission point,
  // the cap, quiet stretches, a batch that needs the window moved or far requests).
  // Flags that live across blocks are ints, not bools, so that they stay scalar.
  while (ok) {
    if (w.n_far != far_seen) {   // far requests placed by the batch loop
      if (w.n_far > kWalkFar) return false;
      w.far_update(far_seen);
      far_seen = w.n_far;
    }
    // a new tail query would get prefill tokens in the next batch (pre_sum >= 0)
    if (n_dec + n_pre < M && (uint32_t)((uint64_t)pre_sum >> 32) == 0u &&
        (uint32_t)pre_sum < (uint32_t)(B - n_dec))
      break;
    if (pre >= cap) {   // the admission batch would exceed the cap
      ok = 0;
      break;
    }
    if (!(n_pre > 0 && n_dec < B && (n_part > 0 || n_dec + n_part < M))) {
      // no prefill token until the next decode finish: D, P = A = 0 stay fixed, C
      // grows by D per batch (the batches Queue::quiet_run folds; it also stops at a
      // clock of +inf, after which the engine steps the same batches one by one)
      const int nf = w.next_finish(g);
      const int n = min(nf - 1 - g, cap - pre);
      if (n > 0) {
        if (!need_C) {
          const double T = batch_time(k, 0, n_dec, 0, 0);
          for (int i = 0; i < n; ++i) E = __dadd_rn(E, T);
        } else {
          int64_t C = c0sum + (int64_t)n_dec * g;
          for (int i = 0; i < n; ++i) {
            E = __dadd_rn(E, batch_time(k, 0, n_dec, C, 0));
            C += n_dec;
          }
        }
        g += n;
        pre += n;
      }
      if (pre >= cap) {
        ok = 0;
        break;
      }
    }
    // the next batch: its window and far requests
    if (g + 1 - w.hb >= kWave) w.roll((g + 1) & ~(kWave - 1));
    int fin = lane_read(w.hv, g + 1 - w.hb);
    int64_t finc = 0;
    if constexpr (QC) finc = lane_read64(w.hvc, g + 1 - w.hb);
    if (g + 1 == w.far_next) w.far_finish(g + 1, fin, finc);
    // Batch loop: batches g + 1, g + 2, ... while the window holds them, no far
    // request finishes, the cap is not reached and a prefill token can be scheduled.
    // The batch loop keeps the list's remaining prefill in 32 bits; a list holding
    // 2^31 tokens or more leaves after one batch, back to the 64-bit count here.
    const int g0 = g, pre0 = pre;
    const int big = (uint64_t)pre_sum > 0x7fffffffull ? 1 : 0;
    const int ps0 = big ? 0x7fffffff : (int)pre_sum;
    int ps = ps0;
    const int g_stop = uni(big ? g0 + 1
                               : min(min(w.hb + kWave - 1, w.far_next - 1),
                                     g0 + min(cap - pre0, 0x7fffffff - g0)));
    for (;;) {
      const int gn = g + 1;
      const int D = n_dec;
      const int64_t C = need_C ? c0sum + (int64_t)D * g : 0;
      n_dec -= fin;
      if (need_C) c0sum -= finc;
      int left = B - D;
      int free_slots = M - D - n_part;   // slots for waiting admissions
      int P = 0;
      int64_t A = 0;
      // prefill chunks in FCFS order: the partial, then waiting entries while slots
      // and budget last
      if (n_part > 0 && left > 0) {
        const int ch = min(h_rp, left);
        P = ch;
        left -= ch;
        if (need_A) A += (int64_t)ch * h_cx + (int64_t)ch * (ch + 1) / 2;
        if (ch < h_rp) {   // still partial: takes the whole budget
          h_rp -= ch;
          h_cx += ch;
        } else {           // completed: decoding from the next batch until gn + rd
          const int nc = h_cx + ch - gn;
          w.place(gn + h_rd, nc, h_rd <= kWalkNear);
          n_dec += 1;
          if (need_C) c0sum += nc;
          n_part = 0;
          n_pre -= 1;
          // entries after the head are waiting: context 0 (past the list's end the
          // slot holds an unused value)
          pos = pos + 1 == rcap ? 0 : pos + 1;
          h_rp = ring_s(e.r_rp, pos);
          h_rd = ring_s(e.r_rd, pos);
          h_cx = 0;
        }
      }
      if (n_part == 0) {
        // waiting entries that may be admitted (one slot each): those whose whole
        // prompt fits the budget left complete here ...
        int adm = min(n_pre, free_slots);
        while (adm > 0 && h_rp <= left) {
          const int ch = h_rp;
          P += ch;
          left -= ch;
          if (need_A) A += (int64_t)ch * (ch + 1) / 2;
          const int nc = ch - gn;
          w.place(gn + h_rd, nc, h_rd <= kWalkNear);
          n_dec += 1;
          if (need_C) c0sum += nc;
          n_pre -= 1;
          adm -= 1;
          // the next entry (past the list's end the slot holds an unused value)
          pos = pos + 1 == rcap ? 0 : pos + 1;
          h_rp = ring_s(e.r_rp, pos);
          h_rd = ring_s(e.r_rd, pos);
        }
        // ... and the next one, if admitted, takes the rest of the budget in part
        if (adm > 0 && left > 0) {
          const int ch = left;
          P += ch;
          left = 0;
          if (need_A) A += (int64_t)ch * (ch + 1) / 2;
          h_rp -= ch;
          h_cx = ch;
          n_part = 1;
        }
      }
      ps -= P;
      g = gn;
      E = __dadd_rn(E, batch_time(k, P, D, C, A));
      if (g >= g_stop) break;
      if (n_dec + n_pre < M && ps < B - n_dec) break;
      if (!(n_pre > 0 && n_dec < B && (n_part > 0 || n_dec + n_part < M))) {
        // quiet until the next decode finish: folded here when that finish is in
        // the window and before the stop (else the outer loop folds)
        const uint64_t m = ballot(w.hv != 0 && w.hb + ln > g);
        const int nf = m ? w.hb + __builtin_ctzll(m) : 0x7fffffff;
        if (nf > g_stop) break;
        const int n = nf - 1 - g;
        if constexpr (!QC) {
          const double T = batch_time(k, 0, n_dec, 0, 0);
          for (int i = 0; i < n; ++i) E = __dadd_rn(E, T);
        } else {
          int64_t C2 = c0sum + (int64_t)n_dec * g;
          for (int i = 0; i < n; ++i) {
            E = __dadd_rn(E, batch_time(k, 0, n_dec, C2, 0));
            C2 += n_dec;
          }
        }
        g = nf - 1;
      }
      fin = lane_read(w.hv, g + 1 - w.hb);
      if constexpr (QC) finc = lane_read64(w.hvc, g + 1 - w.hb);
    }
    pre = pre0 + (g - g0);
    pre_sum -= ps0 - ps;
  }
  if (w.n_far > kWalkFar) return false;
  if (!ok && cap < max_iters) return false;   // past 2^31 - 1 batches: the engine decides
  const int li = n_list - n_pre;
  const int64_t aP = pre_sum, aD = n_dec;
  const int64_t aC = need_C ? c0sum + aD * g : 0;
  int64_t aA = 0;
  if (ok && need_A) {
    // prefill-attention feature of a batch serving the whole list: the head as it
    // stands, the others as the ring holds them (not yet served)
    int64_t a = 0;
    for (int base = 1; base < n_pre; base += kWave) {
      const int x = base + ln;
      if (x < n_pre) {
        int p2 = head + li + x;
        if (p2 >= rcap) p2 -= rcap;
        const int64_t r = e.r_rp[p2];
        a += r * e.r_cx[p2] + r * (r + 1) / 2;
      }
    }
    aA = wave_sum64(a);
    if (n_pre > 0) aA += (int64_t)h_rp * h_cx + (int64_t)h_rp * (h_rp + 1) / 2;
  }

  // decode tail: every list entry completes in the admission batch g + 1 (its last
  // token in batch g + 1 + rd); batch k after it holds the requests whose last token
  // is at or after batch g + 1 + k.
  const int K = tail_count(tr);
  if (ok) {
    // the window back into the ring (bins before g + 1 are spent)
    walk_lds_sync();
    {
      const int x = (w.hb + ln) & (kWalkBins - 1);
      lds.cnt[x] = w.hb + ln > g ? w.hv : 0;
      if constexpr (QC) lds.c0[x] = w.hb + ln > g ? w.hvc : 0;
    }
    walk_lds_sync();
    int64_t c0l = 0;   // context offsets of the list entries as decoding requests
    for (int base = 0; base < n_pre; base += kWave) {
      const int x = base + ln;
      const bool v = x < n_pre;
      int rp = 0, rd = 1, cx = 0;
      if (v) {
        if (x == 0) {
          rp = h_rp; rd = h_rd; cx = h_cx;
        } else {
          int p2 = head + li + x;
          if (p2 >= rcap) p2 -= rcap;
          rp = e.r_rp[p2]; rd = e.r_rd[p2]; cx = e.r_cx[p2];
        }
      }
      const int nl = g + 1 + rd;
      const int nc = cx + rp - (g + 1);
      if (need_C) c0l += v ? (int64_t)nc : 0;
      const bool far = v && rd > kWalkNear;
      const uint64_t fm = ballot(far);
      if (v && !far) {
        atomicAdd(&lds.cnt[nl & (kWalkBins - 1)], 1);
        if constexpr (QC)
          atomicAdd((unsigned long long*)&lds.c0[nl & (kWalkBins - 1)],
                    (unsigned long long)(int64_t)nc);
      }
      if (fm) {
        const int nf = popc(fm);
        if (w.n_far + nf > kWalkFar) return false;
        if (far) {
          const int y = w.n_far + mbcnt(fm);
          lds.flast[y] = nl;
          lds.fc0[y] = nc;
        }
        w.n_far += nf;
        w.far_next = min(w.far_next, wave_min(far ? nl : 0x7fffffff));
      }
    }
    if (need_C) c0l = wave_sum64(c0l);
    // batch g + 1: the decoding requests whose last token it is leave after it
    int64_t D = n_dec, c0 = c0sum;
    int b = g + 1;           // batch whose leavers are subtracted next
    int vb = b & ~(kWave - 1);
    walk_lds_sync();
    int cv = lds.cnt[(vb + ln) & (kWalkBins - 1)];
    int64_t cc = 0;
    if constexpr (QC) cc = lds.c0[(vb + ln) & (kWalkBins - 1)];
    for (int kk = 0; kk < K; ++kk, ++b) {
      if (b - vb >= kWave) {
        // bins read are zeroed, so that batches a whole ring later read zero
        lds.cnt[(vb + ln) & (kWalkBins - 1)] = 0;
        if constexpr (QC) lds.c0[(vb + ln) & (kWalkBins - 1)] = 0;
        vb += kWave;
        walk_lds_sync();
        cv = lds.cnt[(vb + ln) & (kWalkBins - 1)];
        if constexpr (QC) cc = lds.c0[(vb + ln) & (kWalkBins - 1)];
      }
      int f = lane_read(cv, b - vb);
      int64_t fc = 0;
      if constexpr (QC) fc = lane_read64(cc, b - vb);
      if (b == w.far_next) w.far_finish(b, f, fc);
      D -= f;
      c0 -= fc;
      if (kk == 0) {
        D += n_pre;
        c0 += c0l;
      }
      // batch kk + 1 after the admission batch (batch g + 2 + kk)
      if (ln == 0) {
        tr.tailD[(int64_t)kk * ZI + qid] = (int32_t)D;
        tr.tailC[(int64_t)kk * ZI + qid] = need_C ? c0 + D * (int64_t)(g + 1 + kk) : 0;
      }
    }
  } else if (ln == 0) {
    for (int kk = 0; kk < K; ++kk) {
      tr.tailD[(int64_t)kk * ZI + qid] = 0;
      tr.tailC[(int64_t)kk * ZI + qid] = 0;
    }
  }
  if (ln == 0) {
    tr.E[qid] = E;
    tr.pre[qid] = pre;
    tr.P[qid] = aP;
    tr.D[qid] = aD;
    tr.C[qid] = aC;
    tr.A[qid] = aA;
    tr.left[qid] = (int)((int64_t)B - aD - aP);
    tr.ok[qid] = ok;
  }
  return true;
}

}  // namespace lar
