// sfs_limits.h -- the wave batch engine under scheduler limits: a per-request
// prefill chunk cap H, a context limit X and a KV cache of K blocks of 2^sh tokens
// with recompute preemption (the system appendix lists context limits, KV-cache
// allocation and preemption among what the simulation follows; Sec. 2 describes
// paged KV caches and chunked prefill).
//
// The batch, per instance:
//   * running requests in list order: one decode token to each decoding one, then
//     min(rp, H, budget left) to each partial prefill;
//   * when a request's new blocks (ceil((cx + n) / S) - ceil(cx / S)) do not fit, the
//     last running request is preempted until they do or the request itself is
//     out: it returns its blocks (with those taken in this batch) and its tokens of
//     this batch, and becomes the first waiting request with rp = cx + rp, cx = 0;
//   * only in a batch without preemption: admissions in FCFS order while budget is
//     left, fewer than M run and the first chunk's blocks fit.
// The predicted decode is cut to X - (cx + rp) when a request enters, which ends it
// at the context limit.
//
// One wavefront owns one (scenario, instance) queue.  Because a preempted request
// becomes the first waiting one in place, the resident list never reorders: it is
// kept in arrival order, running requests first.  Its first KS*64 entries (KS*64 >= M,
// so every entry a batch can touch) sit in registers, list position s*64 + lane in
// slot s; the rest stay in the queue's HBM ring at index (head + position) mod rcap.
// A batch is composed in parallel (saturating DPP prefix sums for the chunks, a
// block-count test, a prefix rule for the admissions); only a batch that must
// preempt is composed by one lane, step by step, over an LDS copy of the running
// requests.
#pragma once

#include "sfs_device.h"

namespace lar {

// Limits on device, [I] each: chunk cap (0: none), KV blocks (0: unlimited),
// log2 of the block size, context limit (0: none).
struct DevLimits {
  const int32_t *H, *K, *sh, *X;
};

// LDS words per wave of the limits engine: five rows of KS*64 (compaction staging,
// or the serial batch's working copy) and a few scalars.
template <int KS>
constexpr int lim_lds_words() { return 5 * KS * kWave + 4; }

struct LEnv {
  Coef k;
  int H;      // chunk cap, INT_MAX when none
  int K;      // KV blocks, 0 when unlimited
  int sh;     // log2 of the block size
  int X;      // context limit, 0 when none
  bool need_C, need_A;
  int32_t *r_rp, *r_rd, *r_cx, *r_seq;
  int rcap;
  int* lds;   // lim_lds_words<KS>() ints, 16-byte aligned
};

__device__ __forceinline__ LEnv make_lenv(const DevState& S, const DevParams& pr,
                                          const DevLimits& lm, int qid, int j, int* lds) {
  LEnv e;
  e.k = load_coef(pr, j);
  e.need_C = e.k.d != 0.0;
  e.need_A = e.k.e != 0.0;
  const int h = lm.H[j];
  e.H = h > 0 ? h : 0x7fffffff;
  e.K = lm.K[j];
  e.sh = lm.sh[j];
  e.X = lm.X[j];
  e.rcap = S.rcap;
  const int64_t rb = (int64_t)qid * S.rcap;
  e.r_rp = S.r_rp + rb; e.r_rd = S.r_rd + rb; e.r_cx = S.r_cx + rb; e.r_seq = S.r_seq + rb;
  e.lds = lds;
  return e;
}

// Blocks that hold x cached tokens.
__device__ __forceinline__ int kv_blocks(int x, int sh) {
  return (int)(((int64_t)x + (1 << sh) - 1) >> sh);
}

// Predicted decode of a request entering with p prompt tokens: >= 1, cut to what the
// context limit leaves (0 when p does not fit it).
__device__ __forceinline__ int entry_decode(const LEnv& e, int p, int d) {
  d = d < 1 ? 1 : d;
  if (e.X > 0) {
    if (p >= e.X) return 0;
    if (d > e.X - p) d = e.X - p;
  }
  return d;
}

// First-token outputs of a replay that tracks routed queries (see the trace kernels).
struct LTrack {
  double* out;   // [N] first-token time per query of the running trace
  int tag0, N, reading;
};

struct LStep {
  double T;        // batch time
  bool last_dec;   // the last list entry received a decode token
  bool last_fill;  // the last list entry's prefill completed
  bool tail_ok;    // (TAIL steps) a new request at the tail could have been admitted
};

template <int KS>
struct LQueue {
  int rp[KS], rd[KS], cx[KS], sq[KS], tg[KS];
  int nwin;      // window entries (positions 0 .. nwin-1)
  int n_list;    // list length
  int n_run;     // running prefix
  int head;      // ring index of list position 0
  int next_seq;
  int ntrk;      // tracked queries without a first token (tracking replays)
  double clock;
  int64_t iters;
  // a query appended by an estimate to its private copy is written nowhere: while it
  // lies beyond the window it lives here, at list position n_list - 1
  bool vq;
  int vq_p, vq_d;

  template <bool TRK>
  __device__ void fetch(const LEnv& e, const int32_t* tags, int s, int pos) {
    if (vq && pos == n_list - 1) {
      rp[s] = vq_p; rd[s] = vq_d; cx[s] = 0; sq[s] = next_seq - 1;
      if constexpr (TRK) tg[s] = -1;
      return;
    }
    int r = head + pos;
    if (r >= e.rcap) r -= e.rcap;
    rp[s] = e.r_rp[r]; rd[s] = e.r_rd[r]; cx[s] = e.r_cx[r]; sq[s] = e.r_seq[r];
    if constexpr (TRK) tg[s] = tags[r];
  }

  // Bring list positions nwin .. min(n_list, KS*64) - 1 into the window.
  template <bool TRK>
  __device__ void refill(const LEnv& e, const int32_t* tags) {
    const int want = min(n_list, KS * kWave);
    if (nwin >= want) return;
    const int ln = lane_id();
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int pos = s * kWave + ln;
      if (pos >= nwin && pos < want) fetch<TRK>(e, tags, s, pos);
    }
    nwin = want;
  }

  template <bool TRK>
  __device__ void load(const DevState& S, const LEnv& e, int qid, const int32_t* tags) {
    const QScal* q = S.sc + qid;
    n_list = uni(q->n_pre); n_run = uni(q->n_part); head = uni(q->head);
    next_seq = uni(q->next_seq);
    ntrk = TRK ? uni(q->ntrk) : 0;
    clock = q->clock;
    iters = uni64(q->iters);
    vq = false; vq_p = 0; vq_d = 0;
    nwin = 0;
#pragma unroll
    for (int s = 0; s < KS; ++s) { rp[s] = 0; rd[s] = 0; cx[s] = 0; sq[s] = 0; tg[s] = -1; }
    refill<TRK>(e, tags);
  }

  template <bool TRK>
  __device__ void store(const DevState& S, const LEnv& e, int qid, int32_t* tags) const {
    const int ln = lane_id();
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int pos = s * kWave + ln;
      if (pos < nwin) {
        int r = head + pos;
        if (r >= e.rcap) r -= e.rcap;
        e.r_rp[r] = rp[s]; e.r_rd[r] = rd[s]; e.r_cx[r] = cx[s]; e.r_seq[r] = sq[s];
        if constexpr (TRK) tags[r] = tg[s];
      }
    }
    if (ln == 0) {
      QScal* q = S.sc + qid;
      q->g = 0; q->n_dec = 0; q->n_part = n_run; q->n_pre = n_list; q->head = head;
      q->next_seq = next_seq; q->c0sum = 0; q->pre_sum = 0; q->clock = clock;
      q->iters = iters;
      if constexpr (TRK) { q->ntrk = ntrk; q->pend = 0; }
    }
    // the same wave loads this queue again later in the same kernel
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  }

  __device__ int waiting() const { return n_list - n_run; }

  // Append a waiting request at the tail (the caller checked p and the capacity).
  // real == false: an estimate's private copy; nothing is written to HBM.
  template <bool TRK>
  __device__ void append(const LEnv& e, int p, int d, bool real, int32_t* tags, int tag) {
    const int ln = lane_id();
    const int pos = n_list;
    if (nwin == n_list && pos < KS * kWave) {
#pragma unroll
      for (int s = 0; s < KS; ++s)
        if (s * kWave + ln == pos) {
          rp[s] = p; rd[s] = d; cx[s] = 0; sq[s] = next_seq;
          if constexpr (TRK) tg[s] = tag;
        }
      nwin = pos + 1;
    } else if (real) {
      if (ln == 0) {
        int r = head + pos;
        if (r >= e.rcap) r -= e.rcap;
        e.r_rp[r] = p; e.r_rd[r] = d; e.r_cx[r] = 0; e.r_seq[r] = next_seq;
        if constexpr (TRK) tags[r] = tag;
      }
      // other lanes of this wave read the entry back on refill
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    } else {
      vq = true; vq_p = p; vq_d = d;
    }
    n_list += 1;
    next_seq += 1;
  }

  // The batch when it must preempt, following the rule step by step on an LDS copy
  // of the running requests.  Only three kinds of request can change the outcome: the
  // decoding ones that need a new block (in list order), the partial prefills (in
  // list order) and the victims (from the end); the wave lists the first two and one
  // lane walks them.  Every other decoding request is served exactly when it is still
  // running after the walk.  On return dec / chk hold the tokens of each running
  // request, the victims are waiting again (rp, cx updated) and n_run is the new
  // running count.  Admissions do not happen in such a batch.
  __device__ void compose_serial(const LEnv& e, int free0, int (&dec)[KS], int (&chk)[KS]) {
    const int ln = lane_id();
    const int sh = e.sh;
    int* Lrp = e.lds;
    int* Lcx = Lrp + KS * kWave;
    int* Lch = Lcx + KS * kWave;
    int* Lnd = Lch + KS * kWave;   // positions of the decoding requests that need a block
    int* Lpt = Lnd + KS * kWave;   // positions of the partial prefills
    int* Lsc = Lpt + KS * kWave;
    int nn = 0, np = 0, ndec = 0;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int i = s * kWave + ln;
      const bool run = i < n_run;
      if (run) { Lrp[i] = rp[s]; Lcx[i] = cx[s]; Lch[i] = 0; }
      const bool isdec = run && rp[s] == 0;
      const bool needy = isdec && kv_blocks(cx[s] + 1, sh) > kv_blocks(cx[s], sh);
      const bool part = run && rp[s] > 0;
      const uint64_t mn = ballot(needy), mp = ballot(part);
      if (needy) Lnd[nn + mbcnt(mn)] = i;
      if (part) Lpt[np + mbcnt(mp)] = i;
      nn += popc(mn);
      np += popc(mp);
      ndec += popc(ballot(isdec));
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (ln == 0) {
      int run = n_run, freeb = free0, dvict = 0;
      // decode tokens: each decoding request that needs a block takes one, preempting
      // from the end while none is free
      for (int k = 0; k < nn; ++k) {
        const int r = Lnd[k];
        while (freeb < 1 && r < run) {
          const int v = run - 1;
          const int rv = Lrp[v], cv = Lcx[v];
          freeb += kv_blocks(cv, sh);
          dvict += rv == 0 ? 1 : 0;
          Lrp[v] = rv + cv;
          Lcx[v] = 0;
          run = v;
        }
        if (r >= run) break;
        freeb -= 1;
      }
      const int run1 = run;   // decoding requests below run1 hold a decode token
      int left = e.k.B - (ndec - dvict);
      // chunks of the partial prefills; a victim that decodes in this batch returns
      // its token and the block it took for it
      for (int k = 0; k < np; ++k) {
        const int r = Lpt[k];
        if (r >= run || left == 0) break;
        const int g = min(min(Lrp[r], e.H), left);
        const int cr = Lcx[r];
        const int need = kv_blocks(cr + g, sh) - kv_blocks(cr, sh);
        while (freeb < need && r < run) {
          const int v = run - 1;
          const int rv = Lrp[v], cv = Lcx[v];
          if (rv == 0 && v < run1) {
            freeb += kv_blocks(cv + 1, sh);
            left += 1;
          } else {
            freeb += kv_blocks(cv, sh);
          }
          Lrp[v] = rv + cv;
          Lcx[v] = 0;
          run = v;
        }
        if (r >= run) break;
        Lch[r] = g;
        freeb -= need;
        left -= g;
      }
      Lsc[0] = run;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const int run_end = uni(Lsc[0]);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int i = s * kWave + ln;
      if (i < n_run) {
        const bool isdec = rp[s] == 0;
        dec[s] = (isdec && i < run_end) ? 1 : 0;
        chk[s] = (!isdec && i < run_end) ? Lch[i] : 0;
        rp[s] = Lrp[i];
        cx[s] = Lcx[i];
      }
    }
    n_run = run_end;
    // the LDS area is reused by the next batch
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }

  // Remove the finished window entries (fin[s] on this lane), keeping the order, and
  // refill the window from the ring.
  template <bool TRK>
  __device__ void compact(const LEnv& e, const int32_t* tags, const bool (&fin)[KS], int nf) {
    const int ln = lane_id();
    int* Srp = e.lds;
    int* Srd = Srp + KS * kWave;
    int* Scx = Srd + KS * kWave;
    int* Ssq = Scx + KS * kWave;
    int* Stg = Ssq + KS * kWave;
    int base = 0;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const bool keep = s * kWave + ln < nwin && !fin[s];
      const uint64_t m = ballot(keep);
      if (keep) {
        const int dst = base + mbcnt(m);
        Srp[dst] = rp[s]; Srd[dst] = rd[s]; Scx[dst] = cx[s]; Ssq[dst] = sq[s];
        if constexpr (TRK) Stg[dst] = tg[s];
      }
      base += popc(m);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const int nw = nwin - nf;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int pos = s * kWave + ln;
      if (pos < nw) {
        rp[s] = Srp[pos]; rd[s] = Srd[pos]; cx[s] = Scx[pos]; sq[s] = Ssq[pos];
        if constexpr (TRK) tg[s] = Stg[pos];
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    nwin = nw;
    n_list -= nf;
    n_run -= nf;
    head += nf;
    if (head >= e.rcap) head -= e.rcap;
    refill<TRK>(e, tags);
  }

  // One batch: compose, time, (TRK) first tokens at the batch end clk0 + T, apply.
  // Only the window rows that hold entries are visited (wave-uniform row count), the
  // chunk pass is skipped when no request has prefill left, and the admission pass
  // when no request waits.  TAIL: also report whether a request appended at the tail
  // before this batch could have been admitted in it -- no preemption, every waiting
  // request admitted, a sequence slot, budget and a KV block left -- which every
  // admission needs, whatever the request's prompt.
  template <bool TRK, bool TAIL = false>
  __device__ LStep step(const LEnv& e, const int32_t* tags, double clk0, const LTrack* tk) {
    const int ln = lane_id();
    const int sh = e.sh;
    const bool kv = e.K > 0;
    const int B = e.k.B, M = e.k.M;
    const int nrows = (nwin + kWave - 1) >> 6;
    int dec[KS], chk[KS];
    bool wait[KS];
    // decoding requests, their new blocks, the blocks held
    int nd = 0, held = 0, need = 0;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      dec[s] = 0; chk[s] = 0; wait[s] = false;
      if (s < nrows) {
        const int i = s * kWave + ln;
        const bool run = i < n_run;
        dec[s] = (run && rp[s] == 0) ? 1 : 0;
        nd += dec[s];
        if (kv && run) {
          const int h = kv_blocks(cx[s], sh);
          held += h;
          if (dec[s]) need += kv_blocks(cx[s] + 1, sh) - h;
        }
      }
    }
    int D = wave_sum32(nd);
    const int L1 = B - D;
    const bool waiting_any = n_list > n_run;
    const bool prefill_any = waiting_any || n_run > D;
    // chunks: each partial prefill, then each waiting request within the sequence
    // cap, wants min(rp, H); the budget left after the decodes goes to them in list
    // order (exclusive saturating prefix sums, row by row)
    if (prefill_any) {
      unsigned carry = 0;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        if (s < nrows) {
          const int i = s * kWave + ln;
          const bool part = i < n_run && rp[s] > 0;
          wait[s] = i >= n_run && i < nwin && i < M;
          const int want = (part || wait[s]) ? min(min(rp[s], e.H), L1) : 0;
          const unsigned excl =
              min((unsigned)scan_sat(prev_lane(want), L1) + carry, (unsigned)L1);
          chk[s] = min(want, L1 - (int)excl);
          carry = (unsigned)uni(lane_last((int)min(excl + (unsigned)want, (unsigned)L1)));
          if (kv && part) need += kv_blocks(cx[s] + chk[s], sh) - kv_blocks(cx[s], sh);
        }
      }
    }
    bool preempted = false;
    int room = 0;
    if (kv) {
      room = e.K - wave_sum32(held);    // free blocks
      const int n12 = wave_sum32(need);
      if (n12 > room) preempted = true;
      room -= n12;
    }
    int admitted = 0;
    if (preempted) {
#pragma unroll
      for (int s = 0; s < KS; ++s) { dec[s] = 0; chk[s] = 0; }
      compose_serial(e, room + wave_sum32(need), dec, chk);
      int x = 0;
#pragma unroll
      for (int s = 0; s < KS; ++s) x += dec[s];
      D = wave_sum32(x);
    } else if (waiting_any) {
      // admissions: a prefix of the waiting requests, cut where the budget, the
      // sequence cap or the blocks of a first chunk run out
      int bcarry = 0, nadm = 0, nblk = 0;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        if (s < nrows && (s + 1) * kWave > n_run) {
          const int need3 = (kv && wait[s] && chk[s] > 0) ? kv_blocks(chk[s], sh) : 0;
          int cum = bcarry;
          if (kv) {
            cum += scan_add32(need3);
            bcarry = uni(lane_last(cum));
          }
          const bool ok = wait[s] && chk[s] > 0 && (!kv || cum <= room);
          if (wait[s] && !ok) chk[s] = 0;
          nadm += ok ? 1 : 0;
          if constexpr (TAIL) nblk += ok ? need3 : 0;
        }
      }
      admitted = wave_sum32(nadm);
      if constexpr (TAIL) room -= kv ? wave_sum32(nblk) : 0;
    }
    // features and time
    int P = 0;
    int64_t C = 0, A = 0;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      if (s < nrows) {
        P += chk[s];
        if (e.need_C && dec[s]) C += cx[s];
        if (e.need_A && chk[s])
          A += (int64_t)chk[s] * cx[s] + (int64_t)chk[s] * (chk[s] + 1) / 2;
      }
    }
    P = prefill_any ? wave_sum32(P) : 0;
    if (e.need_C) C = wave_sum64(C);
    if (e.need_A) A = wave_sum64(A);
    LStep o;
    o.T = batch_time(e.k, P, D, C, A);
    o.tail_ok = false;
    if constexpr (TAIL)
      o.tail_ok = !preempted && admitted == n_list - n_run && n_run + admitted < M &&
                  L1 - P > 0 && (!kv || room >= 1);
    // the last list entry (an estimate's query)
    const int lp = n_list - 1;
    bool ld = false, lf = false;
#pragma unroll
    for (int s = 0; s < KS; ++s)
      if (s == (lp >> 6) && ln == (lp & (kWave - 1))) {
        ld = dec[s] != 0;
        lf = chk[s] > 0 && chk[s] == rp[s];
      }
    o.last_dec = ballot(ld) != 0;
    o.last_fill = ballot(lf) != 0;
    if constexpr (TRK) {
      const double end = __dadd_rn(clk0, o.T);
      int hit = 0;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        if (s < nrows) {
          const bool first =
              tk->reading == 1 ? (chk[s] > 0 && chk[s] == rp[s]) : dec[s] != 0;
          const int q = tg[s] - tk->tag0;
          if (first && tg[s] >= 0 && q >= 0 && q < tk->N) {
            tk->out[q] = end;
            tg[s] = -1;
            ++hit;
          }
        }
      }
      ntrk -= wave_sum32(hit);
    }
    // apply; decoding requests whose predicted decode is used up leave
    bool fin[KS];
    int nf = 0;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      fin[s] = false;
      if (s < nrows) {
        if (dec[s]) { cx[s] += 1; rd[s] -= 1; }
        if (chk[s]) { cx[s] += chk[s]; rp[s] -= chk[s]; }
        fin[s] = dec[s] && rd[s] == 0;
        nf += fin[s] ? 1 : 0;
      }
    }
    n_run += admitted;
    nf = wave_sum32(nf);
    if (nf > 0) compact<TRK>(e, tags, fin, nf);
    return o;
  }
};

}  // namespace lar
