// lar_board.cpp -- snapshot board: the consistency mechanism by which instances
// publish their resident-request snapshots to the router without pausing
// generation (appendix on the system: query workload snapshots and robustness to
// incomplete snapshots).
//
// One slot per instance, guarded by a sequence number.  A publisher makes the
// number odd (update in progress), writes the slot, and makes it even again
// (update complete).  The router copies a slot and keeps the copy only when the
// number was even before the copy and unchanged after it; otherwise it keeps the
// last complete copy it has.  Slot fields are written and read with relaxed atomic
// accesses, ordered by a release fence after the odd mark and an acquire fence
// before the final re-read, so a torn copy is always detected.
#include <atomic>
#include <cstdint>
#include <cstring>
#include <new>
#include <vector>

#include "../../include/lar.h"

namespace {

struct Slot {
  std::atomic<uint64_t> seq{0};
  int32_t n = 0;                  // written / read through relaxed atomics
  double clock = 0.0;
  std::vector<int32_t> rp, rd, cx;
};

struct Cached {
  bool have = false;
  uint64_t version = 0;           // sequence number of the copy
  int32_t n = 0;
  double clock = 0.0;
  std::vector<int32_t> rp, rd, cx;
};

template <class T>
inline void st(T* p, T v) { __atomic_store_n(p, v, __ATOMIC_RELAXED); }
template <class T>
inline T ld(const T* p) { return __atomic_load_n(p, __ATOMIC_RELAXED); }

inline void st_f64(double* p, double v) {
  uint64_t b;
  std::memcpy(&b, &v, 8);
  __atomic_store_n(reinterpret_cast<uint64_t*>(p), b, __ATOMIC_RELAXED);
}
inline double ld_f64(const double* p) {
  const uint64_t b = __atomic_load_n(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED);
  double v;
  std::memcpy(&v, &b, 8);
  return v;
}

constexpr int kAttempts = 4;   // copies tried per instance and collect

}  // namespace

struct lar_board {
  int32_t n_inst = 0, max_req = 0;
  std::vector<Slot> slots;
  std::vector<Cached> cache;
};

extern "C" {

lar_status lar_board_create(lar_board** out, int32_t n_inst, int32_t max_requests) {
  if (!out) return LAR_E_ARG;
  *out = nullptr;
  if (n_inst < 1 || max_requests < 0) return LAR_E_ARG;
  lar_board* b = new (std::nothrow) lar_board;
  if (!b) return LAR_E_ARG;
  try {
    b->n_inst = n_inst;
    b->max_req = max_requests;
    b->slots = std::vector<Slot>(n_inst);
    b->cache.resize(n_inst);
    for (auto& s : b->slots) {
      s.rp.assign(max_requests, 0);
      s.rd.assign(max_requests, 0);
      s.cx.assign(max_requests, 0);
    }
    for (auto& c : b->cache) {
      c.rp.assign(max_requests, 0);
      c.rd.assign(max_requests, 0);
      c.cx.assign(max_requests, 0);
    }
  } catch (...) {
    delete b;
    return LAR_E_ARG;
  }
  *out = b;
  return LAR_OK;
}

lar_status lar_board_destroy(lar_board* b) {
  delete b;
  return LAR_OK;
}

lar_status lar_board_publish(lar_board* b, int32_t inst, int32_t n_req,
                             const int32_t* rem_prefill, const int32_t* rem_decode,
                             const int32_t* context, double clock_ms) {
  if (!b || inst < 0 || inst >= b->n_inst || n_req < 0 || n_req > b->max_req) return LAR_E_ARG;
  if (n_req > 0 && (!rem_prefill || !rem_decode || !context)) return LAR_E_ARG;
  Slot& s = b->slots[inst];
  const uint64_t q = s.seq.load(std::memory_order_relaxed);
  s.seq.store(q + 1, std::memory_order_relaxed);          // odd: update in progress
  std::atomic_thread_fence(std::memory_order_release);
  st(&s.n, n_req);
  st_f64(&s.clock, clock_ms);
  for (int32_t i = 0; i < n_req; ++i) {
    st(&s.rp[i], rem_prefill[i]);
    st(&s.rd[i], rem_decode[i]);
    st(&s.cx[i], context[i]);
  }
  s.seq.store(q + 2, std::memory_order_release);          // even: complete
  return LAR_OK;
}

lar_status lar_board_collect(lar_board* b, int32_t* offsets, int32_t* rem_prefill,
                             int32_t* rem_decode, int32_t* context, double* clock_ms,
                             int64_t out_cap, int32_t* fresh, uint64_t* versions) {
  if (!b || !offsets || !clock_ms) return LAR_E_ARG;
  // refresh the cached copies
  std::vector<int32_t> tp(b->max_req), td(b->max_req), tc(b->max_req);
  for (int32_t j = 0; j < b->n_inst; ++j) {
    Slot& s = b->slots[j];
    Cached& c = b->cache[j];
    int32_t got = 0;
    for (int a = 0; a < kAttempts && !got; ++a) {
      const uint64_t q1 = s.seq.load(std::memory_order_acquire);
      if (q1 & 1) continue;                                  // update in progress
      if (c.have && q1 == c.version) { got = 2; break; }     // nothing new
      if (q1 == 0) break;                                    // never published
      int32_t n = ld(&s.n);
      const double clk = ld_f64(&s.clock);
      if (n < 0 || n > b->max_req) n = 0;                    // torn: rejected below
      for (int32_t i = 0; i < n; ++i) {
        tp[i] = ld(&s.rp[i]);
        td[i] = ld(&s.rd[i]);
        tc[i] = ld(&s.cx[i]);
      }
      std::atomic_thread_fence(std::memory_order_acquire);
      const uint64_t q2 = s.seq.load(std::memory_order_relaxed);
      if (q1 != q2) continue;                                // modified during the copy
      c.have = true;
      c.version = q1;
      c.n = n;
      c.clock = clk;
      std::copy(tp.begin(), tp.begin() + n, c.rp.begin());
      std::copy(td.begin(), td.begin() + n, c.rd.begin());
      std::copy(tc.begin(), tc.begin() + n, c.cx.begin());
      got = 1;
    }
    if (fresh) fresh[j] = got == 1 ? 1 : 0;
    if (versions) versions[j] = c.version;
  }
  // every instance needs a complete snapshot before the router can use the board
  int64_t total = 0;
  for (int32_t j = 0; j < b->n_inst; ++j) {
    if (!b->cache[j].have) return LAR_E_STATE;
    total += b->cache[j].n;
  }
  if (total > out_cap) return LAR_E_CAPACITY;
  if (total > 0 && (!rem_prefill || !rem_decode || !context)) return LAR_E_ARG;
  int64_t pos = 0;
  offsets[0] = 0;
  for (int32_t j = 0; j < b->n_inst; ++j) {
    const Cached& c = b->cache[j];
    std::copy(c.rp.begin(), c.rp.begin() + c.n, rem_prefill + pos);
    std::copy(c.rd.begin(), c.rd.begin() + c.n, rem_decode + pos);
    std::copy(c.cx.begin(), c.cx.begin() + c.n, context + pos);
    pos += c.n;
    offsets[j + 1] = (int32_t)pos;
    clock_ms[j] = c.clock;
  }
  return LAR_OK;
}

}  // extern "C"
