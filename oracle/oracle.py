"""ctypes wrapper over the plain C oracle (``sfs_oracle.c``).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the CPU-baseline leg
of the benchmark use it.  The product path never imports this module.

``build()`` compiles the oracle with gcc (-O2 -ffp-contract=off: binary64
round-to-nearest-even, no fused multiply-add); ``lib()`` loads it, building it
first if it is missing.

Threads: ``set_threads(n)`` lets the oracle run the independent estimates of one
query (one per instance), the replays of the instances and the pairs of a what-if
matrix on n threads; ``trace_scenarios`` runs independent scenarios on threads of
their own.  Each thread runs the same sequential code on its own instance or
scenario and results are gathered in order, so threaded runs are bit-identical to
single-threaded ones (a CPU test checks it).  The default is one thread.
"""

from __future__ import annotations

import ctypes as C
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sfs_oracle.c")
_LIB = os.path.join(_HERE, "libsfs_oracle.so")

OK, E_ARG, E_STATE, E_CAPACITY, E_ITER = 0, -1, -2, -3, -4
READING_DECODE_BATCH = 0      # first token = first batch in which the query decodes
READING_PREFILL_BATCH = 1     # first token = batch completing the query's prefill


class OracleError(RuntimeError):
    def __init__(self, code, where=""):
        super().__init__(f"oracle error {code} {where}")
        self.code = code


class Params(C.Structure):
    _fields_ = [("a", C.c_double), ("b", C.c_double), ("c", C.c_double), ("d", C.c_double),
                ("e", C.c_double), ("budget", C.c_int32), ("max_seqs", C.c_int32)]


def build(force: bool = True) -> str:
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math",
                        "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra", "-o", tmp, _SRC],
                       check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None

_i32p = np.ctypeslib.ndpointer(np.int32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(np.int64, flags="C_CONTIGUOUS")


def _opt(ptr_type):
    """ndpointer that also accepts None."""
    class _Opt(ptr_type):
        @classmethod
        def from_param(cls, obj):
            if obj is None:
                return None
            return super().from_param(obj)
    return _Opt


def lib():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build(force=True)
    L = C.CDLL(_LIB)
    L.orc_queue_new.restype = C.c_void_p
    L.orc_queue_new.argtypes = [C.POINTER(Params), C.c_int64, _i32p, _i32p, _i32p, C.c_double,
                                C.POINTER(C.c_int)]
    L.orc_queue_free.argtypes = [C.c_void_p]
    L.orc_queue_size.restype = C.c_int64
    L.orc_queue_size.argtypes = [C.c_void_p]
    L.orc_queue_waiting.restype = C.c_int64
    L.orc_queue_waiting.argtypes = [C.c_void_p]
    L.orc_queue_get.argtypes = [C.c_void_p, _i32p, _i32p, _i32p, C.POINTER(C.c_double),
                                C.POINTER(C.c_int64)]
    L.orc_queue_step.restype = C.c_double
    L.orc_queue_step.argtypes = [C.c_void_p, _i64p]
    L.orc_queue_advance.restype = C.c_int
    L.orc_queue_advance.argtypes = [C.c_void_p, C.c_double, C.c_int64]
    L.orc_queue_append.restype = C.c_int
    L.orc_queue_append.argtypes = [C.c_void_p, C.c_int32, C.c_int32, C.c_int64]
    L.orc_queue_estimate.restype = C.c_int
    L.orc_queue_estimate.argtypes = [C.c_void_p, C.c_int32, C.c_int32, C.c_double, C.c_int32,
                                     C.c_int64, C.POINTER(C.c_double), C.POINTER(C.c_int32)]
    L.orc_route_row.restype = C.c_int32
    L.orc_route_row.argtypes = [C.c_int32, _f64p, _f64p, _f64p, _i32p, C.c_double, C.c_double,
                                C.POINTER(C.c_double)]
    L.orc_trace.restype = C.c_int
    L.orc_trace.argtypes = [C.c_int32, C.POINTER(Params), _i32p, _i32p, _i32p, _i32p, _i32p,
                            _f64p, C.c_int32, _i32p, _i32p, _f64p, _f64p, _f64p, C.c_int32,
                            C.c_double, C.c_double, _opt(_f64p), C.c_int32, C.c_int64, C.c_int64,
                            _i32p, _opt(_f64p), _opt(_f64p), _opt(_f64p), _opt(_i32p),
                            _opt(_i32p), _opt(_i32p), _opt(_i32p), _opt(_i32p), _opt(_f64p),
                            _opt(_i64p), C.c_int64, _opt(_f64p), _opt(_i32p),
                            C.POINTER(C.c_int32)]
    L.orc_queue_preemptions.restype = C.c_int64
    L.orc_queue_preemptions.argtypes = [C.c_void_p]
    L.orc_queue_set_sched.restype = C.c_int
    L.orc_queue_set_sched.argtypes = [C.c_void_p, _i32p]
    L.orc_route_row_constrained.restype = C.c_int32
    L.orc_route_row_constrained.argtypes = [C.c_int32, _f64p, C.c_double, _f64p, _f64p, _i32p,
                                            C.c_double]
    L.orc_ttft_target.restype = C.c_double
    L.orc_ttft_target.argtypes = [C.c_int32, C.c_double, C.c_double]
    L.orc_ttft_targets.restype = None
    L.orc_ttft_targets.argtypes = [C.c_int32, _i32p, _f64p, _f64p, _f64p]
    L.orc_ontime_utility.restype = C.c_int
    L.orc_ontime_utility.argtypes = [C.c_int32, _i32p, _f64p, _f64p, _f64p, _f64p, C.c_int32,
                                     _i32p, C.c_double, C.POINTER(C.c_double)]
    L.orc_set_threads.restype = None
    L.orc_set_threads.argtypes = [C.c_int]
    L.orc_get_threads.restype = C.c_int
    L.orc_get_threads.argtypes = []
    L.orc_estimate_matrix.restype = C.c_int
    L.orc_estimate_matrix.argtypes = [C.c_int32, C.POINTER(C.c_void_p), C.c_int32, _i32p, _i32p,
                                      C.c_double, C.c_int32, C.c_int64, _f64p, _i32p]
    L.orc_lps_wait.restype = C.c_double
    L.orc_lps_wait.argtypes = [C.c_double, C.c_double, C.c_int32, C.c_int32, C.c_double,
                               C.c_double]
    L.orc_lps_ttft.restype = C.c_double
    L.orc_lps_ttft.argtypes = [C.c_double, C.c_double, C.c_int32, C.c_int32, C.c_double,
                               C.c_double, C.c_double, C.c_double, C.c_int32]
    L.orc_lps_matrix.restype = None
    L.orc_lps_matrix.argtypes = [C.c_int32, _f64p, _f64p, _i32p, _f64p, _f64p, _f64p, _f64p,
                                 C.c_int32, C.c_int32, _i32p, _f64p]
    L.orc_stats.restype = C.c_int
    L.orc_stats.argtypes = [C.c_int32, _i32p, _f64p, _f64p, _f64p, C.c_int32, _i32p, C.c_double,
                            _f64p]
    _lib = L
    return L


def set_threads(n: int) -> None:
    """Threads for the independent per-instance work of one query (default 1)."""
    lib().orc_set_threads(int(n))


def get_threads() -> int:
    return int(lib().orc_get_threads())


def make_params(a, b, c, d, e, budget, max_seqs) -> Params:
    return Params(float(a), float(b), float(c), float(d), float(e), int(budget), int(max_seqs))


def params_of(wl, j) -> Params:
    return make_params(wl.a[j], wl.b[j], wl.c[j], wl.d[j], wl.e[j], wl.budget[j], wl.max_seqs[j])


def _i32(x):
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


class Queue:
    """One instance's resident list with its clock (the oracle's state)."""

    def __init__(self, params: Params, rp, rd, cx, clock=0.0, sched=None):
        self._L = lib()
        st = C.c_int(0)
        rp, rd, cx = _i32(rp), _i32(rd), _i32(cx)
        self._p = params
        self._q = self._L.orc_queue_new(C.byref(params), len(rp), rp, rd, cx, float(clock),
                                        C.byref(st))
        if st.value != OK:
            raise OracleError(st.value, "queue_new")
        if sched is not None:
            self.set_sched(sched)

    def set_sched(self, sched):
        """Scheduler limits (chunk_cap, kv_blocks, block_size, max_ctx); 0 = none."""
        st = self._L.orc_queue_set_sched(self._q, _i32(sched))
        if st != OK:
            raise OracleError(st, "set_sched")

    def __del__(self):
        q = getattr(self, "_q", None)
        if q:
            self._L.orc_queue_free(q)
            self._q = None

    def size(self) -> int:
        return int(self._L.orc_queue_size(self._q))

    def preemptions(self) -> int:
        """Requests preempted since the queue was created (its clones start at 0)."""
        return int(self._L.orc_queue_preemptions(self._q))

    def waiting(self) -> int:
        return int(self._L.orc_queue_waiting(self._q))

    def state(self):
        n = self.size()
        rp, rd, cx = (np.zeros(n, np.int32) for _ in range(3))
        clk, it = C.c_double(0), C.c_int64(0)
        self._L.orc_queue_get(self._q, rp, rd, cx, C.byref(clk), C.byref(it))
        return rp, rd, cx, clk.value, it.value

    def step(self):
        f = np.zeros(4, np.int64)
        T = self._L.orc_queue_step(self._q, f)
        return T, tuple(int(x) for x in f)

    def advance(self, t, max_iters=10_000_000):
        st = self._L.orc_queue_advance(self._q, float(t), int(max_iters))
        if st != OK:
            raise OracleError(st, "advance")

    def append(self, p, d, queue_cap=1 << 40):
        st = self._L.orc_queue_append(self._q, int(p), int(d), int(queue_cap))
        if st != OK:
            raise OracleError(st, "append")

    def estimate(self, p, d, t, reading=READING_DECODE_BATCH, max_iters=10_000_000):
        tt, it = C.c_double(0), C.c_int32(0)
        st = self._L.orc_queue_estimate(self._q, int(p), int(d), float(t), int(reading),
                                        int(max_iters), C.byref(tt), C.byref(it))
        if st != OK:
            raise OracleError(st, "estimate")
        return tt.value, it.value


def route_row(ttft, acc_row, cost_row, col, w_cost, w_lat):
    ttft = np.ascontiguousarray(ttft, np.float64)
    bu = C.c_double(0)
    m = lib().orc_route_row(len(ttft), ttft, np.ascontiguousarray(acc_row, np.float64),
                            np.ascontiguousarray(cost_row, np.float64), _i32(col),
                            float(w_cost), float(w_lat), C.byref(bu))
    return int(m), bu.value


def route_row_constrained(ttft, tau, acc_row, cost_row, col, w_cost):
    """Eq. 3: best utility within the TTFT target, else the least estimated TTFT."""
    ttft = np.ascontiguousarray(ttft, np.float64)
    return int(lib().orc_route_row_constrained(len(ttft), ttft, float(tau),
                                               np.ascontiguousarray(acc_row, np.float64),
                                               np.ascontiguousarray(cost_row, np.float64),
                                               _i32(col), float(w_cost)))


def ttft_target(p, u_ms, v):
    return float(lib().orc_ttft_target(int(p), float(u_ms), float(v)))


def ttft_targets(p, u_ms, v):
    """Per-query TTFT targets (ms) from the prompt lengths and the drawn u, v."""
    p = _i32(p)
    out = np.zeros(len(p))
    lib().orc_ttft_targets(len(p), p, np.ascontiguousarray(u_ms, np.float64),
                           np.ascontiguousarray(v, np.float64), out)
    return out


def ontime_utility(choice, ttft_real, tau, acc, cost, col, w_cost):
    """Eq. 4 over a routed trace, from the realised TTFT of each query."""
    n = len(choice)
    out = C.c_double(0)
    st = lib().orc_ontime_utility(n, _i32(choice), np.ascontiguousarray(ttft_real, np.float64),
                                  np.ascontiguousarray(tau[:n], np.float64),
                                  np.ascontiguousarray(acc[:n], np.float64),
                                  np.ascontiguousarray(cost[:n], np.float64), acc.shape[1],
                                  _i32(col), float(w_cost), C.byref(out))
    if st != OK:
        raise OracleError(st, "ontime_utility")
    return out.value


@dataclass
class TraceResult:
    choice: np.ndarray
    ttft_chosen: np.ndarray
    util_chosen: np.ndarray
    ttft_all: np.ndarray | None
    iters_all: np.ndarray | None
    offsets: np.ndarray | None
    rem_prefill: np.ndarray | None
    rem_decode: np.ndarray | None
    context: np.ndarray | None
    clock_ms: np.ndarray | None
    iterations: np.ndarray | None
    realized: np.ndarray          # realised TTFT of each query in the replay


def trace(wl, scenario: int = 0, *, n_q: int | None = None, reading=READING_DECODE_BATCH,
          max_iters=10_000_000, full_rows=False, final_state=True, queue_cap=None,
          tau=None) -> TraceResult:
    """Sequential routing trace of one scenario of workload ``wl`` (first n_q queries);
    Lagrangian route, or the constrained route of Eq. 3 when per-query targets
    ``tau`` (ms) are given.  The workload's scheduler limits (``wl.sched``, [I][4])
    apply when set."""
    L = lib()
    I = wl.n_inst
    N = wl.n_q if n_q is None else int(n_q)
    params = (Params * I)(*[params_of(wl, j) for j in range(I)])
    choice = np.zeros(N, np.int32)
    ttft_c = np.zeros(N)
    util_c = np.zeros(N)
    ttft_all = np.zeros((N, I)) if full_rows else None
    iters_all = np.zeros((N, I), np.int32) if full_rows else None
    cap = int(wl.queue_cap if queue_cap is None else queue_cap)
    if final_state:
        out_cap = int(wl.offsets[-1]) + N
        out_off = np.zeros(I + 1, np.int32)
        out_rp, out_rd, out_cx = (np.zeros(out_cap, np.int32) for _ in range(3))
        out_clock = np.zeros(I)
        out_iters = np.zeros(I, np.int64)
    else:
        out_cap = 0
        out_off = out_rp = out_rd = out_cx = out_clock = out_iters = None
    realized = np.zeros(N)
    failed = C.c_int32(-1)
    st = L.orc_trace(I, params, _i32(wl.col), _i32(wl.offsets), _i32(wl.rem_prefill),
                     _i32(wl.rem_decode), _i32(wl.context),
                     np.ascontiguousarray(wl.clock_ms, np.float64), N,
                     _i32(wl.q_prefill[:N]), _i32(wl.q_decode[:N]),
                     np.ascontiguousarray(wl.q_t_ms[:N], np.float64),
                     np.ascontiguousarray(wl.acc[:N], np.float64),
                     np.ascontiguousarray(wl.cost[:N], np.float64), wl.n_cols,
                     float(wl.w_cost[scenario]), float(wl.w_lat_ms[scenario]),
                     None if tau is None else np.ascontiguousarray(tau[:N], np.float64),
                     int(reading),
                     int(max_iters), cap, choice, ttft_c, util_c, ttft_all, iters_all,
                     out_off, out_rp, out_rd, out_cx, out_clock, out_iters, out_cap,
                     realized, sched_of(wl), C.byref(failed))
    if st != OK:
        raise OracleError(st, f"trace (query {failed.value})")
    if final_state:
        n = int(out_off[-1])
        out_rp, out_rd, out_cx = out_rp[:n], out_rd[:n], out_cx[:n]
    return TraceResult(choice, ttft_c, util_c, ttft_all, iters_all, out_off, out_rp, out_rd,
                       out_cx, out_clock, out_iters, realized)


def stats(choice, ttft_chosen, acc, cost, col, w_cost):
    """Mean accuracy, mean cost, mean utility, p50 and p99 TTFT of a routed trace."""
    n = len(choice)
    out = np.zeros(5)
    st = lib().orc_stats(n, _i32(choice), np.ascontiguousarray(ttft_chosen, np.float64),
                         np.ascontiguousarray(acc[:n], np.float64),
                         np.ascontiguousarray(cost[:n], np.float64), acc.shape[1], _i32(col),
                         float(w_cost), out)
    if st != OK:
        raise OracleError(st, "stats")
    return out


def sched_of(wl):
    """The workload's scheduler limits as a flat int32 [I*4] array, or None."""
    sc = getattr(wl, "sched", None)
    return None if sc is None else _i32(np.asarray(sc).reshape(-1))


def instance_queue(wl, j) -> Queue:
    rp, rd, cx = wl.instance_requests(j)
    sc = getattr(wl, "sched", None)
    return Queue(params_of(wl, j), rp, rd, cx, wl.clock_ms[j],
                 sched=None if sc is None else np.asarray(sc)[j])


def estimate_matrix(wl, queries, instances, t_ms=0.0, reading=READING_DECODE_BATCH,
                    max_iters=10_000_000):
    """Literal per-pair SFS estimates for the given query and instance indices."""
    qs = {j: instance_queue(wl, j) for j in sorted(set(int(j) for j in instances))}
    out = np.zeros((len(queries), len(instances)))
    its = np.zeros((len(queries), len(instances)), np.int32)
    for a, i in enumerate(queries):
        for b, j in enumerate(instances):
            out[a, b], its[a, b] = qs[int(j)].estimate(int(wl.q_prefill[i]),
                                                       int(wl.q_decode[i]), t_ms, reading,
                                                       max_iters)
    return out, its


def estimate_matrix_all(wl, t_ms=0.0, *, queries=None, reading=READING_DECODE_BATCH,
                        max_iters=10_000_000):
    """The literal what-if matrix: TTFT and batch count of every query (all, or the
    given indices) at every instance of ``wl``, each pair simulated on its own copy
    of the instance (runs on ``set_threads`` threads).  Returns (ttft, iters), both
    [Q][I]."""
    qidx = np.arange(wl.n_q) if queries is None else np.asarray(queries, np.int64)
    qs = [instance_queue(wl, j) for j in range(wl.n_inst)]
    for q in qs:
        if q._L is None or q._q is None:
            raise OracleError(E_ARG, "queue")
    ptrs = (C.c_void_p * wl.n_inst)(*[q._q for q in qs])
    p = _i32(np.asarray(wl.q_prefill)[qidx])
    d = _i32(np.asarray(wl.q_decode)[qidx])
    ttft = np.zeros((len(qidx), wl.n_inst))
    iters = np.zeros((len(qidx), wl.n_inst), np.int32)
    st = lib().orc_estimate_matrix(wl.n_inst, ptrs, len(qidx), p, d, float(t_ms), int(reading),
                                   int(max_iters), ttft, iters)
    if st != OK:
        raise OracleError(st, "estimate_matrix")
    del qs
    return ttft, iters


def trace_scenarios(wl, scenarios, n_threads: int, **kw):
    """``trace(wl, z, **kw)`` for each z in ``scenarios``, the scenarios on up to
    n_threads threads at once (each trace single-threaded inside).  Returns the
    results in the order of ``scenarios``."""
    if n_threads <= 1:
        return [trace(wl, scenario=z, **kw) for z in scenarios]
    with ThreadPoolExecutor(max_workers=n_threads) as ex:
        return list(ex.map(lambda z: trace(wl, scenario=z, **kw), scenarios))


LPS_POISSON = 0        # Eqs. 10 and 12
LPS_VARIABILITY = 1    # Eq. 13


def lps_wait(alpha, mu, k, mode=LPS_POISSON, ca2=1.0, cs2=1.0):
    """Expected LPS queueing delay (ms) of an instance; NaN outside the model."""
    return float(lib().orc_lps_wait(float(alpha), float(mu), int(k), int(mode), float(ca2),
                                    float(cs2)))


def lps_ttft(alpha, mu, k, theta, t_dec, p, mode=LPS_POISSON, ca2=1.0, cs2=1.0):
    """Average-case TTFT estimate (Eq. 11), ms."""
    return float(lib().orc_lps_ttft(float(alpha), float(mu), int(k), int(mode), float(ca2),
                                    float(cs2), float(theta), float(t_dec), int(p)))


def lps_matrix(prm, p, mode=LPS_POISSON, n_threads=1):
    """LPS TTFT of every query (prompts p) at every instance; prm holds per-instance
    arrays alpha, mu, k, ca2, cs2, theta, t_dec.  Returns [Q][I].  With n_threads > 1
    the rows are split into chunks computed on threads of their own (each row is
    independent; the same code runs per chunk)."""
    f = lambda k: np.ascontiguousarray(prm[k], np.float64)  # noqa: E731
    I = len(prm["alpha"])
    p = _i32(p)
    out = np.zeros((len(p), I))
    args = (f("alpha"), f("mu"), _i32(prm["k"]), f("ca2"), f("cs2"), f("theta"), f("t_dec"))

    def rows(lo, hi):
        if hi > lo:
            blk = np.zeros((hi - lo, I))
            lib().orc_lps_matrix(I, *args, int(mode), hi - lo, np.ascontiguousarray(p[lo:hi]),
                                 blk)
            out[lo:hi] = blk

    if n_threads <= 1:
        rows(0, len(p))
    else:
        cuts = np.linspace(0, len(p), n_threads + 1).astype(int)
        with ThreadPoolExecutor(max_workers=n_threads) as ex:
            list(ex.map(lambda t: rows(cuts[t], cuts[t + 1]), range(n_threads)))
    return out
