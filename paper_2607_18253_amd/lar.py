"""Python binding of ``liblar.so`` (the C ABI in include/lar.h): argument
marshalling only.  Device arrays are torch tensors on the GPU; snapshots go in and
out as host numpy arrays.  Every step of the estimator and router runs in the HIP
kernels behind the C ABI; there is no fallback path -- a missing library raises.
"""

from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liblar.so")

LAR_OK, LAR_E_ARG, LAR_E_STATE, LAR_E_CAPACITY, LAR_E_ITER, LAR_E_HIP, LAR_E_SYNC = (
    0, -1, -2, -3, -4, -5, -6)
FIRST_TOKEN_DECODE_BATCH, FIRST_TOKEN_PREFILL_BATCH = 0, 1

EXPORTED = ("lar_create", "lar_destroy", "lar_error_string", "lar_load_state", "lar_reload_state",
            "lar_estimate_ttft", "lar_route", "lar_route_constrained", "lar_ttft_targets",
            "lar_commit", "lar_route_step", "lar_route_trace", "lar_route_trace_constrained",
            "lar_stats", "lar_set_scheduler",
            "lar_ontime_utility", "lar_read_state", "lar_sync", "lar_trace_work", "lar_board_create",
            "lar_board_destroy", "lar_board_publish", "lar_board_collect",
            "lar_whatif_noalloc", "lar_noalloc_error_string", "lar_estimate_lps")
LPS_POISSON, LPS_VARIABILITY = 0, 1


class LarError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"lar error {code}: {msg}")
        self.code = code


class Config(C.Structure):
    _fields_ = [("n_scen", C.c_int32), ("n_inst", C.c_int32), ("max_seqs_cap", C.c_int32),
                ("queue_cap", C.c_int32), ("max_prompt", C.c_int32), ("flags", C.c_int32),
                ("max_iters", C.c_int64), ("stream", C.c_void_p)]


class SchedLimits(C.Structure):
    _fields_ = [("chunk_cap", C.c_int32), ("kv_blocks", C.c_int32), ("block_size", C.c_int32),
                ("max_ctx", C.c_int32)]


class WhatifConfig(C.Structure):
    _fields_ = [("n_inst", C.c_int32), ("max_seqs_cap", C.c_int32), ("max_resident", C.c_int32),
                ("max_prompt", C.c_int32), ("n_cols", C.c_int32), ("flags", C.c_int32),
                ("max_iters", C.c_int64), ("stream", C.c_void_p)]


class LpsParams(C.Structure):
    _fields_ = [("arrival_rate", C.c_double), ("service_rate", C.c_double),
                ("prefill_rate", C.c_double), ("decode_ms", C.c_double), ("ca2", C.c_double),
                ("cs2", C.c_double), ("k", C.c_int32), ("reserved", C.c_int32)]


LPS_DTYPE = np.dtype([("arrival_rate", "<f8"), ("service_rate", "<f8"), ("prefill_rate", "<f8"),
                      ("decode_ms", "<f8"), ("ca2", "<f8"), ("cs2", "<f8"), ("k", "<i4"),
                      ("reserved", "<i4")])


class InstanceParams(C.Structure):
    _fields_ = [("a", C.c_double), ("b", C.c_double), ("c", C.c_double), ("d", C.c_double),
                ("e", C.c_double), ("token_budget", C.c_int32), ("max_seqs", C.c_int32),
                ("col", C.c_int32), ("reserved", C.c_int32)]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load liblar.so (after torch, so both share torch's HIP runtime)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run __graft_entry__.build() "
                           "or python paper_2607_18253_amd/build.py")
    import torch  # noqa: F401  -- maps torch's HIP runtime before the library's
    L = C.CDLL(path)
    vp, i32, i64, dbl = C.c_void_p, C.c_int32, C.c_int64, C.c_double
    L.lar_create.restype = i32
    L.lar_create.argtypes = [C.POINTER(vp), C.POINTER(Config)]
    L.lar_destroy.restype = i32
    L.lar_destroy.argtypes = [vp]
    L.lar_error_string.restype = C.c_char_p
    L.lar_error_string.argtypes = [vp]
    L.lar_load_state.restype = i32
    L.lar_load_state.argtypes = [vp, C.POINTER(InstanceParams), vp, vp, vp, vp, vp]
    L.lar_reload_state.restype = i32
    L.lar_reload_state.argtypes = [vp]
    L.lar_set_scheduler.restype = i32
    L.lar_set_scheduler.argtypes = [vp, vp]
    L.lar_estimate_ttft.restype = i32
    L.lar_estimate_ttft.argtypes = [vp, i32, vp, dbl, vp, vp]
    L.lar_route.restype = i32
    L.lar_route.argtypes = [vp, i32, vp, vp, vp, i32, vp, vp, vp, vp, vp]
    L.lar_commit.restype = i32
    L.lar_commit.argtypes = [vp, vp, i32, i32, dbl]
    L.lar_route_step.restype = i32
    L.lar_route_step.argtypes = [vp, vp, vp, vp, vp, vp, vp, i32, vp, vp, vp, vp, vp, vp]
    L.lar_route_trace.restype = i32
    L.lar_route_trace.argtypes = [vp, i32, vp, vp, vp, dbl, vp, vp, i32, vp, vp, vp, vp, vp, vp]
    L.lar_route_constrained.restype = i32
    L.lar_route_constrained.argtypes = [vp, i32, vp, vp, vp, vp, i32, vp, vp, vp, vp]
    L.lar_ttft_targets.restype = i32
    L.lar_ttft_targets.argtypes = [vp, i32, vp, vp, vp, vp]
    L.lar_route_trace_constrained.restype = i32
    L.lar_route_trace_constrained.argtypes = [vp, i32, vp, vp, vp, dbl, vp, vp, vp, i32, vp, vp,
                                              vp, vp, vp]
    L.lar_ontime_utility.restype = i32
    L.lar_ontime_utility.argtypes = [vp, i32, vp, vp, vp, vp, vp, i32, vp, vp]
    L.lar_trace_work.restype = i32
    L.lar_trace_work.argtypes = [vp, vp]
    L.lar_board_create.restype = i32
    L.lar_board_create.argtypes = [C.POINTER(vp), i32, i32]
    L.lar_board_destroy.restype = i32
    L.lar_board_destroy.argtypes = [vp]
    L.lar_board_publish.restype = i32
    L.lar_board_publish.argtypes = [vp, i32, i32, vp, vp, vp, dbl]
    L.lar_board_collect.restype = i32
    L.lar_board_collect.argtypes = [vp, vp, vp, vp, vp, vp, i64, vp, vp]
    L.lar_stats.restype = i32
    L.lar_stats.argtypes = [vp, i32, vp, vp, vp, vp, i32, vp, vp]
    L.lar_read_state.restype = i32
    L.lar_read_state.argtypes = [vp, i32, vp, vp, vp, vp, vp, vp, i64, C.POINTER(i64)]
    L.lar_sync.restype = i32
    L.lar_sync.argtypes = [vp]
    L.lar_estimate_lps.restype = i32
    L.lar_estimate_lps.argtypes = [vp, vp, i32, i32, vp, vp]
    L.lar_whatif_noalloc.restype = i32
    L.lar_whatif_noalloc.argtypes = [C.POINTER(WhatifConfig), vp, vp, vp, vp, vp, vp, i32, vp, dbl,
                                     vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    L.lar_noalloc_error_string.restype = C.c_char_p
    L.lar_noalloc_error_string.argtypes = []
    _lib = L
    return L


def _dev(t, dtype, name, numel=None):
    """Device pointer of a contiguous GPU tensor of the given torch dtype (None -> NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} < {numel} elements")
    return t.data_ptr()


def _host(a, dtype):
    return np.ascontiguousarray(np.asarray(a, dtype=dtype))


class LarContext:
    """One estimator/router context: Z scenarios x I instances of device state."""

    def __init__(self, n_scen: int, n_inst: int, *, max_seqs_cap: int, queue_cap: int,
                 max_prompt: int, flags: int = FIRST_TOKEN_DECODE_BATCH,
                 max_iters: int = 10_000_000, stream=None):
        import torch
        self._torch = torch
        self._L = load_library()
        if stream is None:
            stream = torch.cuda.current_stream()
        self.stream = stream
        cfg = Config(int(n_scen), int(n_inst), int(max_seqs_cap), int(queue_cap),
                     int(max_prompt), int(flags), int(max_iters), C.c_void_p(stream.cuda_stream))
        h = C.c_void_p()
        st = self._L.lar_create(C.byref(h), C.byref(cfg))
        if st != LAR_OK:
            raise LarError(st, "lar_create failed")
        self._h = h
        self.Z, self.I = int(n_scen), int(n_inst)
        self.n_cols = None

    # ------------------------------------------------------------------ plumbing
    def _check(self, st: int):
        if st != LAR_OK:
            msg = self._L.lar_error_string(self._h)
            raise LarError(st, msg.decode() if msg else "")

    def close(self):
        if getattr(self, "_h", None):
            self._L.lar_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    # ------------------------------------------------------------------ calls
    def load_state(self, *, a, b, c, d, e, budget, max_seqs, col, offsets, rem_prefill,
                   rem_decode, context, clock_ms):
        I = self.I
        params = (InstanceParams * I)()
        for j in range(I):
            params[j] = InstanceParams(float(a[j]), float(b[j]), float(c[j]), float(d[j]),
                                       float(e[j]), int(budget[j]), int(max_seqs[j]),
                                       int(col[j]), 0)
        off = _host(offsets, np.int32)
        rp, rd, cx = _host(rem_prefill, np.int32), _host(rem_decode, np.int32), _host(context, np.int32)
        clk = _host(clock_ms, np.float64)
        if off.shape[0] != I + 1 or clk.shape[0] != I:
            raise ValueError("offsets must have I+1 entries and clock_ms I entries")
        n = int(off[-1])
        if min(rp.shape[0], rd.shape[0], cx.shape[0]) < n:
            raise ValueError("request arrays shorter than offsets[I]")
        self._check(self._L.lar_load_state(self._h, params, off.ctypes.data, rp.ctypes.data,
                                           rd.ctypes.data, cx.ctypes.data, clk.ctypes.data))

    def reload_state(self):
        self._check(self._L.lar_reload_state(self._h))

    def set_scheduler(self, limits):
        """Scheduler limits per instance, [I][4] (chunk cap, KV blocks, block size,
        context limit; 0 = none), or None for the default scheduler.  A load_state
        must follow."""
        if limits is None:
            self._check(self._L.lar_set_scheduler(self._h, None))
            return
        lim = np.asarray(limits, np.int32).reshape(self.I, 4)
        arr = (SchedLimits * self.I)(*[SchedLimits(*(int(v) for v in lim[j]))
                                       for j in range(self.I)])
        self._check(self._L.lar_set_scheduler(self._h, C.cast(arr, C.c_void_p)))

    def load_workload(self, wl):
        self.load_state(a=wl.a, b=wl.b, c=wl.c, d=wl.d, e=wl.e, budget=wl.budget,
                        max_seqs=wl.max_seqs, col=wl.col, offsets=wl.offsets,
                        rem_prefill=wl.rem_prefill, rem_decode=wl.rem_decode,
                        context=wl.context, clock_ms=wl.clock_ms)

    def estimate(self, q_prefill, t_ms: float, ttft=None, iters=None, want_iters=True):
        torch = self._torch
        Q = int(q_prefill.numel())
        dev = q_prefill.device
        if ttft is None:
            ttft = torch.empty((self.Z, Q, self.I), dtype=torch.float64, device=dev)
        if iters is None and want_iters:
            iters = torch.empty((self.Z, Q, self.I), dtype=torch.int32, device=dev)
        n = self.Z * Q * self.I
        self._check(self._L.lar_estimate_ttft(
            self._h, Q, _dev(q_prefill, torch.int32, "q_prefill"), float(t_ms),
            _dev(ttft, torch.float64, "ttft", n), _dev(iters, torch.int32, "iters", n)))
        return ttft, iters

    def estimate_lps(self, params, q_prefill, mode=LPS_POISSON, ttft=None):
        """Average-case LPS TTFT (lar_estimate_lps): params is a GPU uint8 tensor of
        Z*I lar_lps_params records (see lps_params_array), scenario-major; returns
        ttft [Z][Q][I]."""
        torch = self._torch
        Q = int(q_prefill.numel())
        if params.dtype != torch.uint8 or params.numel() != self.Z * self.I * LPS_DTYPE.itemsize:
            raise ValueError("params must hold Z*I lar_lps_params records")
        if ttft is None:
            ttft = torch.empty((self.Z, Q, self.I), dtype=torch.float64,
                               device=q_prefill.device)
        self._check(self._L.lar_estimate_lps(
            self._h, _dev(params, torch.uint8, "params"), int(mode), Q,
            _dev(q_prefill, torch.int32, "q_prefill"),
            _dev(ttft, torch.float64, "ttft", self.Z * Q * self.I)))
        return ttft

    def route(self, ttft, acc, cost, w_cost, w_lat, choice=None, chosen_ttft=None,
              utility=None):
        torch = self._torch
        Q = int(acc.shape[0])
        n_cols = int(acc.shape[1])
        dev = acc.device
        if choice is None:
            choice = torch.empty((self.Z, Q), dtype=torch.int32, device=dev)
        self._check(self._L.lar_route(
            self._h, Q, _dev(ttft, torch.float64, "ttft", self.Z * Q * self.I),
            _dev(acc, torch.float64, "acc", Q * n_cols), _dev(cost, torch.float64, "cost", Q * n_cols),
            n_cols, _dev(w_cost, torch.float64, "w_cost", self.Z),
            _dev(w_lat, torch.float64, "w_lat", self.Z), _dev(choice, torch.int32, "choice", self.Z * Q),
            _dev(chosen_ttft, torch.float64, "chosen_ttft", self.Z * Q),
            _dev(utility, torch.float64, "utility", self.Z * Q)))
        return choice

    def route_constrained(self, ttft, tau_ms, acc, cost, w_cost, choice=None, chosen_ttft=None,
                          utility=None):
        torch = self._torch
        Q = int(acc.shape[0])
        n_cols = int(acc.shape[1])
        if choice is None:
            choice = torch.empty((self.Z, Q), dtype=torch.int32, device=acc.device)
        self._check(self._L.lar_route_constrained(
            self._h, Q, _dev(ttft, torch.float64, "ttft", self.Z * Q * self.I),
            _dev(tau_ms, torch.float64, "tau_ms", Q),
            _dev(acc, torch.float64, "acc", Q * n_cols), _dev(cost, torch.float64, "cost", Q * n_cols),
            n_cols, _dev(w_cost, torch.float64, "w_cost", self.Z),
            _dev(choice, torch.int32, "choice", self.Z * Q),
            _dev(chosen_ttft, torch.float64, "chosen_ttft", self.Z * Q),
            _dev(utility, torch.float64, "utility", self.Z * Q)))
        return choice

    def ttft_targets(self, q_prefill, u_ms, v, out=None):
        torch = self._torch
        n = int(q_prefill.numel())
        if out is None:
            out = torch.empty(n, dtype=torch.float64, device=q_prefill.device)
        self._check(self._L.lar_ttft_targets(
            self._h, n, _dev(q_prefill, torch.int32, "q_prefill", n),
            _dev(u_ms, torch.float64, "u_ms", n), _dev(v, torch.float64, "v", n),
            _dev(out, torch.float64, "tau_ms", n)))
        return out

    def commit(self, choice, q_prefill: int, q_decode: int, t_next_ms: float):
        torch = self._torch
        self._check(self._L.lar_commit(self._h, _dev(choice, torch.int32, "choice", self.Z),
                                       int(q_prefill), int(q_decode), float(t_next_ms)))

    def advance(self, t_ms: float):
        self.commit(None, 1, 1, t_ms)

    def route_step(self, q_prefill, q_decode, t_ms, t_next_ms, acc_row, cost_row, w_cost,
                   w_lat=None, tau_ms=None, choice=None, chosen_ttft=None, utility=None):
        """One routing step (estimate, route, commit) with the query's values in device
        tensors ([1] each; acc_row / cost_row [n_cols]), read when the step runs:
        capturable in a CUDA/HIP graph and replayed per query."""
        torch = self._torch
        n_cols = int(acc_row.numel())
        if choice is None:
            choice = torch.empty(self.Z, dtype=torch.int32, device=acc_row.device)
        self._check(self._L.lar_route_step(
            self._h, _dev(q_prefill, torch.int32, "q_prefill", 1),
            _dev(q_decode, torch.int32, "q_decode", 1), _dev(t_ms, torch.float64, "t_ms", 1),
            _dev(t_next_ms, torch.float64, "t_next_ms", 1),
            _dev(acc_row, torch.float64, "acc_row", n_cols),
            _dev(cost_row, torch.float64, "cost_row", n_cols), n_cols,
            _dev(w_cost, torch.float64, "w_cost", self.Z), _dev(w_lat, torch.float64, "w_lat", self.Z),
            _dev(tau_ms, torch.float64, "tau_ms", 1), _dev(choice, torch.int32, "choice", self.Z),
            _dev(chosen_ttft, torch.float64, "chosen_ttft", self.Z),
            _dev(utility, torch.float64, "utility", self.Z)))
        return choice

    def route_trace(self, q_prefill, q_decode, q_t_ms, t_after_ms, acc, cost, w_cost, w_lat,
                    choice=None, chosen_ttft=None, utility=None, realized=None):
        torch = self._torch
        N = int(q_prefill.numel())
        n_cols = int(acc.shape[1])
        dev = q_prefill.device
        if choice is None:
            choice = torch.empty((self.Z, N), dtype=torch.int32, device=dev)
        self._check(self._L.lar_route_trace(
            self._h, N, _dev(q_prefill, torch.int32, "q_prefill"),
            _dev(q_decode, torch.int32, "q_decode", N), _dev(q_t_ms, torch.float64, "q_t_ms", N),
            float(t_after_ms), _dev(acc, torch.float64, "acc", N * n_cols),
            _dev(cost, torch.float64, "cost", N * n_cols), n_cols,
            _dev(w_cost, torch.float64, "w_cost", self.Z), _dev(w_lat, torch.float64, "w_lat", self.Z),
            _dev(choice, torch.int32, "choice", self.Z * N),
            _dev(chosen_ttft, torch.float64, "chosen_ttft", self.Z * N),
            _dev(utility, torch.float64, "utility", self.Z * N),
            _dev(realized, torch.float64, "realized", self.Z * N)))
        return choice

    def route_trace_constrained(self, q_prefill, q_decode, q_t_ms, t_after_ms, tau_ms, acc, cost,
                                w_cost, choice=None, chosen_ttft=None, utility=None,
                                realized=None):
        torch = self._torch
        N = int(q_prefill.numel())
        n_cols = int(acc.shape[1])
        if choice is None:
            choice = torch.empty((self.Z, N), dtype=torch.int32, device=q_prefill.device)
        self._check(self._L.lar_route_trace_constrained(
            self._h, N, _dev(q_prefill, torch.int32, "q_prefill"),
            _dev(q_decode, torch.int32, "q_decode", N), _dev(q_t_ms, torch.float64, "q_t_ms", N),
            float(t_after_ms), _dev(tau_ms, torch.float64, "tau_ms", N),
            _dev(acc, torch.float64, "acc", N * n_cols),
            _dev(cost, torch.float64, "cost", N * n_cols), n_cols,
            _dev(w_cost, torch.float64, "w_cost", self.Z),
            _dev(choice, torch.int32, "choice", self.Z * N),
            _dev(chosen_ttft, torch.float64, "chosen_ttft", self.Z * N),
            _dev(utility, torch.float64, "utility", self.Z * N),
            _dev(realized, torch.float64, "realized", self.Z * N)))
        return choice

    def ontime_utility(self, choice, realized, tau_ms, acc, cost, w_cost, out=None):
        torch = self._torch
        N = int(choice.shape[-1])
        n_cols = int(acc.shape[1])
        if out is None:
            out = torch.empty(self.Z, dtype=torch.float64, device=choice.device)
        self._check(self._L.lar_ontime_utility(
            self._h, N, _dev(choice, torch.int32, "choice", self.Z * N),
            _dev(realized, torch.float64, "realized", self.Z * N),
            _dev(tau_ms, torch.float64, "tau_ms", N),
            _dev(acc, torch.float64, "acc", N * n_cols), _dev(cost, torch.float64, "cost", N * n_cols),
            n_cols, _dev(w_cost, torch.float64, "w_cost", self.Z),
            _dev(out, torch.float64, "out", self.Z)))
        return out

    def stats(self, choice, chosen_ttft, acc, cost, w_cost, out=None):
        torch = self._torch
        N = int(choice.shape[-1])
        n_cols = int(acc.shape[1])
        if out is None:
            out = torch.empty((self.Z, 5), dtype=torch.float64, device=choice.device)
        self._check(self._L.lar_stats(
            self._h, N, _dev(choice, torch.int32, "choice", self.Z * N),
            _dev(chosen_ttft, torch.float64, "chosen_ttft", self.Z * N),
            _dev(acc, torch.float64, "acc", N * n_cols), _dev(cost, torch.float64, "cost", N * n_cols),
            n_cols, _dev(w_cost, torch.float64, "w_cost", self.Z),
            _dev(out, torch.float64, "stats", self.Z * 5)))
        return out

    def trace_work(self):
        """Per-scenario batches behind the last trace's estimates (synchronises)."""
        out = np.zeros(self.Z, np.int64)
        self._check(self._L.lar_trace_work(self._h, out.ctypes.data))
        return out

    def sync(self):
        self._check(self._L.lar_sync(self._h))

    def status(self) -> int:
        """Synchronise and return the sticky status code without raising."""
        return int(self._L.lar_sync(self._h))

    def read_state(self, scen: int = 0, cap: int | None = None):
        I = self.I
        off = np.zeros(I + 1, np.int32)
        clk = np.zeros(I)
        its = np.zeros(I, np.int64)
        n_total = C.c_int64(0)
        cap = 0 if cap is None else int(cap)
        rp = np.zeros(max(cap, 1), np.int32)
        rd = np.zeros(max(cap, 1), np.int32)
        cx = np.zeros(max(cap, 1), np.int32)
        st = self._L.lar_read_state(self._h, int(scen), off.ctypes.data, rp.ctypes.data,
                                    rd.ctypes.data, cx.ctypes.data, clk.ctypes.data,
                                    its.ctypes.data, cap, C.byref(n_total))
        if st == LAR_E_CAPACITY and n_total.value > cap:
            return self.read_state(scen, int(n_total.value))
        self._check(st)
        n = int(n_total.value)
        return dict(offsets=off, rem_prefill=rp[:n], rem_decode=rd[:n], context=cx[:n],
                    clock_ms=clk, iterations=its)


def context_for(wl, *, flags=FIRST_TOKEN_DECODE_BATCH, max_iters=10_000_000, stream=None,
                queue_cap=None, max_seqs_cap=None) -> LarContext:
    """A context sized for workload ``wl`` with its snapshot loaded (max_seqs_cap
    defaults to the largest M of the pool), under the workload's scheduler limits
    when it has them."""
    mcap = int(np.max(wl.max_seqs)) if max_seqs_cap is None else int(max_seqs_cap)
    ctx = LarContext(wl.n_scen, wl.n_inst, max_seqs_cap=mcap,
                     queue_cap=int(wl.queue_cap if queue_cap is None else queue_cap),
                     max_prompt=int(wl.max_prompt), flags=flags, max_iters=max_iters,
                     stream=stream)
    if getattr(wl, "sched", None) is not None:
        ctx.set_scheduler(wl.sched)
    ctx.load_workload(wl)
    return ctx


class SnapshotBoard:
    """Host-side snapshot board (seqlock per instance): publishers replace their
    instance's snapshot, the router collects the latest complete copies in the
    layout of LarContext.load_state."""

    def __init__(self, n_inst: int, max_requests: int, lib_path: str = LIB_PATH):
        self._L = load_library(lib_path)
        self.I, self.max_req = int(n_inst), int(max_requests)
        h = C.c_void_p()
        st = self._L.lar_board_create(C.byref(h), self.I, self.max_req)
        if st != LAR_OK:
            raise LarError(st, "lar_board_create failed")
        self._h = h

    def publish(self, inst: int, rem_prefill, rem_decode, context, clock_ms: float):
        rp = np.ascontiguousarray(rem_prefill, np.int32)
        rd = np.ascontiguousarray(rem_decode, np.int32)
        cx = np.ascontiguousarray(context, np.int32)
        st = self._L.lar_board_publish(self._h, int(inst), len(rp), rp.ctypes.data,
                                       rd.ctypes.data, cx.ctypes.data, float(clock_ms))
        if st != LAR_OK:
            raise LarError(st, "lar_board_publish failed")

    def collect(self, cap: int | None = None):
        cap = self.I * self.max_req if cap is None else int(cap)
        off = np.zeros(self.I + 1, np.int32)
        rp, rd, cx = (np.zeros(max(cap, 1), np.int32) for _ in range(3))
        clk = np.zeros(self.I)
        fresh = np.zeros(self.I, np.int32)
        ver = np.zeros(self.I, np.uint64)
        st = self._L.lar_board_collect(self._h, off.ctypes.data, rp.ctypes.data, rd.ctypes.data,
                                       cx.ctypes.data, clk.ctypes.data, cap, fresh.ctypes.data,
                                       ver.ctypes.data)
        if st != LAR_OK:
            raise LarError(st, "lar_board_collect failed")
        n = int(off[-1])
        return dict(offsets=off, rem_prefill=rp[:n], rem_decode=rd[:n], context=cx[:n],
                    clock_ms=clk, fresh=fresh, versions=ver)

    def close(self):
        if self._h:
            self._L.lar_board_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def params_array(a, b, c, d, e, budget, max_seqs, col):
    """Instance parameters as a numpy array of lar_instance_params records (to copy
    into device memory for lar_whatif_noalloc)."""
    I = len(a)
    rec = np.zeros(I, dtype=np.dtype([("a", "<f8"), ("b", "<f8"), ("c", "<f8"), ("d", "<f8"),
                                      ("e", "<f8"), ("token_budget", "<i4"),
                                      ("max_seqs", "<i4"), ("col", "<i4"), ("reserved", "<i4")]))
    rec["a"], rec["b"], rec["c"], rec["d"], rec["e"] = a, b, c, d, e
    rec["token_budget"], rec["max_seqs"], rec["col"] = budget, max_seqs, col
    assert rec.dtype.itemsize == C.sizeof(InstanceParams)
    return rec


def whatif_noalloc(params, offsets, rem_prefill, rem_decode, context, clock_ms, q_prefill,
                   t_ms, acc, cost, w_cost, w_lat, ttft, choice, status, *, max_seqs_cap,
                   max_resident, max_prompt, flags=FIRST_TOKEN_DECODE_BATCH,
                   max_iters=10_000_000, iters=None, chosen_ttft=None, utility=None,
                   stream=None):
    """lar_whatif_noalloc: every argument array is a GPU tensor the caller allocated
    (params: uint8 tensor holding lar_instance_params records, see params_array);
    writes ttft [Q][I], choice [Q], status [1] (and iters, chosen_ttft, utility
    when given).  Enqueues on the current stream (or ``stream``) and returns."""
    import torch
    L = load_library()
    I = int(offsets.numel()) - 1
    Q = int(q_prefill.numel())
    n_cols = int(acc.shape[1]) if acc.dim() == 2 else 1
    if stream is None:
        stream = torch.cuda.current_stream().cuda_stream
    cfg = WhatifConfig(I, int(max_seqs_cap), int(max_resident), int(max_prompt), n_cols,
                       int(flags), int(max_iters), C.c_void_p(stream))
    if params.dtype != torch.uint8 or params.numel() != I * C.sizeof(InstanceParams):
        raise ValueError("params must hold one lar_instance_params record per instance")
    st = L.lar_whatif_noalloc(
        C.byref(cfg), _dev(params, torch.uint8, "params"), _dev(offsets, torch.int32, "offsets"),
        _dev(rem_prefill, torch.int32, "rem_prefill"), _dev(rem_decode, torch.int32, "rem_decode"),
        _dev(context, torch.int32, "context"), _dev(clock_ms, torch.float64, "clock_ms", I), Q,
        _dev(q_prefill, torch.int32, "q_prefill"), float(t_ms),
        _dev(acc, torch.float64, "acc", Q * n_cols), _dev(cost, torch.float64, "cost", Q * n_cols),
        _dev(w_cost, torch.float64, "w_cost", 1), _dev(w_lat, torch.float64, "w_lat", 1),
        _dev(ttft, torch.float64, "ttft", Q * I),
        _dev(iters, torch.int32, "iters", Q * I) if iters is not None else None,
        _dev(choice, torch.int32, "choice", Q),
        _dev(chosen_ttft, torch.float64, "chosen_ttft", Q) if chosen_ttft is not None else None,
        _dev(utility, torch.float64, "utility", Q) if utility is not None else None,
        _dev(status, torch.int32, "status", 1))
    if st != LAR_OK:
        raise LarError(st, L.lar_noalloc_error_string().decode())


def lps_params_array(arrival_rate, service_rate, prefill_rate, decode_ms, k, ca2=None, cs2=None):
    """LPS parameters as a numpy array of lar_lps_params records (rates per ms, times
    in ms); copy its bytes to the GPU for LarContext.estimate_lps."""
    n = len(arrival_rate)
    rec = np.zeros(n, dtype=LPS_DTYPE)
    rec["arrival_rate"], rec["service_rate"] = arrival_rate, service_rate
    rec["prefill_rate"], rec["decode_ms"], rec["k"] = prefill_rate, decode_ms, k
    rec["ca2"] = 1.0 if ca2 is None else ca2
    rec["cs2"] = 1.0 if cs2 is None else cs2
    assert rec.dtype.itemsize == C.sizeof(LpsParams)
    return rec
