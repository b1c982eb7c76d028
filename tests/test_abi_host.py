"""CPU-side checks of the C ABI library and the workload generator (no GPU calls)."""

import ctypes
import os
import re
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lar.h")
LIB = os.path.join(ROOT, "paper_2607_18253_amd", "liblar.so")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lar_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("lar_create", "lar_destroy", "lar_load_state", "lar_estimate_ttft", "lar_route",
              "lar_commit", "lar_route_trace", "lar_stats", "lar_read_state", "lar_sync",
              "lar_error_string"):
        assert n in names


def test_library_exports_every_declared_symbol():
    if not os.path.exists(LIB):
        pytest.skip("liblar.so not built (run __graft_entry__.build())")
    lib = ctypes.CDLL(LIB)
    for n in _declared():
        assert hasattr(lib, n), n
    from paper_2607_18253_amd.lar import EXPORTED
    assert sorted(EXPORTED) == _declared()


def test_null_arguments_rejected_without_gpu():
    if not os.path.exists(LIB):
        pytest.skip("liblar.so not built")
    lib = ctypes.CDLL(LIB)
    lib.lar_create.restype = ctypes.c_int32
    assert lib.lar_create(None, None) == -1
    out = ctypes.c_void_p(1)
    assert lib.lar_create(ctypes.byref(out), None) == -1
    assert out.value is None
    lib.lar_sync.restype = ctypes.c_int32
    assert lib.lar_sync(None) == -1
    lib.lar_destroy.restype = ctypes.c_int32
    assert lib.lar_destroy(None) == 0
    # every other entry point rejects a null context before touching the device
    for name, n_args in (("lar_route", 11), ("lar_route_constrained", 11),
                         ("lar_ttft_targets", 6), ("lar_route_trace_constrained", 15),
                         ("lar_route_trace", 15), ("lar_ontime_utility", 10), ("lar_stats", 9),
                         ("lar_reload_state", 1), ("lar_route_step", 14),
                         ("lar_set_scheduler", 2)):
        f = getattr(lib, name)
        f.restype = ctypes.c_int32
        args = [None] * n_args
        if name == "lar_route_trace_constrained":
            f.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                          ctypes.c_void_p, ctypes.c_double] + [ctypes.c_void_p] * 3 + \
                         [ctypes.c_int32] + [ctypes.c_void_p] * 5
            args = [None, 1, None, None, None, 0.0, None, None, None, 1, None, None, None, None,
                    None]
        if name == "lar_route_step":
            f.argtypes = [ctypes.c_void_p] * 7 + [ctypes.c_int32] + [ctypes.c_void_p] * 6
            args = [None] * 7 + [1] + [None] * 6
        if name == "lar_route_trace":
            f.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                          ctypes.c_void_p, ctypes.c_double] + [ctypes.c_void_p] * 2 + \
                         [ctypes.c_int32] + [ctypes.c_void_p] * 6
            args = [None, 1, None, None, None, 0.0, None, None, 1, None, None, None, None, None,
                    None]
        assert f(*args) == -1, name


# ------------------------------------------------------------------ generator
def _check_state(wl):
    for j in range(wl.n_inst):
        rp, rd, cx = wl.instance_requests(j)
        assert np.all(rp >= 0) and np.all(rd >= 1) and np.all(cx >= 0)
        assert not np.any((rp == 0) & (cx == 0))
        run = cx > 0
        if run.any() and (~run).any():
            assert np.argmin(run) >= np.sum(run) - 0  # running block first
            assert np.all(run[:np.sum(run)])
        assert np.sum(run) <= wl.max_seqs[j]


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5", "c6", "c7"])
def test_generator_shapes_and_invariants(name):
    from workloads import make_workload
    kw = dict(n_q=500) if name != "c3" else {}
    if name in ("c3", "c4"):
        kw["n_inst"] = 16
    wl = make_workload(name, **kw)
    _check_state(wl)
    cfg = wl.meta
    assert wl.n_scen == len(cfg["weights"])
    assert wl.acc.shape == wl.cost.shape == (wl.n_q, wl.n_cols)
    assert np.all(wl.col < wl.n_cols)
    assert np.all(np.diff(wl.q_t_ms) >= 0)
    assert wl.q_prefill.min() >= 1 and wl.q_prefill.max() <= wl.max_prompt
    R = cfg["resident"]
    n_dec = min(R // 2, cfg["max_seqs"] - 1)
    rp, rd, cx = wl.instance_requests(0)
    assert len(rp) == R
    assert np.sum((rp == 0) & (cx > 0)) == n_dec
    assert np.sum((rp > 0) & (cx > 0)) == 1
    assert np.sum(cx == 0) == R - n_dec - 1


def test_generator_c7_fits_its_limits():
    from workloads import make_workload
    wl = make_workload("c7", n_q=500)
    for j in range(wl.n_inst):
        H, K, S, X = (int(v) for v in wl.sched[j])
        rp, rd, cx = wl.instance_requests(j)
        assert np.all(rp + cx < X)
        assert sum(-(-int(c) // S) for c in cx if c > 0) <= K
        assert K * S >= X and S & (S - 1) == 0
    assert wl.q_prefill.max() < int(wl.sched[0][3])


def test_generator_is_deterministic():
    from workloads import make_workload
    a = make_workload("c2", n_q=100)
    b = make_workload("c2", n_q=100)
    for f in ("rem_prefill", "rem_decode", "context", "q_prefill", "q_decode", "q_t_ms", "acc",
              "cost"):
        assert np.array_equal(getattr(a, f), getattr(b, f))


def test_c5_weight_grid():
    from workloads import make_workload
    wl = make_workload("c5", n_q=10)
    vals = [10.0 ** (-2 + 3 * k / 7) for k in range(8)]
    assert wl.n_scen == 64
    for s in range(64):
        assert wl.w_cost[s] == vals[s // 8]
        assert wl.w_lat_ms[s] == vals[s % 8] / 1000.0
    assert abs(vals[0] - 0.01) < 1e-15 and abs(vals[7] - 10.0) < 1e-12


@pytest.mark.parametrize("seed", range(20))
def test_tiny_generator_states_valid(seed):
    from workloads import make_tiny_workload
    _check_state(make_tiny_workload(seed))


def test_missing_library_fails_loudly():
    """The binding raises when the HIP library is absent: there is no CPU fallback."""
    import subprocess
    code = ("import paper_2607_18253_amd.lar as L\n"
            "try:\n    L.load_library('/nonexistent/liblar.so')\n"
            "except RuntimeError as e:\n    print('RAISED', e)\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True,
                       timeout=300)
    assert "RAISED" in r.stdout and "not built" in r.stdout, r.stdout + r.stderr


def test_product_package_never_touches_the_oracle():
    """No module of the package (binding, build, C/HIP sources) imports, links or names
    the oracle: the oracle is test infrastructure only."""
    pkg = os.path.join(ROOT, "paper_2607_18253_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert "oracle" not in text.lower(), os.path.join(dirpath, f)
