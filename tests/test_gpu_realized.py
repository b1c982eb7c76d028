"""GPU parity of the realised TTFT that a trace reports for each query (the replay's
first-token time minus the arrival; Fig. 2 sets the estimates against measured
TTFTs, and Eq. 4 counts it), against the oracle, bit for bit, with the choices, the
chosen estimates and the final state unchanged by the tracking."""

from __future__ import annotations

import os
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
from gpu_util import T, assert_state_equal, bits, gpu_trace, gpu_trace_realized  # noqa: E402
from oracle import oracle as O  # noqa: E402
from paper_2607_18253_amd import context_for  # noqa: E402
from workloads import make_tiny_workload, make_workload  # noqa: E402


def _check(wl, got, scenarios, *, reading=0, tau=None, state=(0,), queue_cap=None):
    choice, chosen, real, ctx = got
    refs = {}
    for z in scenarios:
        ref = O.trace(wl, scenario=z, n_q=choice.shape[1], reading=reading, tau=tau,
                      queue_cap=queue_cap, final_state=z in state)
        np.testing.assert_array_equal(choice[z], ref.choice, err_msg=f"scenario {z}")
        np.testing.assert_array_equal(bits(chosen[z]), bits(ref.ttft_chosen))
        np.testing.assert_array_equal(bits(real[z]), bits(ref.realized),
                                      err_msg=f"realised, scenario {z}")
        if z in state:
            assert_state_equal(ctx, z, ref)
        refs[z] = ref
    ctx.refs = refs
    return ctx


@pytest.mark.parametrize("seed", range(12))
@pytest.mark.parametrize("flags", [0, 1])
def test_realized_tiny_pools(seed, flags):
    wl = make_tiny_workload(500 + seed, n_inst=4, max_res=6, n_q=50, mean_gap_ms=1.0,
                            n_scen=3, dyadic=(seed % 2 == 0))
    got = gpu_trace_realized(wl, flags=flags, queue_cap=10 ** 4)
    _check(wl, got, range(3), reading=flags, state=(0, 1, 2), queue_cap=10 ** 4).close()


@pytest.mark.parametrize("seed", range(4))
def test_realized_tiny_pools_hbm_state_kernel(seed):
    """Prompts past 64 decode-only tail batches take the HBM-state trace kernel."""
    wl = make_tiny_workload(600 + seed, n_inst=5, max_res=8, n_q=30, prompt=(1, 300),
                            budget=(1, 6), max_seqs=(1, 3), mean_gap_ms=2.0, n_scen=2)
    got = gpu_trace_realized(wl, queue_cap=10 ** 4)
    _check(wl, got, range(2), state=(0, 1), queue_cap=10 ** 4).close()


@pytest.mark.parametrize("flags", [0, 1])
def test_realized_c1_full(flags):
    wl = make_workload("c1")
    got = gpu_trace_realized(wl, flags=flags)
    ctx = _check(wl, got, [0], reading=flags)
    ctx.close()
    real, chosen = got[2][0], got[1][0]
    assert (real >= chosen).all() and (real > chosen).any()


def test_realized_c2_prefix():
    """Config 2 (32 instances, clustered kernel over 8 workgroups), 3000 queries."""
    wl = make_workload("c2", n_q=3000)
    _check(wl, gpu_trace_realized(wl), [0]).close()


def test_realized_c2_prefix_hbm_state_kernel():
    """The same trace with 1024-slot queues, which take the HBM-state kernel."""
    wl = make_workload("c2", n_q=800)
    _check(wl, gpu_trace_realized(wl, max_seqs_cap=1024), [0]).close()


def test_realized_c4_prefix():
    """Config 4's instances (512 slots, 1024 resident requests, long prompts,
    context-dependent batch time), 8 of them so that queries share instances."""
    wl = make_workload("c4", n_q=12, n_inst=8)
    _check(wl, gpu_trace_realized(wl), [0]).close()


def test_realized_c5_scenarios_prefix():
    wl = make_workload("c5", n_q=200)
    _check(wl, gpu_trace_realized(wl), [0, 9, 27, 63], state=(0, 63)).close()


def test_realized_c6_bursty_prefix():
    wl = make_workload("c6", n_q=3000)
    _check(wl, gpu_trace_realized(wl), [0]).close()


def test_realized_constrained_c2_and_ontime():
    """Eq. 3 routing with the paper's targets; OnTimeUtility (Eq. 4) of the realised
    TTFTs against the oracle's."""
    wl = make_workload("c2", n_q=3000)
    tau = O.ttft_targets(wl.q_prefill, wl.tau_u_ms, wl.tau_v)
    got = gpu_trace_realized(wl, tau=tau)
    ctx = _check(wl, got, [0], tau=tau)
    choice, _, real, _ = got
    ref = ctx.refs[0]
    out = ctx.ontime_utility(T(choice, torch.int32), T(real, torch.float64),
                             T(tau, torch.float64), T(wl.acc, torch.float64),
                             T(wl.cost, torch.float64), T(wl.w_cost, torch.float64))
    ctx.sync()
    want = O.ontime_utility(ref.choice, ref.realized, tau, wl.acc, wl.cost, wl.col,
                            wl.w_cost[0])
    assert bits(out.cpu().numpy()[0]) == bits(want)
    ctx.close()


def test_realized_constrained_c5_scenarios_prefix():
    wl = make_workload("c5", n_q=60)
    tau = O.ttft_targets(wl.q_prefill, wl.tau_u_ms, wl.tau_v)
    _check(wl, gpu_trace_realized(wl, tau=tau), [0, 31, 63], tau=tau, state=(0,)).close()


def test_realized_tracking_leaves_trace_unchanged():
    """With and without tracking: identical choices, estimates and final state."""
    wl = make_workload("c2", n_q=1500)
    c0, t0, _, ctx0 = gpu_trace(wl)
    c1, t1, _, ctx1 = gpu_trace_realized(wl)
    np.testing.assert_array_equal(c0, c1)
    np.testing.assert_array_equal(bits(t0), bits(t1))
    s0, s1 = ctx0.read_state(0), ctx1.read_state(0)
    for k in ("offsets", "rem_prefill", "rem_decode", "context", "iterations"):
        np.testing.assert_array_equal(s0[k], s1[k], err_msg=k)
    np.testing.assert_array_equal(bits(s0["clock_ms"]), bits(s1["clock_ms"]))
    ctx0.close()
    ctx1.close()


@pytest.mark.parametrize("name", ["c2", "c7"])
def test_realized_split_calls(name):
    """One context, two trace calls: each call reports its own queries, and its end
    is the end of arrivals for the queries still waiting for a first token, so call
    1 equals the oracle's trace of the prefix and call 2 the whole trace's tail (c7:
    under scheduler limits)."""
    wl = make_workload(name, n_q=1200, n_inst=8)
    N, N1 = wl.n_q, 500
    ctx = context_for(wl)
    ctx.advance(float(wl.q_t_ms[0]))
    reals = []
    for lo, hi, t_after in ((0, N1, float(wl.q_t_ms[N1])), (N1, N, float(wl.q_t_ms[-1]))):
        r = torch.full((1, hi - lo), -1.0, dtype=torch.float64, device="cuda:0")
        ctx.route_trace(T(wl.q_prefill[lo:hi], torch.int32), T(wl.q_decode[lo:hi], torch.int32),
                        T(wl.q_t_ms[lo:hi], torch.float64), t_after,
                        T(wl.acc[lo:hi], torch.float64), T(wl.cost[lo:hi], torch.float64),
                        T(wl.w_cost, torch.float64), T(wl.w_lat_ms, torch.float64),
                        realized=r)
        reals.append(r)
    ctx.sync()
    pre = O.trace(wl, n_q=N1, final_state=False)
    full = O.trace(wl, final_state=False)
    np.testing.assert_array_equal(bits(reals[0].cpu().numpy()[0]), bits(pre.realized))
    np.testing.assert_array_equal(bits(reals[1].cpu().numpy()[0]), bits(full.realized[N1:]))
    ctx.close()


@pytest.mark.parametrize("name", ["c2", "c7"])
def test_realized_tag_counter_wrap(monkeypatch, name):
    """The tag counter starts just below its end: the first call's tags run up to it,
    the second call wraps (every ring slot untagged, tags from 0 again); both calls
    still report exactly the oracle's realised TTFTs (c7: under scheduler limits)."""
    monkeypatch.setenv("LAR_TEST_TAG_START", str(2 ** 31 - 1 - 1000))
    wl = make_workload(name, n_q=1200, n_inst=8)
    N, N1 = wl.n_q, 500
    ctx = context_for(wl)
    monkeypatch.delenv("LAR_TEST_TAG_START")
    ctx.advance(float(wl.q_t_ms[0]))
    reals = []
    for lo, hi, t_after in ((0, N1, float(wl.q_t_ms[N1])), (N1, N, float(wl.q_t_ms[-1]))):
        r = torch.full((1, hi - lo), -1.0, dtype=torch.float64, device="cuda:0")
        ctx.route_trace(T(wl.q_prefill[lo:hi], torch.int32), T(wl.q_decode[lo:hi], torch.int32),
                        T(wl.q_t_ms[lo:hi], torch.float64), t_after,
                        T(wl.acc[lo:hi], torch.float64), T(wl.cost[lo:hi], torch.float64),
                        T(wl.w_cost, torch.float64), T(wl.w_lat_ms, torch.float64),
                        realized=r)
        reals.append(r)
    ctx.sync()
    pre = O.trace(wl, n_q=N1, final_state=False)
    full = O.trace(wl, final_state=False)
    np.testing.assert_array_equal(bits(reals[0].cpu().numpy()[0]), bits(pre.realized))
    np.testing.assert_array_equal(bits(reals[1].cpu().numpy()[0]), bits(full.realized[N1:]))
    ctx.close()
