"""GPU parity at full size, in the launch configurations bench.py times.

* c5: all 64 scenarios x 100k queries x 64 instances routed together; four scenarios
  checked in full against the oracle (every choice and chosen-TTFT bit, the
  per-scenario stats, final states).
* c4: 256 instances x 50k queries; the oracle cannot replay the whole trace in a
  test (each estimate walks a backlog of ~10^3 batches of 512 sequences), so the GPU
  routes the first 49,992 queries, the oracle takes the GPU's state at that point
  (validated on load: every resident list invariant) and routes the last 8 queries
  from it, and the GPU's last 8 choices, chosen TTFTs and final state must be the
  oracle's.
* c6 in full, and c2 in full under Eq. 3 with realised-TTFT tracking.
"""

from __future__ import annotations

import dataclasses
import os
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
from gpu_util import T, assert_state_equal, bits, gpu_trace  # noqa: E402
from oracle import oracle as O  # noqa: E402
from paper_2607_18253_amd import context_for  # noqa: E402
from workloads import make_workload  # noqa: E402


def test_c5_full_size_four_scenarios():
    wl = make_workload("c5")
    choice, chosen, util, ctx = gpu_trace(wl)
    st = ctx.stats(T(choice, torch.int32), T(chosen, torch.float64), T(wl.acc, torch.float64),
                   T(wl.cost, torch.float64), T(wl.w_cost, torch.float64))
    ctx.sync()
    st = st.cpu().numpy()
    for z in (0, 21, 42, 63):
        ref = O.trace(wl, scenario=z)
        np.testing.assert_array_equal(choice[z], ref.choice, err_msg=f"scenario {z}")
        np.testing.assert_array_equal(bits(chosen[z]), bits(ref.ttft_chosen))
        np.testing.assert_array_equal(bits(util[z]), bits(ref.util_chosen))
        assert_state_equal(ctx, z, ref)
        want = O.stats(ref.choice, ref.ttft_chosen, wl.acc, wl.cost, wl.col, wl.w_cost[z])
        np.testing.assert_array_equal(bits(st[z]), bits(want), err_msg=f"stats {z}")
    ctx.close()


def test_c4_full_size_last_queries():
    wl = make_workload("c4")
    N, tail = wl.n_q, 8
    N1 = N - tail
    ctx = context_for(wl)
    ctx.advance(float(wl.q_t_ms[0]))

    def run(lo, hi, t_after):
        chosen = torch.full((1, hi - lo), -1.0, dtype=torch.float64, device="cuda:0")
        util = torch.full((1, hi - lo), -1.0, dtype=torch.float64, device="cuda:0")
        ch = ctx.route_trace(T(wl.q_prefill[lo:hi], torch.int32), T(wl.q_decode[lo:hi], torch.int32),
                             T(wl.q_t_ms[lo:hi], torch.float64), t_after,
                             T(wl.acc[lo:hi], torch.float64), T(wl.cost[lo:hi], torch.float64),
                             T(wl.w_cost, torch.float64), T(wl.w_lat_ms, torch.float64),
                             chosen_ttft=chosen, utility=util)
        ctx.sync()
        return ch.cpu().numpy()[0], chosen.cpu().numpy()[0], util.cpu().numpy()[0]

    run(0, N1, float(wl.q_t_ms[N1]))
    s = ctx.read_state(0)
    c2, t2, u2 = run(N1, N, float(wl.q_t_ms[-1]))
    # the oracle from the GPU's state after the first N1 queries (the oracle checks every
    # resident-list invariant when it loads the state)
    rest = dataclasses.replace(
        wl, offsets=s["offsets"], rem_prefill=s["rem_prefill"], rem_decode=s["rem_decode"],
        context=s["context"], clock_ms=s["clock_ms"], q_prefill=wl.q_prefill[N1:],
        q_decode=wl.q_decode[N1:], q_t_ms=wl.q_t_ms[N1:], acc=wl.acc[N1:], cost=wl.cost[N1:],
        tau_u_ms=wl.tau_u_ms[N1:], tau_v=wl.tau_v[N1:])
    ref = O.trace(rest, queue_cap=10 ** 6)
    np.testing.assert_array_equal(c2, ref.choice)
    np.testing.assert_array_equal(bits(t2), bits(ref.ttft_chosen))
    np.testing.assert_array_equal(bits(u2), bits(ref.util_chosen))
    fin = ctx.read_state(0)
    np.testing.assert_array_equal(fin["offsets"], ref.offsets)
    np.testing.assert_array_equal(fin["rem_prefill"], ref.rem_prefill)
    np.testing.assert_array_equal(fin["rem_decode"], ref.rem_decode)
    np.testing.assert_array_equal(fin["context"], ref.context)
    np.testing.assert_array_equal(bits(fin["clock_ms"]), bits(ref.clock_ms))
    np.testing.assert_array_equal(fin["iterations"] - s["iterations"], ref.iterations)
    ctx.close()


def test_c6_full_size():
    """c6 (c2's pool under two-state MMPP arrivals), 100k queries."""
    wl = make_workload("c6")
    choice, chosen, util, ctx = gpu_trace(wl)
    ref = O.trace(wl)
    np.testing.assert_array_equal(choice[0], ref.choice)
    np.testing.assert_array_equal(bits(chosen[0]), bits(ref.ttft_chosen))
    np.testing.assert_array_equal(bits(util[0]), bits(ref.util_chosen))
    assert_state_equal(ctx, 0, ref)
    ctx.close()


def test_c2_full_size_constrained_realized():
    """c2, 100k queries under Eq. 3 with the paper's targets and realised-TTFT
    tracking, as bench.py --objective constrained runs it: choices, estimated and
    realised TTFT bits, OnTimeUtility and the final state."""
    from gpu_util import gpu_trace_realized
    wl = make_workload("c2")
    tau = O.ttft_targets(wl.q_prefill, wl.tau_u_ms, wl.tau_v)
    choice, chosen, real, ctx = gpu_trace_realized(wl, tau=tau)
    ref = O.trace(wl, tau=tau)
    np.testing.assert_array_equal(choice[0], ref.choice)
    np.testing.assert_array_equal(bits(chosen[0]), bits(ref.ttft_chosen))
    np.testing.assert_array_equal(bits(real[0]), bits(ref.realized))
    assert_state_equal(ctx, 0, ref)
    out = ctx.ontime_utility(T(choice, torch.int32), T(real, torch.float64), T(tau, torch.float64),
                             T(wl.acc, torch.float64), T(wl.cost, torch.float64),
                             T(wl.w_cost, torch.float64))
    ctx.sync()
    want = O.ontime_utility(ref.choice, ref.realized, tau, wl.acc, wl.cost, wl.col, wl.w_cost[0])
    assert bits(out.cpu().numpy()[0]) == bits(want)
    ctx.close()
