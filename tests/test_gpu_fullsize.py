"""GPU parity at full size, in the launch configurations bench.py times, against
expected values the oracle wrote (``tests/golden/make_fullsize.py``, oracle only):

* c3: every entry of the 4096 x 1024 what-if matrix (TTFT bits and batch counts, in
  blocks of 16 rows) and the route of every row (choices, Eq. 2 utility at the
  choice).
* c4: the 256-instance trace from the original snapshot over every query block the
  oracle has covered (blocks of 1000 queries; all 50,000 when complete): choices,
  chosen-TTFT and utility bits per block, the batches behind the estimates, and the
  state of every instance after the last covered block.
* c5: all 64 scenarios x 100k queries routed together: per scenario every choice,
  chosen-TTFT and utility bit, the stats, the final state and the batches behind
  the estimates.
* c6 in full, and c2 in full under Eq. 3 with realised-TTFT tracking, against the
  oracle run in the test.

A mismatch names the first differing block or scenario; the oracle can then be run
on that part alone.
"""

from __future__ import annotations

import json
import os
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)
sys.path.insert(0, os.path.join(HERE, "golden"))
from digests import digest, state_digest  # noqa: E402
from gpu_util import T, assert_state_equal, bits, gpu_trace  # noqa: E402
from oracle import oracle as O  # noqa: E402
from paper_2607_18253_amd import context_for  # noqa: E402
from workloads import make_workload  # noqa: E402


def _golden(name):
    path = os.path.join(HERE, "golden", f"fullsize_{name}.json")
    if not os.path.exists(path):
        pytest.fail(f"missing {path}: run tests/golden/make_fullsize.py {name}")
    with open(path) as f:
        return json.load(f)


def _state_digest(ctx, z):
    s = ctx.read_state(z)
    return state_digest(s["offsets"], s["rem_prefill"], s["rem_decode"], s["context"],
                        s["clock_ms"], s["iterations"])


def test_c3_full_matrix_every_entry():
    g = _golden("c3")
    wl = make_workload("c3")
    assert (g["rows"], g["instances"]) == (wl.n_q, wl.n_inst)
    ctx = context_for(wl)
    tt, it = ctx.estimate(T(wl.q_prefill, torch.int32), 0.0)
    util = torch.empty((1, wl.n_q), dtype=torch.float64, device="cuda:0")
    chosen = torch.empty((1, wl.n_q), dtype=torch.float64, device="cuda:0")
    ch = ctx.route(tt, T(wl.acc, torch.float64), T(wl.cost, torch.float64),
                   T(wl.w_cost, torch.float64), T(wl.w_lat_ms, torch.float64),
                   chosen_ttft=chosen, utility=util)
    ctx.sync()
    tt = tt.cpu().numpy()[0]
    it = it.cpu().numpy()[0].astype(np.int32)
    ch = ch.cpu().numpy()[0].astype(np.int32)
    B = g["block_rows"]
    bad_t = [b for b, d in enumerate(g["ttft_blocks"]) if digest(tt[b * B:(b + 1) * B]) != d]
    bad_i = [b for b, d in enumerate(g["iters_blocks"]) if digest(it[b * B:(b + 1) * B]) != d]
    assert not bad_t, f"TTFT differs in row blocks {bad_t[:8]} (rows of {B})"
    assert not bad_i, f"batch counts differ in row blocks {bad_i[:8]} (rows of {B})"
    assert int(it.sum(dtype=np.int64)) == g["iters_total"]
    assert digest(ch) == g["choice"], "route choices differ"
    assert digest(util.cpu().numpy()[0]) == g["utility"], "utility at the choice differs"
    np.testing.assert_array_equal(bits(chosen.cpu().numpy()[0]),
                                  bits(tt[np.arange(wl.n_q), ch]))
    ctx.close()


def test_c4_full_size_from_original_snapshot():
    g = _golden("c4")
    blocks = g["blocks"]
    assert blocks, "no c4 block written yet"
    wl = make_workload("c4")
    N = blocks[-1]["end"]
    assert all(b["first"] == k * g["block_queries"] for k, b in enumerate(blocks))
    ctx = context_for(wl)
    ctx.advance(float(wl.q_t_ms[0]))
    chosen = torch.full((1, N), -1.0, dtype=torch.float64, device="cuda:0")
    util = torch.full((1, N), -1.0, dtype=torch.float64, device="cuda:0")
    ch = ctx.route_trace(T(wl.q_prefill[:N], torch.int32), T(wl.q_decode[:N], torch.int32),
                         T(wl.q_t_ms[:N], torch.float64), float(wl.q_t_ms[N - 1]),
                         T(wl.acc[:N], torch.float64), T(wl.cost[:N], torch.float64),
                         T(wl.w_cost, torch.float64), T(wl.w_lat_ms, torch.float64),
                         chosen_ttft=chosen, utility=util)
    assert ctx.status() == 0
    ch = ch.cpu().numpy()[0].astype(np.int32)
    chosen = chosen.cpu().numpy()[0]
    util = util.cpu().numpy()[0]
    for k, b in enumerate(blocks):
        sl = slice(b["first"], b["end"])
        assert digest(ch[sl]) == b["choice"], f"choices differ in block {k} ({sl})"
        assert digest(chosen[sl]) == b["ttft"], f"chosen TTFT differs in block {k}"
        assert digest(util[sl]) == b["utility"], f"utility differs in block {k}"
    assert int(ctx.trace_work()[0]) == sum(b["estimate_batches"] for b in blocks)
    assert _state_digest(ctx, 0) == blocks[-1]["state"], f"state after {N} queries differs"
    ctx.close()


def test_c5_all_scenarios_full_size():
    g = _golden("c5")
    wl = make_workload("c5")
    assert (g["scenarios"], g["queries"]) == (wl.n_scen, wl.n_q)
    choice, chosen, util, ctx = gpu_trace(wl)
    assert ctx.status() == 0
    st = ctx.stats(T(choice, torch.int32), T(chosen, torch.float64), T(wl.acc, torch.float64),
                   T(wl.cost, torch.float64), T(wl.w_cost, torch.float64))
    ctx.sync()
    st = st.cpu().numpy()
    work = ctx.trace_work()
    bad = []
    for z, want in enumerate(g["per_scenario"]):
        got = dict(choice=digest(choice[z].astype(np.int32)), ttft=digest(chosen[z]),
                   utility=digest(util[z]),
                   stats_bits=[format(int(v), "016x") for v in st[z].view(np.uint64)],
                   state=_state_digest(ctx, z), estimate_batches=int(work[z]))
        diff = [k for k in got if got[k] != want[k]]
        if diff:
            bad.append((z, diff))
    assert not bad, f"scenarios differing from the oracle: {bad[:8]}"
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
