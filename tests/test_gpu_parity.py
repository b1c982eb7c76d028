"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Integer results (iteration counts, choices, final states) must match exactly;
fp64 TTFT must match within 1e-9 relative error -- the kernels evaluate every
batch time in the same operation order with the same roundings as the oracle, so
the tests demand bit equality, which implies that bound.
"""

import json
import os

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from gpu_util import DEV, T, assert_state_equal, bits, gpu_trace  # noqa: E402
from oracle import oracle as O  # noqa: E402
from paper_2607_18253_amd import LarContext, LarError, context_for  # noqa: E402
from paper_2607_18253_amd import lar as L  # noqa: E402
from workloads import make_tiny_workload, make_workload  # noqa: E402

GOLD = os.path.join(os.path.dirname(__file__), "golden", "hand_worked.json")
REL_TOL = 1e-9


def _close(a, b):
    a, b = np.asarray(a), np.asarray(b)
    return np.all(np.abs(a - b) <= REL_TOL * np.maximum(np.abs(a), np.abs(b)))


def _single(coef, B, M, reqs, clock=0.0, flags=0, max_prompt=64, mcap=None, qcap=64):
    ctx = LarContext(1, 1, max_seqs_cap=mcap or M, queue_cap=qcap, max_prompt=max_prompt,
                     flags=flags)
    ctx.load_state(a=[coef["a"]], b=[coef["b"]], c=[coef["c"]], d=[coef["d"]], e=[coef["e"]],
                   budget=[B], max_seqs=[M], col=[0], offsets=[0, len(reqs)],
                   rem_prefill=[r[0] for r in reqs], rem_decode=[r[1] for r in reqs],
                   context=[r[2] for r in reqs], clock_ms=[clock])
    return ctx


# ------------------------------------------------------------------ hand-worked
@pytest.mark.parametrize("flags", [0, 1])
def test_hand_worked_gpu(flags):
    g = json.load(open(GOLD))
    for case in g["estimates"]:
        ctx = _single(g["coef"], case["budget"], case["max_seqs"], case["requests"],
                      case["clock"], flags=flags)
        if "advance_to" in case:
            ctx.advance(case["advance_to"])
        tt, it = ctx.estimate(T([case["p"]], torch.int32), case["t"])
        ctx.sync()
        key = "B" if flags == 0 else "A"
        assert tt.item() == case["ttft_" + key], case["name"]
        assert it.item() == case["iters_" + key], case["name"]
        ctx.close()


def test_hand_worked_routes_gpu():
    g = json.load(open(GOLD))
    for case in g["routes"]:
        n = len(case["ttft"])
        ctx = LarContext(1, n, max_seqs_cap=1, queue_cap=4, max_prompt=4)
        ctx.load_state(a=[1] * n, b=[1] * n, c=[1] * n, d=[0] * n, e=[0] * n, budget=[1] * n,
                       max_seqs=[1] * n, col=list(range(n)), offsets=[0] * (n + 1),
                       rem_prefill=[], rem_decode=[], context=[], clock_ms=[0.0] * n)
        util = torch.empty((1, 1), dtype=torch.float64, device=DEV)
        ch = ctx.route(T([[case["ttft"]]], torch.float64), T([case["acc"]], torch.float64),
                       T([case["cost"]], torch.float64), T([case["w_cost"]], torch.float64),
                       T([case["w_lat"]], torch.float64), utility=util)
        ctx.sync()
        assert ch.item() == case["choice"], case["name"]
        ctx.close()


# ------------------------------------------------------------------ what-if estimates
@pytest.mark.parametrize("seed", range(12))
@pytest.mark.parametrize("flags", [0, 1])
def test_estimate_tiny_pools(seed, flags):
    wl = make_tiny_workload(seed, n_inst=7, max_res=6, n_q=9, budget=(1, 9), max_seqs=(1, 5),
                            prompt=(1, 14), dyadic=(seed % 3 == 0))
    ref, ref_it = O.estimate_matrix(wl, range(wl.n_q), range(wl.n_inst), 0.0, reading=flags)
    ctx = context_for(wl, flags=flags)
    tt, it = ctx.estimate(T(wl.q_prefill, torch.int32), 0.0)
    ctx.sync()
    np.testing.assert_array_equal(it.cpu().numpy()[0], ref_it)
    np.testing.assert_array_equal(bits(tt.cpu().numpy()[0]), bits(ref))
    ctx.close()


def test_estimate_many_slots_and_ragged():
    """Wide running sets (several 64-slot passes per lane group), a ragged instance
    count, empty instances, long prompts crossing many budget windows."""
    rng = np.random.default_rng(11)
    I = 67
    M_all = rng.choice([1, 3, 64, 65, 130, 300, 700], size=I)
    B_all = M_all + rng.integers(0, 2000, size=I)
    reqs, offs = [], [0]
    for j in range(I):
        n = int(rng.integers(0, 900)) if j % 5 else 0
        n_run = int(min(n, M_all[j], rng.integers(0, n + 1)))
        rp = np.where(np.arange(n) < n_run, np.where(rng.random(n) < 0.85, 0,
                      rng.integers(1, 300, n)), rng.integers(1, 3000, n))
        cx = np.where(np.arange(n) < n_run, rng.integers(1, 5000, n), 0)
        rd = rng.integers(1, 400, n)
        reqs.append((rp, rd, cx))
        offs.append(offs[-1] + n)
    coef = rng.random((5, I))
    coef[3] *= 1e-3
    coef[4] *= 1e-6
    ctx = LarContext(1, I, max_seqs_cap=int(M_all.max()), queue_cap=1024, max_prompt=20000)
    ctx.load_state(a=coef[0], b=coef[1], c=coef[2], d=coef[3], e=coef[4], budget=B_all,
                   max_seqs=M_all, col=np.zeros(I, np.int32), offsets=offs,
                   rem_prefill=np.concatenate([r[0] for r in reqs]),
                   rem_decode=np.concatenate([r[1] for r in reqs]),
                   context=np.concatenate([r[2] for r in reqs]), clock_ms=np.zeros(I))
    ps = np.array([1, 2, 63, 64, 65, 1000, 4096, 19999], np.int32)
    tt, it = ctx.estimate(T(ps, torch.int32), 0.0)
    ctx.sync()
    tt, it = tt.cpu().numpy()[0], it.cpu().numpy()[0]
    for j in range(I):
        q = O.Queue(O.make_params(*coef[:, j], B_all[j], M_all[j]), *reqs[j], 0.0)
        for a, p in enumerate(ps):
            want, wit = q.estimate(int(p), 1, 0.0)
            assert it[a, j] == wit and bits(tt[a, j]) == bits(want), (j, p)
    ctx.close()


@pytest.mark.parametrize("flags", [0, 1])
def test_max_budget_adjacent_large_waiting(flags):
    """The largest token budget, 2^30 - 1, with four waiting entries of nearly that
    many tokens behind a smaller first one: the saturating prefix sum that composes
    the batch adds two saturated partial sums (2B - 2 < 2^31).  Estimates at several
    prompts and a replay, against the oracle."""
    B = (1 << 30) - 1
    M = 8
    coef = dict(a=1.0, b=2.0 ** -20, c=0.5, d=0.0, e=2.0 ** -40)
    reqs = [(5, 3, 0), (B - 1, 2, 0), (B - 2, 4, 0), (B - 3, 1, 0), (B - 4, 2, 0)]
    ctx = _single(coef, B, M, reqs, flags=flags, max_prompt=B)
    ps = [1, 3, 1000, B - 7, B]
    tt, it = ctx.estimate(T(ps, torch.int32), 0.0)
    ctx.sync()
    tt, it = tt.cpu().numpy()[0, :, 0], it.cpu().numpy()[0, :, 0]
    par = O.make_params(coef["a"], coef["b"], coef["c"], coef["d"], coef["e"], B, M)
    q = O.Queue(par, [r[0] for r in reqs], [r[1] for r in reqs], [r[2] for r in reqs])
    for k, p in enumerate(ps):
        want, wit = q.estimate(p, 1, 0.0, reading=flags)
        assert it[k] == wit and bits(tt[k]) == bits(want), (p, tt[k], want, it[k], wit)
    t_next = float(tt[2]) * 0.75
    ctx.advance(t_next)
    q.advance(t_next)
    s = ctx.read_state(0)
    rp, rd, cx, clk, its = q.state()
    np.testing.assert_array_equal(s["rem_prefill"], rp)
    np.testing.assert_array_equal(s["rem_decode"], rd)
    np.testing.assert_array_equal(s["context"], cx)
    assert bits(s["clock_ms"][0]) == bits(clk) and s["iterations"][0] == its
    ctx.close()


# ------------------------------------------------------------------ sequential traces
@pytest.mark.parametrize("seed", range(16))
@pytest.mark.parametrize("flags", [0, 1])
def test_trace_tiny_pools(seed, flags):
    wl = make_tiny_workload(seed, n_inst=5, max_res=6, n_q=40, dyadic=(seed % 2 == 0),
                            n_scen=3)
    choice, chosen, util, ctx = gpu_trace(wl, flags=flags, queue_cap=10 ** 4)
    for z in range(wl.n_scen):
        ref = O.trace(wl, scenario=z, reading=flags, queue_cap=10 ** 4)
        np.testing.assert_array_equal(choice[z], ref.choice)
        np.testing.assert_array_equal(bits(chosen[z]), bits(ref.ttft_chosen))
        np.testing.assert_array_equal(bits(util[z]), bits(ref.util_chosen))
        assert_state_equal(ctx, z, ref)
    ctx.close()


def _tail_k(wl):
    """Bound on the decode-only batches after an admission batch (one lane each in the
    clustered trace kernel, which needs it <= 64; larger bounds take the HBM-state
    trace kernel)."""
    return int(max(-(-(wl.max_prompt - 1) // (int(b) - int(m) + 1)) + 1
                   for b, m in zip(wl.budget, wl.max_seqs)))


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("prompt_max,path", [(60, "clustered"), (300, "hbm-state")])
def test_trace_tiny_pools_long_prompts(seed, prompt_max, path):
    """Prompts many batches long: deep frontier tails (clustered kernel) and, past 64
    tail batches, the HBM-state trace kernel."""
    wl = make_tiny_workload(100 + seed, n_inst=6, max_res=8, n_q=30, prompt=(1, prompt_max),
                            budget=(1, 6), max_seqs=(1, 3), n_scen=2)
    k = _tail_k(wl)
    assert (k <= 64) == (path == "clustered"), k
    choice, chosen, util, ctx = gpu_trace(wl, queue_cap=10 ** 4)
    for z in range(wl.n_scen):
        ref = O.trace(wl, scenario=z, queue_cap=10 ** 4)
        np.testing.assert_array_equal(choice[z], ref.choice)
        np.testing.assert_array_equal(bits(chosen[z]), bits(ref.ttft_chosen))
        np.testing.assert_array_equal(bits(util[z]), bits(ref.util_chosen))
        assert_state_equal(ctx, z, ref)
    ctx.close()


@pytest.mark.parametrize("n_q", [1, 63, 64, 65, 128, 129])
def test_trace_query_block_boundaries(n_q):
    """The clustered trace reads the queries in blocks of 64, one lane each, with the
    next block fetched ahead: traces one query long, one short of a block, exactly one
    block, one past it, two blocks and one past two, over three workgroups per
    scenario (9 instances, 4 waves each) and two scenarios."""
    wl = make_tiny_workload(200 + n_q, n_inst=9, max_res=5, n_q=n_q, n_scen=2)
    assert _tail_k(wl) <= 64   # the clustered kernel
    choice, chosen, util, ctx = gpu_trace(wl, queue_cap=10 ** 4)
    for z in range(wl.n_scen):
        ref = O.trace(wl, scenario=z, queue_cap=10 ** 4)
        np.testing.assert_array_equal(choice[z], ref.choice)
        np.testing.assert_array_equal(bits(chosen[z]), bits(ref.ttft_chosen))
        np.testing.assert_array_equal(bits(util[z]), bits(ref.util_chosen))
        assert_state_equal(ctx, z, ref)
    ctx.close()


def _identical_empty_pool(seed, n_inst, n_q, n_scen):
    """A tiny workload whose instances are identical and empty and share one
    accuracy / cost column: the utilities of instances in the same state tie exactly."""
    import dataclasses
    wl = make_tiny_workload(seed, n_inst=n_inst, max_res=1, n_q=n_q, n_scen=n_scen,
                            dyadic=True, budget=(6, 6), max_seqs=(2, 2))
    same = {f: np.full_like(getattr(wl, f), getattr(wl, f)[0])
            for f in ("a", "b", "c", "d", "e", "budget", "max_seqs")}
    return dataclasses.replace(
        wl, **same, col=np.zeros(n_inst, np.int32), offsets=np.zeros(n_inst + 1, np.int32),
        rem_prefill=np.zeros(0, np.int32), rem_decode=np.zeros(0, np.int32),
        context=np.zeros(0, np.int32), clock_ms=np.zeros(n_inst))


@pytest.mark.parametrize("n_inst", [13, 40])
def test_trace_ties_across_workgroups(n_inst):
    """Every query's best utility is shared by all instances in the same state, so the
    lowest index among them must win: within a workgroup (one comparison and a ballot
    over its waves) and across workgroups (one over the posts) -- 13 instances are 4
    workgroups of 4 waves, 40 are 10; two scenarios."""
    wl = _identical_empty_pool(31 + n_inst, n_inst, 120, 2)
    assert _tail_k(wl) <= 64   # the clustered kernel
    choice, chosen, util, ctx = gpu_trace(wl, queue_cap=10 ** 4)
    for z in range(wl.n_scen):
        ref = O.trace(wl, scenario=z, queue_cap=10 ** 4)
        np.testing.assert_array_equal(choice[z], ref.choice)
        np.testing.assert_array_equal(bits(chosen[z]), bits(ref.ttft_chosen))
        np.testing.assert_array_equal(bits(util[z]), bits(ref.util_chosen))
        assert_state_equal(ctx, z, ref)
        # ties did decide: some query went to a non-zero index while a lower one tied
        assert len(set(ref.choice.tolist())) > 1
    ctx.close()


def test_trace_c1_full():
    wl = make_workload("c1")
    choice, chosen, util, ctx = gpu_trace(wl)
    ref = O.trace(wl)
    np.testing.assert_array_equal(choice[0], ref.choice)
    np.testing.assert_array_equal(bits(chosen[0]), bits(ref.ttft_chosen))
    np.testing.assert_array_equal(bits(util[0]), bits(ref.util_chosen))
    assert_state_equal(ctx, 0, ref)
    ctx.close()


def test_trace_c2_prefix():
    wl = make_workload("c2", n_q=2000)
    choice, chosen, util, ctx = gpu_trace(wl)
    ref = O.trace(wl)
    np.testing.assert_array_equal(choice[0], ref.choice)
    np.testing.assert_array_equal(bits(chosen[0]), bits(ref.ttft_chosen))
    assert_state_equal(ctx, 0, ref)
    ctx.close()


def test_trace_c2_full_bench_configuration():
    """Config 2 at full size in the launch configuration bench.py times (100k queries,
    32 instances, one trace launch): every choice, chosen TTFT and utility bit, and the
    final state of every instance."""
    wl = make_workload("c2")
    choice, chosen, util, ctx = gpu_trace(wl)
    ref = O.trace(wl)
    np.testing.assert_array_equal(choice[0], ref.choice)
    np.testing.assert_array_equal(bits(chosen[0]), bits(ref.ttft_chosen))
    np.testing.assert_array_equal(bits(util[0]), bits(ref.util_chosen))
    assert_state_equal(ctx, 0, ref)
    ctx.close()


def test_trace_c5_two_scenarios_1000():
    """Config 5: all 64 scenarios routed together for 1000 queries; the two extreme
    weight scenarios (0 and 63) checked in full, states included."""
    wl = make_workload("c5", n_q=1000)
    choice, chosen, util, ctx = gpu_trace(wl)
    for z in (0, 63):
        ref = O.trace(wl, scenario=z)
        np.testing.assert_array_equal(choice[z], ref.choice, err_msg=f"scenario {z}")
        np.testing.assert_array_equal(bits(chosen[z]), bits(ref.ttft_chosen))
        np.testing.assert_array_equal(bits(util[z]), bits(ref.util_chosen))
        assert_state_equal(ctx, z, ref)
    ctx.close()


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("flags", [0, 1])
def test_trace_tiny_pools_sixteen_waves(seed, flags):
    """Tiny random pools with every coefficient term (d and e too), 256 scenarios of 5
    instances: 1280 queues take the 16-wave workgroups, whose replays of summarised
    instances fold quiet batches on the summary (keeping its first decode batch's
    context sum current) and whose chosen instances step their admission batch from
    it. Every 17th scenario against the oracle, states included, both readings."""
    wl = make_tiny_workload(1100 + seed, n_inst=5, max_res=6, n_q=40, n_scen=256,
                            dyadic=(seed % 2 == 0))
    assert (wl.d != 0).any() and (wl.e != 0).any()
    choice, chosen, util, ctx = gpu_trace(wl, flags=flags, queue_cap=10 ** 4)
    for z in range(0, wl.n_scen, 17):
        ref = O.trace(wl, scenario=z, reading=flags, queue_cap=10 ** 4)
        np.testing.assert_array_equal(choice[z], ref.choice, err_msg=f"scenario {z}")
        np.testing.assert_array_equal(bits(chosen[z]), bits(ref.ttft_chosen))
        np.testing.assert_array_equal(bits(util[z]), bits(ref.util_chosen))
        assert_state_equal(ctx, z, ref)
    ctx.close()


def test_trace_c6_bursty_prefix():
    """Config 6: the medium pool under MMPP-2 arrivals (bursts at 6x the low rate),
    first 5000 queries."""
    wl = make_workload("c6", n_q=5000)
    choice, chosen, util, ctx = gpu_trace(wl)
    ref = O.trace(wl)
    np.testing.assert_array_equal(choice[0], ref.choice)
    np.testing.assert_array_equal(bits(chosen[0]), bits(ref.ttft_chosen))
    np.testing.assert_array_equal(bits(util[0]), bits(ref.util_chosen))
    assert_state_equal(ctx, 0, ref)
    ctx.close()


def test_trace_c4_prefix():
    wl = make_workload("c4", n_q=4)
    choice, chosen, util, ctx = gpu_trace(wl)
    ref = O.trace(wl)
    np.testing.assert_array_equal(choice[0], ref.choice)
    np.testing.assert_array_equal(bits(chosen[0]), bits(ref.ttft_chosen))
    assert_state_equal(ctx, 0, ref)
    ctx.close()


@pytest.mark.parametrize("n_inst,n_q", [(8, 80), (4, 120)])
def test_trace_c4_instances_shared(n_inst, n_q):
    """Config 4's instances (512 slots, 1024-deep queues, prompts up to 131k tokens,
    context-dependent batch time), few of them so that many queries join the same
    instance: each joins at the instance's cached admission point and is walked to
    the next one over the cached decode-only batches."""
    wl = make_workload("c4", n_q=n_q, n_inst=n_inst)
    choice, chosen, util, ctx = gpu_trace(wl)
    ref = O.trace(wl)
    np.testing.assert_array_equal(choice[0], ref.choice)
    np.testing.assert_array_equal(bits(chosen[0]), bits(ref.ttft_chosen))
    np.testing.assert_array_equal(bits(util[0]), bits(ref.util_chosen))
    assert_state_equal(ctx, 0, ref)
    ctx.close()


@pytest.mark.parametrize("limits", [False, True])
def test_trace_large_pool_hbm_kernel(limits):
    """600 instances in 8 scenarios (4800 queues, more than the clustered shapes
    take): the HBM-state trace, each of 8 waves owning 75 instances, so the
    instances past a wave's 64th read their accuracy and cost from memory; under
    scheduler limits 1100 instances over 16 waves (69 each).  Three scenarios
    against the oracle."""
    n_inst = 1100 if limits else 600
    wl = make_tiny_workload(11, n_inst=n_inst, n_scen=8, n_q=12, max_res=6, budget=(4, 16),
                            max_seqs=(2, 6), prompt=(1, 20))
    if limits:
        wl.sched = np.tile(np.array([[3, 0, 0, 64]], np.int32), (wl.n_inst, 1))
    choice, chosen, util, ctx = gpu_trace(wl)
    for z in (0, 3, 7):
        ref = O.trace(wl, scenario=z)
        np.testing.assert_array_equal(choice[z], ref.choice, err_msg=f"scenario {z}")
        np.testing.assert_array_equal(bits(chosen[z]), bits(ref.ttft_chosen))
        np.testing.assert_array_equal(bits(util[z]), bits(ref.util_chosen))
        assert_state_equal(ctx, z, ref)
    ctx.close()


def test_trace_c5_all_scenarios_prefix_and_stats():
    wl = make_workload("c5", n_q=24)
    choice, chosen, util, ctx = gpu_trace(wl)
    acc, cost = T(wl.acc, torch.float64), T(wl.cost, torch.float64)
    st = ctx.stats(T(choice, torch.int32), T(chosen, torch.float64), acc, cost,
                   T(wl.w_cost, torch.float64))
    ctx.sync()
    st = st.cpu().numpy()
    for z in range(wl.n_scen):
        ref = O.trace(wl, scenario=z)
        np.testing.assert_array_equal(choice[z], ref.choice, err_msg=f"scenario {z}")
        np.testing.assert_array_equal(bits(chosen[z]), bits(ref.ttft_chosen))
        if z in (0, 27, 63):
            assert_state_equal(ctx, z, ref)
        want = O.stats(ref.choice, ref.ttft_chosen, wl.acc, wl.cost, wl.col, wl.w_cost[z])
        np.testing.assert_array_equal(bits(st[z]), bits(want), err_msg=f"stats {z}")
    ctx.close()


@pytest.mark.parametrize("n", [1, 2, 3, 100, 1023, 1024, 1025, 4097])
def test_stats_ragged_lengths_and_ties(n):
    """The statistics kernel (means folded in query order by one block, p50 / p99 by
    radix passes in another) on trace lengths around its 1024-query chunks, with TTFTs
    that all tie (scenario 0), take a few values (1), or differ only in their low bits
    over several magnitudes (2), against the oracle bit for bit."""
    rng = np.random.default_rng(n)
    I, Z, n_cols = 5, 3, 3
    col = np.array([0, 1, 2, 0, 1], np.int32)
    ctx = LarContext(Z, I, max_seqs_cap=4, queue_cap=4, max_prompt=16)
    ones = np.ones(I)
    ctx.load_state(a=ones, b=ones, c=ones, d=0 * ones, e=0 * ones, budget=np.full(I, 8, np.int32),
                   max_seqs=np.full(I, 4, np.int32), col=col, offsets=np.zeros(I + 1, np.int32),
                   rem_prefill=np.zeros(0, np.int32), rem_decode=np.zeros(0, np.int32),
                   context=np.zeros(0, np.int32), clock_ms=np.zeros(I))
    choice = rng.integers(0, I, size=(Z, n)).astype(np.int32)
    ttft = np.empty((Z, n))
    ttft[0] = 157.25
    ttft[1] = rng.choice([3.5, 40.0, 40.0, 1200.125], size=n)
    base = rng.choice([0.75, 12.0, 480.0, 9000.0], size=n)
    ttft[2] = base + rng.integers(0, 64, size=n) * np.spacing(base)
    acc, cost = rng.random((n, n_cols)), rng.random((n, n_cols))
    w_cost = np.array([0.0, 0.5, 2.0])
    st = ctx.stats(T(choice, torch.int32), T(ttft, torch.float64), T(acc, torch.float64),
                   T(cost, torch.float64), T(w_cost, torch.float64))
    ctx.sync()
    st = st.cpu().numpy()
    for z in range(Z):
        want = O.stats(choice[z], ttft[z], acc, cost, col, w_cost[z])
        np.testing.assert_array_equal(bits(st[z]), bits(want), err_msg=f"scenario {z}")
    ctx.close()


@pytest.mark.parametrize("name", ["c2", "c7"])
def test_checkpoint_resume_identical(name):
    """read_state -> load_state into a fresh context, continue: same results (c7: under
    scheduler limits, the snapshot holding preempted requests and cut decodes)."""
    wl = make_workload(name, n_q=600, n_inst=8)
    full_c, full_t, _, ctx = gpu_trace(wl)
    ctx.close()
    N1 = 250
    from paper_2607_18253_amd import context_for as cf
    ctx1 = cf(wl)
    ctx1.advance(float(wl.q_t_ms[0]))
    c1 = ctx1.route_trace(T(wl.q_prefill[:N1], torch.int32), T(wl.q_decode[:N1], torch.int32),
                          T(wl.q_t_ms[:N1], torch.float64), float(wl.q_t_ms[N1]),
                          T(wl.acc[:N1], torch.float64), T(wl.cost[:N1], torch.float64),
                          T(wl.w_cost, torch.float64), T(wl.w_lat_ms, torch.float64))
    ctx1.sync()
    st = ctx1.read_state(0)
    ctx2 = LarContext(1, wl.n_inst, max_seqs_cap=int(wl.max_seqs.max()), queue_cap=wl.queue_cap,
                      max_prompt=wl.max_prompt)
    if wl.sched is not None:
        ctx2.set_scheduler(wl.sched)
    ctx2.load_state(a=wl.a, b=wl.b, c=wl.c, d=wl.d, e=wl.e, budget=wl.budget,
                    max_seqs=wl.max_seqs, col=wl.col, offsets=st["offsets"],
                    rem_prefill=st["rem_prefill"], rem_decode=st["rem_decode"],
                    context=st["context"], clock_ms=st["clock_ms"])
    c2 = ctx2.route_trace(T(wl.q_prefill[N1:], torch.int32), T(wl.q_decode[N1:], torch.int32),
                          T(wl.q_t_ms[N1:], torch.float64), float(wl.q_t_ms[-1]),
                          T(wl.acc[N1:], torch.float64), T(wl.cost[N1:], torch.float64),
                          T(wl.w_cost, torch.float64), T(wl.w_lat_ms, torch.float64))
    ctx2.sync()
    got = np.concatenate([c1.cpu().numpy()[0], c2.cpu().numpy()[0]])
    np.testing.assert_array_equal(got, full_c[0])
    ctx1.close()
    ctx2.close()


# ------------------------------------------------------------------ edge cases / errors
def test_empty_pool_and_single_slot():
    """All instances empty; M = 1; prompts equal to, below and above the budget."""
    coef = dict(a=1.0, b=0.5, c=0.25, d=0.125, e=0.0625)
    ctx = _single(coef, 1, 1, [], max_prompt=50)
    tt, it = ctx.estimate(T([1, 2, 50], torch.int32), 0.0)
    ctx.sync()
    q = O.Queue(O.make_params(1, .5, .25, .125, .0625, 1, 1), [], [], [])
    for a, p in enumerate([1, 2, 50]):
        want, wit = q.estimate(p, 1, 0.0)
        assert tt.cpu().numpy()[0, a, 0] == want and it.cpu().numpy()[0, a, 0] == wit
    ctx.close()


def test_empty_batches_are_noops():
    """A batch of zero queries is valid and does nothing: estimate, route (both
    objectives), targets and traces (both objectives) with n = 0 return OK, enqueue
    nothing and leave every instance as it was; negative counts are argument errors."""
    wl = make_tiny_workload(3, n_inst=3, n_q=4)
    ctx = context_for(wl)
    ctx.advance(float(wl.q_t_ms[0]))
    ctx.sync()
    before = ctx.read_state(0)
    I = wl.n_inst
    e_i = torch.empty(0, dtype=torch.int32, device=DEV)
    e_d = torch.empty(0, dtype=torch.float64, device=DEV)
    e_rows = torch.empty((0, int(wl.acc.shape[1])), dtype=torch.float64, device=DEV)
    wc, wlat = T(wl.w_cost, torch.float64), T(wl.w_lat_ms, torch.float64)
    tt, it = ctx.estimate(e_i, float(wl.q_t_ms[0]))
    assert tt.shape == (1, 0, I) and it.shape == (1, 0, I)
    ch = ctx.route(torch.empty((1, 0, I), dtype=torch.float64, device=DEV), e_rows, e_rows,
                   wc, wlat)
    assert ch.shape == (1, 0)
    ctx.route_constrained(torch.empty((1, 0, I), dtype=torch.float64, device=DEV), e_d,
                          e_rows, e_rows, wc)
    assert ctx.ttft_targets(e_i, e_d, e_d).shape == (0,)
    ctx.route_trace(e_i, e_i, e_d, float(wl.q_t_ms[-1]) + 1e6, e_rows, e_rows, wc, wlat)
    ctx.route_trace_constrained(e_i, e_i, e_d, float(wl.q_t_ms[-1]) + 1e6, e_d, e_rows,
                                e_rows, wc)
    ctx.sync()
    after = ctx.read_state(0)
    for k in ("offsets", "rem_prefill", "rem_decode", "context", "iterations"):
        np.testing.assert_array_equal(after[k], before[k], err_msg=k)
    np.testing.assert_array_equal(bits(after["clock_ms"]), bits(before["clock_ms"]))
    assert ctx._L.lar_estimate_ttft(ctx._h, -1, None, 0.0, None, None) == L.LAR_E_ARG
    assert ctx._L.lar_ttft_targets(ctx._h, -1, None, None, None, None) == L.LAR_E_ARG
    ctx.close()


def test_sticky_errors():
    coef = dict(a=1.0, b=0.5, c=0.25, d=0.0, e=0.0)
    # prompt above max_prompt -> LAR_E_ARG from the kernel, sticky until reload
    ctx = _single(coef, 8, 2, [[0, 3, 4]], max_prompt=10)
    ctx.estimate(T([11], torch.int32), 0.0)
    assert ctx.status() == L.LAR_E_ARG
    with pytest.raises(LarError):
        ctx.estimate(T([3], torch.int32), 0.0)
    ctx.load_state(a=[1.0], b=[0.5], c=[0.25], d=[0.0], e=[0.0], budget=[8], max_seqs=[2],
                   col=[0], offsets=[0, 0], rem_prefill=[], rem_decode=[], context=[],
                   clock_ms=[0.0])
    ctx.estimate(T([3], torch.int32), 0.0)
    assert ctx.status() == L.LAR_OK
    # estimate at a time the instance has not reached -> LAR_E_STATE
    ctx.estimate(T([3], torch.int32), 5.0)
    assert ctx.status() == L.LAR_E_STATE
    ctx.close()
    # waiting queue overflow on commit -> LAR_E_CAPACITY
    ctx = _single(coef, 8, 1, [[0, 50, 4], [5, 1, 0]], qcap=2)
    ch = T([0], torch.int32)
    ctx.commit(ch, 4, 1, 0.0)
    assert ctx.status() == L.LAR_OK
    ctx.commit(ch, 4, 1, 0.0)
    assert ctx.status() == L.LAR_E_CAPACITY
    ctx.close()
    # iteration cap -> LAR_E_ITER, for estimates and for the replay
    ctx = LarContext(1, 1, max_seqs_cap=1, queue_cap=4, max_prompt=100, max_iters=5)
    ctx.load_state(a=[1.0], b=[1.0], c=[1.0], d=[0.0], e=[0.0], budget=[1], max_seqs=[1],
                   col=[0], offsets=[0, 1], rem_prefill=[0], rem_decode=[20], context=[3],
                   clock_ms=[0.0])
    ctx.estimate(T([1], torch.int32), 0.0)
    assert ctx.status() == L.LAR_E_ITER
    ctx.close()
    ctx = LarContext(1, 1, max_seqs_cap=1, queue_cap=4, max_prompt=100, max_iters=5)
    ctx.load_state(a=[1.0], b=[1.0], c=[1.0], d=[0.0], e=[0.0], budget=[1], max_seqs=[1],
                   col=[0], offsets=[0, 1], rem_prefill=[0], rem_decode=[20], context=[3],
                   clock_ms=[0.0])
    ctx.advance(1000.0)
    assert ctx.status() == L.LAR_E_ITER
    ctx.close()


def test_host_argument_errors():
    with pytest.raises(LarError):
        LarContext(0, 1, max_seqs_cap=1, queue_cap=1, max_prompt=1)
    ctx = LarContext(1, 2, max_seqs_cap=4, queue_cap=4, max_prompt=8)
    good = dict(a=[1, 1], b=[1, 1], c=[1, 1], d=[0, 0], e=[0, 0], budget=[8, 8], max_seqs=[4, 4],
                col=[0, 1], offsets=[0, 1, 2], rem_prefill=[0, 3], rem_decode=[1, 1],
                context=[2, 0], clock_ms=[0.0, 0.0])
    ctx.load_state(**good)
    for k, v, code in [("max_seqs", [5, 4], L.LAR_E_ARG), ("budget", [3, 8], L.LAR_E_ARG),
                       ("rem_decode", [0, 1], L.LAR_E_STATE),
                       ("context", [0, 0], L.LAR_E_STATE), ("a", [np.nan, 1], L.LAR_E_ARG)]:
        bad = dict(good)
        bad[k] = v
        with pytest.raises(LarError) as e:
            ctx.load_state(**bad)
        assert e.value.code == code, k
    ctx.load_state(**good)
    with pytest.raises(LarError):   # n_cols does not cover col 1
        ctx.route(T(np.zeros((1, 1, 2)), torch.float64), T(np.zeros((1, 1)), torch.float64),
                  T(np.zeros((1, 1)), torch.float64), T([0.0], torch.float64),
                  T([0.0], torch.float64))
    ctx.close()


def test_snapshot_board_feeds_the_estimator():
    """Instances publish their snapshots on the board; the router's collected copy,
    loaded with lar_load_state, gives bit for bit the estimates of the oracle on the
    same snapshot (config 1, 16 resident requests per instance)."""
    from paper_2607_18253_amd.lar import SnapshotBoard
    wl = make_workload("c1")
    board = SnapshotBoard(wl.n_inst, 64)
    for j in range(wl.n_inst):
        rp, rd, cx = wl.instance_requests(j)
        board.publish(j, rp, rd, cx, float(wl.clock_ms[j]))
    snap = board.collect()
    board.close()
    ctx = context_for(wl)
    ctx.load_state(a=wl.a, b=wl.b, c=wl.c, d=wl.d, e=wl.e, budget=wl.budget,
                   max_seqs=wl.max_seqs, col=wl.col, offsets=snap["offsets"],
                   rem_prefill=snap["rem_prefill"], rem_decode=snap["rem_decode"],
                   context=snap["context"], clock_ms=snap["clock_ms"])
    qp = wl.q_prefill[:50]
    tt, it = ctx.estimate(T(qp, torch.int32), 0.0)
    ctx.sync()
    tt, it = tt.cpu().numpy()[0], it.cpu().numpy()[0]
    ref, ref_it = O.estimate_matrix(wl, range(50), range(wl.n_inst), 0.0)
    np.testing.assert_array_equal(it, ref_it)
    np.testing.assert_array_equal(bits(tt), bits(ref))
    ctx.close()


def test_trace_sync_timeout_is_reported(monkeypatch):
    """The bounded cross-workgroup wait, forced from the host: workgroup 3 of config
    2's clustered trace (32 instances, 8 workgroups of 4) leaves out its post for
    query 5; the other workgroups wait until the bound (2 ms here), and the trace ends
    with the sticky LAR_E_SYNC instead of hanging.  A context created without the
    hooks then routes the same trace like the oracle."""
    wl = make_workload("c2", n_q=200)
    monkeypatch.setenv("LAR_SYNC_TIMEOUT_MS", "2")
    monkeypatch.setenv("LAR_TEST_SKIP_POST", "3:5")
    ctx = context_for(wl)
    monkeypatch.delenv("LAR_SYNC_TIMEOUT_MS")
    monkeypatch.delenv("LAR_TEST_SKIP_POST")
    ctx.advance(float(wl.q_t_ms[0]))
    args = (T(wl.q_prefill, torch.int32), T(wl.q_decode, torch.int32),
            T(wl.q_t_ms, torch.float64), float(wl.q_t_ms[-1]), T(wl.acc, torch.float64),
            T(wl.cost, torch.float64), T(wl.w_cost, torch.float64),
            T(wl.w_lat_ms, torch.float64))
    ctx.route_trace(*args)
    assert ctx.status() == L.LAR_E_SYNC
    ctx.close()
    choice, chosen, util, ctx = gpu_trace(wl)
    ref = O.trace(wl)
    np.testing.assert_array_equal(choice[0], ref.choice)
    ctx.close()


@pytest.mark.parametrize("mcap,kernel", [(100, "2 slots per lane"), (300, "8 slots per lane"),
                                         (1024, "16 slots per lane: HBM-state kernel")])
@pytest.mark.parametrize("seed", range(3))
def test_trace_slot_widths(mcap, kernel, seed):
    """The trace kernels instantiated for wider decode-slot arrays (the context's
    max_seqs_cap sets the slots per lane): tiny pools routed in contexts of 100, 300
    and 1024 sequence slots give the oracle's results."""
    wl = make_tiny_workload(500 + seed, n_inst=5, max_res=6, n_q=40, n_scen=2,
                            dyadic=(seed % 2 == 0))
    choice, chosen, util, ctx = gpu_trace(wl, queue_cap=10 ** 4, max_seqs_cap=mcap)
    for z in range(wl.n_scen):
        ref = O.trace(wl, scenario=z, queue_cap=10 ** 4)
        np.testing.assert_array_equal(choice[z], ref.choice)
        np.testing.assert_array_equal(bits(chosen[z]), bits(ref.ttft_chosen))
        np.testing.assert_array_equal(bits(util[z]), bits(ref.util_chosen))
        assert_state_equal(ctx, z, ref)
    ctx.close()


@pytest.mark.parametrize("seed", range(10))
@pytest.mark.parametrize("flags", [0, 1])
def test_trace_fast_walk_tiny_pools(seed, flags):
    """Queues of 8 decode slots per lane take the fast walk (a query joining an
    instance at its cached admission point is folded over the cached decode-only
    batches).  Tiny random pools with backlogs -- budgets of 1..8 tokens, 1..4
    sequences, prompts up to 40 tokens and 1..3 decode tokens, so that a query
    often completes its prefill, or even its decodes, inside the fold -- against the
    oracle, both first-token readings, all coefficient terms."""
    wl = make_tiny_workload(700 + seed, n_inst=3, max_res=8, n_q=60, prompt=(1, 40),
                            decode=(1, 3), mean_gap_ms=0.5, n_scen=2, dyadic=(seed % 2 == 0))
    choice, chosen, util, ctx = gpu_trace(wl, flags=flags, queue_cap=10 ** 4, max_seqs_cap=300)
    for z in range(wl.n_scen):
        ref = O.trace(wl, scenario=z, reading=flags, queue_cap=10 ** 4)
        np.testing.assert_array_equal(choice[z], ref.choice)
        np.testing.assert_array_equal(bits(chosen[z]), bits(ref.ttft_chosen))
        np.testing.assert_array_equal(bits(util[z]), bits(ref.util_chosen))
        assert_state_equal(ctx, z, ref)
    ctx.close()


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("flags", [0, 1])
def test_trace_fast_walk_shifted_tails(seed, flags):
    """Queues of 8 decode slots per lane, with a decode-only tail of only a few batches
    (short prompts against budgets of 6..8 tokens): the tail of the admission point a
    query is walked to is then taken from the previous one by a shift while the 64
    held batches last, and afresh when they run out (every couple of dozen walks).
    Long traces on two instances with 1..3-token decodes, so queries are still in the
    list, decoding, or done at the new admission point; arrivals every 0.4 ms (a
    growing backlog), 1.5 ms or 3 ms (the query often admitted at once, a shift of
    zero batches); against the oracle, both first-token readings."""
    wl = make_tiny_workload(900 + seed, n_inst=2, max_res=8, n_q=400, prompt=(1, 8),
                            decode=(1, 3), budget=(6, 8), max_seqs=(1, 3),
                            mean_gap_ms=(0.4, 1.5, 3.0)[seed % 3], n_scen=2,
                            dyadic=(seed % 2 == 0))
    assert _tail_k(wl) <= 4
    choice, chosen, util, ctx = gpu_trace(wl, flags=flags, queue_cap=10 ** 4, max_seqs_cap=300)
    for z in range(wl.n_scen):
        ref = O.trace(wl, scenario=z, reading=flags, queue_cap=10 ** 4)
        np.testing.assert_array_equal(choice[z], ref.choice)
        np.testing.assert_array_equal(bits(chosen[z]), bits(ref.ttft_chosen))
        np.testing.assert_array_equal(bits(util[z]), bits(ref.util_chosen))
        assert_state_equal(ctx, z, ref)
    ctx.close()


@pytest.mark.parametrize("reading", [0, 1])
def test_exhaustive_tiny_states_one_context(reading):
    """Every tiny state of the oracle's exhaustive pins (up to 3 residents of every
    kind, six (B, M) shapes) as the instances of one context: the what-if estimates
    (shared trajectory, k_traj + k_est) of three prompts at every instance, then a
    replay of every instance to t = 6 ms, against the oracle instance by instance."""
    from paper_2607_18253_amd.lar import LarContext
    import test_oracle_pins as TP
    coef = dict(a=0.75, b=0.3, c=0.2, d=0.01, e=0.003)
    cases = [(reqs, B, M) for reqs, n_run in TP._tiny_states()
             for B, M in [(1, 1), (2, 1), (2, 2), (3, 2), (4, 3), (4, 1)] if n_run <= M]
    I = len(cases)
    offsets = np.zeros(I + 1, np.int32)
    rp, rd, cx = [], [], []
    for j, (reqs, B, M) in enumerate(cases):
        offsets[j + 1] = offsets[j] + len(reqs)
        for r in reqs:
            rp.append(r[0]); rd.append(r[1]); cx.append(r[2])
    ctx = LarContext(1, I, max_seqs_cap=3, queue_cap=8, max_prompt=5, flags=reading)
    ctx.load_state(a=[coef["a"]] * I, b=[coef["b"]] * I, c=[coef["c"]] * I,
                   d=[coef["d"]] * I, e=[coef["e"]] * I, budget=[B for _, B, _ in cases],
                   max_seqs=[M for _, _, M in cases], col=[0] * I, offsets=offsets,
                   rem_prefill=np.array(rp, np.int32), rem_decode=np.array(rd, np.int32),
                   context=np.array(cx, np.int32), clock_ms=np.zeros(I))
    ps = [1, 2, 5]
    tt, it = ctx.estimate(T(np.array(ps), torch.int32), 0.0)
    ctx.advance(6.0)
    ctx.sync()
    tt, it = tt.cpu().numpy()[0], it.cpu().numpy()[0]
    st = ctx.read_state(0)
    ctx.close()
    for j, (reqs, B, M) in enumerate(cases):
        q = TP._queue(coef, B, M, reqs)
        for a, p in enumerate(ps):
            want, wit = q.estimate(p, 1, 0.0, reading)
            assert bits(tt[a, j]) == bits(want) and it[a, j] == wit, (reqs, B, M, p)
        q.advance(6.0)
        grp, grd, gcx, gclk, gits = q.state()
        lo, hi = st["offsets"][j], st["offsets"][j + 1]
        assert list(st["rem_prefill"][lo:hi]) == list(grp), (reqs, B, M)
        assert list(st["rem_decode"][lo:hi]) == list(grd), (reqs, B, M)
        assert list(st["context"][lo:hi]) == list(gcx), (reqs, B, M)
        assert bits(st["clock_ms"][j]) == bits(gclk) and st["iterations"][j] == gits
