"""GPU parity of the scheduler limits (chunk cap, context limit, KV-cache blocks with
recompute preemption; the system appendix lists them among what the SFS simulation
follows) against the oracle, bit for bit: traces under both objectives and both
readings with realised TTFT, what-if estimates, single routing steps, final states;
and the limits engine with every limit off against the default engine."""

from __future__ import annotations

import os
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
from gpu_util import DEV, T, assert_state_equal, bits  # noqa: E402
from oracle import oracle as O  # noqa: E402
from paper_2607_18253_amd import context_for  # noqa: E402
from workloads import make_tiny_workload, make_workload  # noqa: E402
from workloads.gen import make_tiny_sched_workload  # noqa: E402

MAX_ITERS = 200_000   # bounds every estimate and replay call of these tests


def _trace(wl, n_q=None, *, flags=0, tau=None, realized=True, max_seqs_cap=None):
    N = wl.n_q if n_q is None else int(n_q)
    ctx = context_for(wl, flags=flags, max_iters=MAX_ITERS, max_seqs_cap=max_seqs_cap)
    ctx.advance(float(wl.q_t_ms[0]))
    Z = wl.n_scen
    chosen = torch.full((Z, N), -1.0, dtype=torch.float64, device=DEV)
    util = torch.full((Z, N), -1.0, dtype=torch.float64, device=DEV)
    real = torch.full((Z, N), -1.0, dtype=torch.float64, device=DEV) if realized else None
    args = (T(wl.q_prefill[:N], torch.int32), T(wl.q_decode[:N], torch.int32),
            T(wl.q_t_ms[:N], torch.float64), float(wl.q_t_ms[N - 1]))
    if tau is None:
        choice = ctx.route_trace(*args, T(wl.acc[:N], torch.float64),
                                 T(wl.cost[:N], torch.float64), T(wl.w_cost, torch.float64),
                                 T(wl.w_lat_ms, torch.float64), chosen_ttft=chosen,
                                 utility=util, realized=real)
    else:
        choice = ctx.route_trace_constrained(*args, T(tau[:N], torch.float64),
                                             T(wl.acc[:N], torch.float64),
                                             T(wl.cost[:N], torch.float64),
                                             T(wl.w_cost, torch.float64), chosen_ttft=chosen,
                                             utility=util, realized=real)
    ctx.sync()
    return (choice.cpu().numpy(), chosen.cpu().numpy(), util.cpu().numpy(),
            None if real is None else real.cpu().numpy(), ctx)


def _check(wl, got, *, reading=0, tau=None, scenarios=(0,), state=(0,)):
    choice, chosen, util, real, ctx = got
    N = choice.shape[1]
    for z in scenarios:
        ref = O.trace(wl, scenario=z, n_q=N, reading=reading, tau=tau, max_iters=MAX_ITERS,
                      final_state=z in state)
        np.testing.assert_array_equal(choice[z], ref.choice, err_msg=f"{wl.name} scenario {z}")
        np.testing.assert_array_equal(bits(chosen[z]), bits(ref.ttft_chosen),
                                      err_msg=f"{wl.name} scenario {z}")
        np.testing.assert_array_equal(bits(util[z]), bits(ref.util_chosen))
        if real is not None:
            np.testing.assert_array_equal(bits(real[z]), bits(ref.realized),
                                          err_msg=f"{wl.name} realised, scenario {z}")
        if z in state:
            assert_state_equal(ctx, z, ref)
    ctx.close()


@pytest.mark.parametrize("seed", range(16))
def test_limits_tiny_pools(seed):
    wl = make_tiny_sched_workload(seed, n_q=25, max_res=5)
    reading = seed % 2
    print(f"tiny limits seed {seed} reading {reading}", flush=True)
    _check(wl, _trace(wl, flags=reading), reading=reading)


@pytest.mark.parametrize("n_q", [1, 63, 64, 65, 128, 129])
def test_limits_trace_query_block_boundaries(n_q):
    """The clustered limits trace reads the queries in blocks of 64 as the default
    one does: traces at and around one and two blocks, 9 instances (three
    workgroups per scenario), two scenarios, realised TTFT tracked and untracked."""
    wl = make_tiny_sched_workload(300 + n_q, n_inst=9, n_q=n_q, max_res=5, n_scen=2)
    print(f"limits block boundary n_q {n_q}", flush=True)
    _check(wl, _trace(wl, realized=n_q % 2 == 1), scenarios=(0, 1), state=(0, 1))


@pytest.mark.parametrize("seed", range(8))
def test_limits_tiny_pools_constrained(seed):
    wl = make_tiny_sched_workload(100 + seed, n_q=25, max_res=5)
    tau = np.random.default_rng(seed).uniform(0.0, 40.0, size=wl.n_q)
    print(f"tiny limits constrained seed {seed}", flush=True)
    _check(wl, _trace(wl, tau=tau), tau=tau)


@pytest.mark.parametrize("seed,cap", [(0, None), (1, 100), (2, 200), (3, 300), (4, 1000)])
def test_limits_tiny_pools_scenarios_and_wide_slots(seed, cap):
    """Several scenarios at once; every slot width (64, 128, 256, 512, 1024 entries in
    registers) through a larger max_seqs_cap."""
    wl = make_tiny_sched_workload(200 + seed, n_q=20, max_res=6, n_scen=3)
    print(f"tiny limits scenarios seed {seed} cap {cap}", flush=True)
    _check(wl, _trace(wl, max_seqs_cap=cap), scenarios=(0, 1, 2), state=(0, 2))


@pytest.mark.parametrize("seed", range(6))
def test_limits_off_equals_default_engine(seed):
    """The limits engine with every limit 0 against the default engine and the oracle."""
    wl = make_tiny_workload(seed, n_q=30)
    base = _trace(wl, realized=True)
    ref_c, ref_t = base[0].copy(), base[1].copy()
    base[4].close()
    wl.sched = np.zeros((wl.n_inst, 4), np.int32)
    got = _trace(wl, realized=True)
    np.testing.assert_array_equal(got[0], ref_c)
    np.testing.assert_array_equal(bits(got[1]), bits(ref_t))
    _check(wl, got)


@pytest.mark.parametrize("seed", range(6))
def test_limits_what_if_matrix(seed):
    """lar_estimate_ttft under limits: every (query, instance) pair against the
    oracle's literal estimate, after a replay to a common time."""
    wl = make_tiny_sched_workload(300 + seed, n_q=12, max_res=6)
    reading = seed % 2
    ctx = context_for(wl, flags=reading, max_iters=MAX_ITERS)
    t = float(wl.q_t_ms[3])
    ctx.advance(t)
    qp = T(wl.q_prefill, torch.int32)
    ttft, _ = ctx.estimate(qp, t)
    ctx.sync()
    got = ttft.cpu().numpy().reshape(wl.n_q, wl.n_inst)
    for j in range(wl.n_inst):
        q = O.instance_queue(wl, j)
        q.advance(t, max_iters=MAX_ITERS)
        for i in range(wl.n_q):
            want, _ = q.estimate(int(wl.q_prefill[i]), 1, t, reading)
            assert bits(got[i, j]) == bits(want), (seed, i, j)
    ctx.close()


def test_limits_commit_and_route_step():
    """Single routing steps (lar_route_step) and plain commits under limits follow the
    oracle's trace."""
    wl = make_tiny_sched_workload(400, n_q=30, max_res=5)
    ref = O.trace(wl, max_iters=MAX_ITERS)
    ctx = context_for(wl, max_iters=MAX_ITERS)
    ctx.advance(float(wl.q_t_ms[0]))
    got = []
    for i in range(wl.n_q):
        tn = float(wl.q_t_ms[i + 1]) if i + 1 < wl.n_q else float(wl.q_t_ms[i])
        c = ctx.route_step(T(wl.q_prefill[i:i + 1], torch.int32),
                           T(wl.q_decode[i:i + 1], torch.int32),
                           T(wl.q_t_ms[i:i + 1], torch.float64),
                           T(np.array([tn]), torch.float64), T(wl.acc[i:i + 1], torch.float64),
                           T(wl.cost[i:i + 1], torch.float64), T(wl.w_cost, torch.float64),
                           T(wl.w_lat_ms, torch.float64))
        got.append(int(c.cpu().numpy().reshape(-1)[0]))
    ctx.sync()
    np.testing.assert_array_equal(np.array(got), ref.choice)
    assert_state_equal(ctx, 0, ref)
    ctx.close()


def test_limits_c7_prefix():
    """The c7 pool (32 instances, 512-token chunks, 16-token KV blocks, 8192-token
    context limit), its first 3000 queries: the initial backlog, where the KV cache
    preempts."""
    wl = make_workload("c7", n_q=3000)
    print("c7 prefix 3000", flush=True)
    _check(wl, _trace(wl))


def test_limits_c7_prefix_reading_prefill_constrained():
    wl = make_workload("c7", n_q=1500)
    tau = O.ttft_targets(wl.q_prefill, wl.tau_u_ms, wl.tau_v)
    print("c7 prefix 1500 constrained reading 1", flush=True)
    _check(wl, _trace(wl, flags=1, tau=tau), reading=1, tau=tau)


def test_limits_c7_full():
    """The whole c7 trace (100k queries, 32 instances) in the launch configuration the
    benchmark times, with realised TTFT: every choice, chosen TTFT, utility and
    realised-TTFT bit and the final state equal the oracle's."""
    wl = make_workload("c7")
    print("c7 full", flush=True)
    _check(wl, _trace(wl))


def test_limits_c7_full_constrained_ontime():
    """The whole c7 trace under Eq. 3 with the paper's targets; OnTimeUtility from the
    realised TTFTs."""
    wl = make_workload("c7")
    tau = O.ttft_targets(wl.q_prefill, wl.tau_u_ms, wl.tau_v)
    print("c7 full constrained", flush=True)
    got = _trace(wl, tau=tau)
    choice, real, ctx = got[0], got[3], got[4]
    out = ctx.ontime_utility(T(choice, torch.int32), T(real, torch.float64),
                             T(tau, torch.float64), T(wl.acc, torch.float64),
                             T(wl.cost, torch.float64), T(wl.w_cost, torch.float64))
    ctx.sync()
    ref = O.trace(wl, tau=tau, max_iters=MAX_ITERS, final_state=False)
    want = O.ontime_utility(ref.choice, ref.realized, tau, wl.acc, wl.cost, wl.col, wl.w_cost[0])
    assert bits(out.cpu().numpy())[0] == bits(np.array([want]))[0]
    _check(wl, got, tau=tau)


def test_limits_error_paths():
    """Bad limits are rejected with nothing changed; calls between lar_set_scheduler and
    the next load report LAR_E_STATE; a snapshot breaking the limits is LAR_E_STATE; a
    query whose prompt does not fit the context limit sets the sticky LAR_E_ARG."""
    from paper_2607_18253_amd.lar import LAR_E_ARG, LAR_E_STATE, LarError
    wl = make_tiny_sched_workload(7, n_q=6, max_res=4)
    ctx = context_for(wl, max_iters=MAX_ITERS)
    bad = wl.sched.copy()
    bad[0] = (0, 4, 3, 8)          # block size not a power of two
    with pytest.raises(LarError) as e:
        ctx.set_scheduler(bad)
    assert e.value.code == LAR_E_ARG
    bad[0] = (0, 2, 2, 8)          # 2 blocks of 2 tokens < context limit 8
    with pytest.raises(LarError) as e:
        ctx.set_scheduler(bad)
    assert e.value.code == LAR_E_ARG
    bad[0] = (0, 4, 2, 0)          # a KV cache without a context limit
    with pytest.raises(LarError) as e:
        ctx.set_scheduler(bad)
    assert e.value.code == LAR_E_ARG
    ctx.advance(float(wl.q_t_ms[0]))   # the context is unchanged: still loaded
    ctx.sync()
    ctx.set_scheduler(wl.sched)    # valid: the state must be loaded again
    with pytest.raises(LarError) as e:
        ctx.advance(float(wl.q_t_ms[0]))
    assert e.value.code == LAR_E_STATE
    tight = wl.sched.copy()
    rp, rd, cx = wl.instance_requests(0)
    tight[0, 3] = int((rp + cx).max())   # a resident at the context limit
    tight[0, 1] = 0
    if len(rp):
        ctx.set_scheduler(tight)
        with pytest.raises(LarError) as e:
            ctx.load_workload(wl)
        assert e.value.code == LAR_E_STATE
    ctx.set_scheduler(wl.sched)
    ctx.load_workload(wl)
    ctx.advance(float(wl.q_t_ms[0]))
    ctx.sync()
    ctx.close()


def test_mixed_context_limits():
    """A pool mixing a small context limit (instance 0, the best choice whenever it
    can take a query) with larger ones: the what-if estimate is +inf exactly where
    the limit cannot hold the prompt, the route skips those instances, and the trace
    (both objectives) is the oracle's; a query that no instance can take is routed
    nowhere with the sticky LAR_E_ARG, the queries before it as the oracle routes
    them."""
    from paper_2607_18253_amd.lar import LAR_E_ARG
    from test_oracle_sched import _mixed_limit_pool
    wl = _mixed_limit_pool()
    ctx = context_for(wl, max_iters=MAX_ITERS)
    assert (wl.clock_ms == 0.0).all()
    tt, it = ctx.estimate(T(wl.q_prefill, torch.int32), 0.0)
    ch = ctx.route(tt, T(wl.acc, torch.float64), T(wl.cost, torch.float64),
                   T(wl.w_cost, torch.float64), T(wl.w_lat_ms, torch.float64))
    assert ctx.status() == 0
    tt, it, ch = tt.cpu().numpy()[0], it.cpu().numpy()[0], ch.cpu().numpy()[0]
    ref = O.estimate_matrix(wl, range(wl.n_q), range(wl.n_inst), 0.0)
    np.testing.assert_array_equal(bits(tt), bits(ref[0]))
    np.testing.assert_array_equal(it, ref[1])
    assert np.isinf(tt[:, 0]).sum() > 5
    for i in range(wl.n_q):
        m, _ = O.route_row(ref[0][i], wl.acc[i], wl.cost[i], wl.col, wl.w_cost[0],
                           wl.w_lat_ms[0])
        assert ch[i] == m, i
    ctx.close()
    tau = O.ttft_targets(wl.q_prefill, wl.tau_u_ms, wl.tau_v)
    for t in (None, tau):
        _check(wl, _trace(wl, tau=t), tau=t)
    # a query at every instance's limit
    wl.q_prefill[4] = 64
    ctx = context_for(wl, max_iters=MAX_ITERS)
    ctx.advance(float(wl.q_t_ms[0]))
    chosen = torch.full((1, wl.n_q), -1.0, dtype=torch.float64, device=DEV)
    choice = ctx.route_trace(T(wl.q_prefill, torch.int32), T(wl.q_decode, torch.int32),
                             T(wl.q_t_ms, torch.float64), float(wl.q_t_ms[-1]),
                             T(wl.acc, torch.float64), T(wl.cost, torch.float64),
                             T(wl.w_cost, torch.float64), T(wl.w_lat_ms, torch.float64),
                             chosen_ttft=chosen)
    assert ctx.status() == LAR_E_ARG
    choice, chosen = choice.cpu().numpy(), chosen.cpu().numpy()
    ref = O.trace(wl, n_q=4)
    np.testing.assert_array_equal(choice[0, :4], ref.choice)
    np.testing.assert_array_equal(bits(chosen[0, :4]), bits(ref.ttft_chosen))
    assert choice[0, 4] == -1
    ctx.close()


def test_mixed_context_limits_whole_workgroup():
    """Twelve instances, three workgroups of four: the first workgroup's instances
    have a small context limit and the best accuracy, so for prompts beyond it that
    whole workgroup has no candidate and posts none while the others do; for shorter
    prompts it usually holds the winner.  Trace under both objectives against the
    oracle."""
    rng = np.random.default_rng(17)
    for seed in range(40, 80):
        wl = make_tiny_sched_workload(seed, n_inst=12, n_q=60, max_res=3)
        wl.sched[:, 1] = 0                 # no KV cache (the limit then needs no blocks)
        wl.sched[:, 3] = 64
        wl.sched[:4, 3] = 24
        if all(len(rp) == 0 or (rp + cx).max() < wl.sched[j, 3]
               for j, (rp, _, cx) in ((j, wl.instance_requests(j)) for j in range(12))):
            break
    else:
        pytest.fail("no seed whose residents fit the limits")
    wl.col[:] = np.arange(12) % wl.acc.shape[1]
    wl.acc[:, :] = 0.1
    wl.acc[:, wl.col[0]] = 0.9
    wl.col[4:] = (wl.col[0] + 1) % wl.acc.shape[1]   # the first workgroup alone has the best column
    wl.q_prefill[:] = rng.integers(1, 40, wl.n_q)    # many do not fit the first workgroup's limit
    wl.max_prompt = 64
    assert (wl.q_prefill >= 24).sum() > 10 and (wl.q_prefill < 24).sum() > 10
    tau = O.ttft_targets(wl.q_prefill, wl.tau_u_ms, wl.tau_v)
    for t in (None, tau):
        _check(wl, _trace(wl, tau=t), tau=t)


def test_limits_reload_repeat():
    """The benchmark's step under limits: reload the snapshot, replay to the first
    arrival, trace; two steps give the oracle's results both times."""
    wl = make_workload("c7", n_q=2000, n_inst=16)
    ref = O.trace(wl, max_iters=MAX_ITERS)
    ctx = context_for(wl, max_iters=MAX_ITERS)
    N = wl.n_q
    for rep in range(2):
        ctx.reload_state()
        ctx.advance(float(wl.q_t_ms[0]))
        chosen = torch.full((1, N), -1.0, dtype=torch.float64, device=DEV)
        choice = ctx.route_trace(T(wl.q_prefill, torch.int32), T(wl.q_decode, torch.int32),
                                 T(wl.q_t_ms, torch.float64), float(wl.q_t_ms[-1]),
                                 T(wl.acc, torch.float64), T(wl.cost, torch.float64),
                                 T(wl.w_cost, torch.float64), T(wl.w_lat_ms, torch.float64),
                                 chosen_ttft=chosen)
        ctx.sync()
        np.testing.assert_array_equal(choice.cpu().numpy()[0], ref.choice, err_msg=f"step {rep}")
        np.testing.assert_array_equal(bits(chosen.cpu().numpy()[0]), bits(ref.ttft_chosen))
        assert_state_equal(ctx, 0, ref)
    ctx.close()


def test_limits_capacity_and_iteration_cap():
    """Under limits, a full waiting queue is a sticky LAR_E_CAPACITY and an estimate or
    replay past max_iters a sticky LAR_E_ITER, as the oracle reports them."""
    from paper_2607_18253_amd.lar import LAR_E_CAPACITY, LAR_E_ITER, LarError
    wl = make_workload("c7", n_q=300, n_inst=4)
    ref_err = None
    try:
        O.trace(wl, queue_cap=130, max_iters=MAX_ITERS)
    except O.OracleError as e:
        ref_err = e.code
    assert ref_err == O.E_CAPACITY
    ctx = context_for(wl, max_iters=MAX_ITERS, queue_cap=130)
    ctx.advance(float(wl.q_t_ms[0]))
    with pytest.raises(LarError) as e:
        ctx.route_trace(T(wl.q_prefill, torch.int32), T(wl.q_decode, torch.int32),
                        T(wl.q_t_ms, torch.float64), float(wl.q_t_ms[-1]),
                        T(wl.acc, torch.float64), T(wl.cost, torch.float64),
                        T(wl.w_cost, torch.float64), T(wl.w_lat_ms, torch.float64))
        ctx.sync()
    assert e.value.code == LAR_E_CAPACITY
    ctx.close()
    # an estimate of the first query needs more batches than the cap allows
    with pytest.raises(O.OracleError) as oe:
        O.trace(wl, n_q=1, max_iters=5)
    assert oe.value.code == O.E_ITER
    ctx = context_for(wl, max_iters=5)
    ctx.advance(float(wl.q_t_ms[0]))
    with pytest.raises(LarError) as e:
        ctx.route_trace(T(wl.q_prefill[:1], torch.int32), T(wl.q_decode[:1], torch.int32),
                        T(wl.q_t_ms[:1], torch.float64), float(wl.q_t_ms[0]),
                        T(wl.acc[:1], torch.float64), T(wl.cost[:1], torch.float64),
                        T(wl.w_cost, torch.float64), T(wl.w_lat_ms, torch.float64))
        ctx.sync()
    assert e.value.code == LAR_E_ITER
    ctx.close()


@pytest.mark.parametrize("reading", [0, 1])
def test_limits_exhaustive_tiny_states(reading):
    """Every tiny state of the CPU pins (up to 3 residents of every kind, three (B, M)
    shapes, six limit settings: about 24k cases) as the instances of one context: the
    what-if estimates of two prompts at every instance, then a replay of every instance
    to t = 6 ms, against the oracle instance by instance."""
    from paper_2607_18253_amd.lar import LarContext
    import test_oracle_sched as TS
    coef = dict(a=0.75, b=0.3, c=0.2, d=0.01, e=0.003)
    cases = list(TS._sched_cases(stride=1))
    I = len(cases)
    offsets = np.zeros(I + 1, np.int32)
    rp, rd, cx = [], [], []
    for j, (reqs, B, M, lim) in enumerate(cases):
        offsets[j + 1] = offsets[j] + len(reqs)
        for r in reqs:
            rp.append(r[0]); rd.append(r[1]); cx.append(r[2])
    ctx = LarContext(1, I, max_seqs_cap=3, queue_cap=8, max_prompt=4, flags=reading,
                     max_iters=MAX_ITERS)
    ctx.set_scheduler(np.array([lim for _, _, _, lim in cases], np.int32))
    ctx.load_state(a=[coef["a"]] * I, b=[coef["b"]] * I, c=[coef["c"]] * I,
                   d=[coef["d"]] * I, e=[coef["e"]] * I,
                   budget=[B for _, B, _, _ in cases], max_seqs=[M for _, _, M, _ in cases],
                   col=[0] * I, offsets=offsets, rem_prefill=np.array(rp, np.int32),
                   rem_decode=np.array(rd, np.int32), context=np.array(cx, np.int32),
                   clock_ms=np.zeros(I))
    ps = [1, 4]
    tt, it = ctx.estimate(T(np.array(ps), torch.int32), 0.0)
    ctx.advance(6.0)
    ctx.sync()
    tt, it = tt.cpu().numpy()[0], it.cpu().numpy()[0]
    st = ctx.read_state(0)
    ctx.close()
    for j, (reqs, B, M, lim) in enumerate(cases):
        q = TS._queue(coef, B, M, reqs, lim)
        for a, p in enumerate(ps):
            want, wit = q.estimate(p, 1, 0.0, reading)
            assert bits(tt[a, j]) == bits(want) and it[a, j] == wit, (reqs, B, M, lim, p)
        q.advance(6.0)
        grp, grd, gcx, gclk, gits = q.state()
        lo, hi = st["offsets"][j], st["offsets"][j + 1]
        assert list(st["rem_prefill"][lo:hi]) == list(grp), (reqs, B, M, lim)
        assert list(st["rem_decode"][lo:hi]) == list(grd), (reqs, B, M, lim)
        assert list(st["context"][lo:hi]) == list(gcx), (reqs, B, M, lim)
        assert bits(st["clock_ms"][j]) == bits(gclk) and st["iterations"][j] == gits


def test_limits_prompt_at_the_context_boundary():
    """A prompt of X - 1 tokens fits an instance with context limit X (its decode is cut
    to 1): estimated at every instance as the oracle does, under both readings."""
    for reading in (0, 1):
        wl = make_tiny_sched_workload(9, n_q=4, max_res=4)
        wl.sched[:, 3] = np.maximum(wl.sched[:, 3], 14)
        K, S, Xs = wl.sched[:, 1], wl.sched[:, 2], wl.sched[:, 3]
        wl.sched[:, 1] = np.where(K > 0, np.maximum(K, -(-Xs // S)), 0)   # K*S >= X
        X = int(wl.sched[:, 3].min())
        wl.max_prompt = X
        ctx = context_for(wl, flags=reading, max_iters=MAX_ITERS)
        ps = np.array([X - 1, 1], np.int32)
        tt, it = ctx.estimate(T(ps, torch.int32), 0.0)
        ctx.sync()
        tt, it = tt.cpu().numpy()[0], it.cpu().numpy()[0]
        ctx.close()
        for j in range(wl.n_inst):
            q = O.instance_queue(wl, j)
            for a, p in enumerate(ps):
                want, wit = q.estimate(int(p), 1, 0.0, reading)
                assert bits(tt[a, j]) == bits(want) and it[a, j] == wit, (reading, j, p)
