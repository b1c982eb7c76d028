"""GPU parity of the constrained objective (Eq. 3), the TTFT targets (appendix on
TTFT latency assignment) and OnTimeUtility (Eq. 4) against the CPU oracle.

Choices and final states must match exactly and every fp64 result bit for bit: the
kernels evaluate the same operations in the same order with the same roundings.
"""

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from gpu_util import DEV, T, assert_state_equal, bits, gpu_trace_constrained  # noqa: E402
from oracle import oracle as O  # noqa: E402
from paper_2607_18253_amd import context_for  # noqa: E402
from workloads import make_tiny_workload, make_workload  # noqa: E402


def _gpu_targets(ctx, wl, n=None):
    n = wl.n_q if n is None else n
    tau = ctx.ttft_targets(T(wl.q_prefill[:n], torch.int32), T(wl.tau_u_ms[:n], torch.float64),
                           T(wl.tau_v[:n], torch.float64))
    ctx.sync()
    return tau.cpu().numpy()


def test_ttft_targets_match_oracle():
    """Targets of a 100k-query trace, plus edge inputs that hit both clips."""
    wl = make_workload("c2")
    ctx = context_for(wl, queue_cap=wl.queue_cap)
    got = _gpu_targets(ctx, wl)
    want = O.ttft_targets(wl.q_prefill, wl.tau_u_ms, wl.tau_v)
    np.testing.assert_array_equal(bits(got), bits(want))
    p = np.array([0, 1000, 10 ** 6, 5, 2 ** 31 - 1], np.int32)
    u = np.array([-100.0, 3.0, 1.0, 1.0, 5.0])
    v = np.array([1.0, 1.0, 1.0, 0.98, 1.02])
    got = ctx.ttft_targets(T(p, torch.int32), T(u, torch.float64), T(v, torch.float64))
    ctx.sync()
    np.testing.assert_array_equal(bits(got.cpu().numpy()), bits(O.ttft_targets(p, u, v)))
    ctx.close()


@pytest.mark.parametrize("target", ["paper", "quantile"])
def test_route_constrained_c3(target):
    """Config 3 what-if matrix (1024 instances, 4096 queries): every row's constrained
    choice, chosen TTFT and utility against the oracle's Eq. 3 on the same row.  The
    paper's targets (~150-200 ms) are below every TTFT here, so every row takes the
    least-TTFT fallback; per-row 30% quantile targets make a third of each row
    feasible."""
    wl = make_workload("c3")
    ctx = context_for(wl)
    tt, _ = ctx.estimate(T(wl.q_prefill, torch.int32), 0.0, want_iters=False)
    ctx.sync()
    rows = tt.cpu().numpy()[0]
    if target == "paper":
        tau = _gpu_targets(ctx, wl)
    else:
        tau = np.quantile(rows, 0.3, axis=1, method="lower")
    chosen = torch.empty((1, wl.n_q), dtype=torch.float64, device=DEV)
    util = torch.empty((1, wl.n_q), dtype=torch.float64, device=DEV)
    ch = ctx.route_constrained(tt, T(tau, torch.float64), T(wl.acc, torch.float64),
                               T(wl.cost, torch.float64), T(wl.w_cost, torch.float64),
                               chosen_ttft=chosen, utility=util)
    ctx.sync()
    ch, chosen, util = ch.cpu().numpy()[0], chosen.cpu().numpy()[0], util.cpu().numpy()[0]
    n_feasible_rows = 0
    for i in range(wl.n_q):
        m = O.route_row_constrained(rows[i], tau[i], wl.acc[i], wl.cost[i], wl.col, wl.w_cost[0])
        assert ch[i] == m, i
        assert bits(chosen[i]) == bits(rows[i, m])
        c = wl.col[m]
        assert bits(util[i]) == bits(wl.acc[i, c] - wl.w_cost[0] * wl.cost[i, c])
        n_feasible_rows += bool((rows[i] <= tau[i]).any())
    assert n_feasible_rows == (0 if target == "paper" else wl.n_q)
    ctx.close()


def _tau_within(wl, seed):
    """Targets spread over the range of the trace's Lagrangian TTFTs, so that both
    the feasible branch and the empty-set fallback occur."""
    lam = O.trace(wl, full_rows=True, queue_cap=10 ** 6, final_state=False)
    lo, hi = float(lam.ttft_all.min()), float(lam.ttft_all.max())
    return np.random.default_rng(seed).uniform(lo, hi, size=wl.n_q)


@pytest.mark.parametrize("seed", range(10))
@pytest.mark.parametrize("prompt_max", [12, 60, 300])
def test_trace_constrained_tiny_pools(seed, prompt_max):
    """Whole constrained traces on tiny pools, three scenarios; prompt_max = 300
    takes the HBM-state trace kernel (more than 64 tail batches), the others the
    clustered one."""
    wl = make_tiny_workload(300 + seed, n_inst=5, max_res=6, n_q=30, prompt=(1, prompt_max),
                            budget=(1, 6), max_seqs=(1, 3), n_scen=3, dyadic=(seed % 2 == 0))
    tau = _tau_within(wl, seed)
    choice, chosen, util, ctx = gpu_trace_constrained(wl, tau, queue_cap=10 ** 4)
    for z in range(wl.n_scen):
        ref = O.trace(wl, scenario=z, queue_cap=10 ** 4, tau=tau)
        np.testing.assert_array_equal(choice[z], ref.choice)
        np.testing.assert_array_equal(bits(chosen[z]), bits(ref.ttft_chosen))
        np.testing.assert_array_equal(bits(util[z]), bits(ref.util_chosen))
        assert_state_equal(ctx, z, ref)
    ctx.close()


def test_trace_constrained_c2_prefix_and_ontime():
    """Config 2 (32 instances), first 3000 queries with the paper's targets: the
    initial backlog misses every target, the drained pool meets most of them; then
    OnTimeUtility on the GPU against the oracle's."""
    wl = make_workload("c2", n_q=3000)
    ctx0 = context_for(wl)
    tau = _gpu_targets(ctx0, wl)
    ctx0.close()
    np.testing.assert_array_equal(bits(tau), bits(O.ttft_targets(wl.q_prefill, wl.tau_u_ms,
                                                                   wl.tau_v)))
    choice, chosen, util, ctx = gpu_trace_constrained(wl, tau)
    ref = O.trace(wl, tau=tau)
    np.testing.assert_array_equal(choice[0], ref.choice)
    np.testing.assert_array_equal(bits(chosen[0]), bits(ref.ttft_chosen))
    np.testing.assert_array_equal(bits(util[0]), bits(ref.util_chosen))
    assert_state_equal(ctx, 0, ref)
    on = ref.ttft_chosen <= tau
    assert 0.05 < on.mean() < 0.95, on.mean()
    # OnTimeUtility's arithmetic on the same per-query TTFTs (here the oracle's
    # realised ones; the trace's own are checked with the realised-TTFT tests)
    got = ctx.ontime_utility(T(choice, torch.int32), T(ref.realized[None, :], torch.float64),
                             T(tau, torch.float64), T(wl.acc, torch.float64),
                             T(wl.cost, torch.float64), T(wl.w_cost, torch.float64))
    ctx.sync()
    want = O.ontime_utility(ref.choice, ref.realized, tau, wl.acc, wl.cost, wl.col,
                            wl.w_cost[0])
    assert bits(got.cpu().numpy()[0]) == bits(want)
    ctx.close()


def test_trace_constrained_c5_scenarios_prefix():
    """Config 5: 64 scenarios x 64 instances (16-wave workgroups, 4 per scenario),
    first 24 queries under the paper's targets, every scenario checked."""
    wl = make_workload("c5", n_q=24)
    tau = O.ttft_targets(wl.q_prefill, wl.tau_u_ms, wl.tau_v)
    choice, chosen, util, ctx = gpu_trace_constrained(wl, tau)
    for z in range(wl.n_scen):
        ref = O.trace(wl, scenario=z, tau=tau, final_state=(z in (0, 63)))
        np.testing.assert_array_equal(choice[z], ref.choice, err_msg=f"scenario {z}")
        np.testing.assert_array_equal(bits(chosen[z]), bits(ref.ttft_chosen))
        if z in (0, 63):
            assert_state_equal(ctx, z, ref)
    ctx.close()
