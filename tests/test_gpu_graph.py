"""lar_route_step captured once in a HIP graph (torch.cuda.graph on the context's
stream) and replayed per query, the query's values written into the same device
buffers between replays: every replay's choice and chosen TTFT equal the oracle's
sequential trace, under both objectives, with the host's own eager work and a
synchronisation between replays."""

from __future__ import annotations

import os
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
from gpu_util import assert_state_equal, bits  # noqa: E402
from oracle import oracle as O  # noqa: E402
from paper_2607_18253_amd import context_for  # noqa: E402
from workloads import make_workload  # noqa: E402


@pytest.mark.parametrize("objective,workload", [("lagrangian", "c2"), ("constrained", "c2"),
                                                ("lagrangian", "c7")])
def test_route_step_graph_replays(objective, workload):
    """c7 runs the same step under scheduler limits (KV blocks, chunk cap, context
    limit): what-if, route and commit of the limits engine in the graph."""
    wl = make_workload(workload, n_q=400, n_inst=8)
    N, dev = wl.n_q, "cuda:0"
    tau = O.ttft_targets(wl.q_prefill, wl.tau_u_ms, wl.tau_v) if objective == "constrained" else None
    ref = O.trace(wl, tau=tau)
    s = torch.cuda.Stream()
    f64 = dict(dtype=torch.float64, device=dev)
    i32 = dict(dtype=torch.int32, device=dev)
    qp, qd = torch.zeros(1, **i32), torch.zeros(1, **i32)
    t, tn = torch.zeros(1, **f64), torch.zeros(1, **f64)
    acc, cost = torch.zeros(wl.n_cols, **f64), torch.zeros(wl.n_cols, **f64)
    tq = torch.zeros(1, **f64)
    wc = torch.as_tensor(wl.w_cost, **f64)
    wlat = torch.as_tensor(wl.w_lat_ms, **f64)
    choice, chosen = torch.zeros(1, **i32), torch.zeros(1, **f64)
    ctx = context_for(wl, stream=s)
    with torch.cuda.stream(s):
        ctx.advance(float(wl.q_t_ms[0]))
    s.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        ctx.route_step(qp, qd, t, tn, acc, cost, wc, w_lat=None if tau is not None else wlat,
                       tau_ms=tq if tau is not None else None, choice=choice,
                       chosen_ttft=chosen)
    for i in range(N):
        t_next = float(wl.q_t_ms[i + 1]) if i + 1 < N else float(wl.q_t_ms[i])
        with torch.cuda.stream(s):
            qp.fill_(int(wl.q_prefill[i]))
            qd.fill_(int(wl.q_decode[i]))
            t.fill_(float(wl.q_t_ms[i]))
            tn.fill_(t_next)
            acc.copy_(torch.as_tensor(wl.acc[i], **f64))
            cost.copy_(torch.as_tensor(wl.cost[i], **f64))
            if tau is not None:
                tq.fill_(float(tau[i]))
            g.replay()
        s.synchronize()
        assert int(choice.item()) == int(ref.choice[i]), i
        assert bits(chosen.cpu().numpy())[0] == bits(ref.ttft_chosen[i:i + 1])[0], i
    ctx.sync()
    assert_state_equal(ctx, 0, ref)
    ctx.close()
