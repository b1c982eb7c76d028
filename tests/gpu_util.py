"""Helpers for the GPU parity tests: run the HIP path through the C ABI."""

from __future__ import annotations

import numpy as np

DEV = "cuda:0"


def T(a, dtype):
    import torch
    return torch.as_tensor(np.ascontiguousarray(a), dtype=dtype, device=DEV)


def bits(x):
    return np.ascontiguousarray(x, dtype=np.float64).view(np.int64)


def gpu_trace(wl, n_q=None, *, flags=0, max_iters=10_000_000, queue_cap=None,
              max_seqs_cap=None):
    """Sequential trace of every scenario of ``wl`` on the GPU (first n_q queries).

    Returns (choice [Z][N], chosen_ttft [Z][N], utility [Z][N], ctx) with ctx still
    open so the caller can read the final state."""
    import torch
    from paper_2607_18253_amd import context_for

    N = wl.n_q if n_q is None else int(n_q)
    ctx = context_for(wl, flags=flags, max_iters=max_iters, queue_cap=queue_cap,
                      max_seqs_cap=max_seqs_cap)
    ctx.advance(float(wl.q_t_ms[0]))
    chosen = torch.full((wl.n_scen, N), -1.0, dtype=torch.float64, device=DEV)
    util = torch.full((wl.n_scen, N), -1.0, dtype=torch.float64, device=DEV)
    choice = ctx.route_trace(T(wl.q_prefill[:N], torch.int32), T(wl.q_decode[:N], torch.int32),
                             T(wl.q_t_ms[:N], torch.float64), float(wl.q_t_ms[N - 1]),
                             T(wl.acc[:N], torch.float64), T(wl.cost[:N], torch.float64),
                             T(wl.w_cost, torch.float64), T(wl.w_lat_ms, torch.float64),
                             chosen_ttft=chosen, utility=util)
    ctx.sync()
    return choice.cpu().numpy(), chosen.cpu().numpy(), util.cpu().numpy(), ctx


def assert_state_equal(ctx, scen, ref):
    st = ctx.read_state(scen)
    np.testing.assert_array_equal(st["offsets"], ref.offsets)
    np.testing.assert_array_equal(st["rem_prefill"], ref.rem_prefill)
    np.testing.assert_array_equal(st["rem_decode"], ref.rem_decode)
    np.testing.assert_array_equal(st["context"], ref.context)
    np.testing.assert_array_equal(bits(st["clock_ms"]), bits(ref.clock_ms))
    np.testing.assert_array_equal(st["iterations"], ref.iterations)


def gpu_trace_constrained(wl, tau, n_q=None, *, queue_cap=None):
    """As gpu_trace, under the constrained objective (Eq. 3) with targets tau [N]."""
    import torch
    from paper_2607_18253_amd import context_for

    N = wl.n_q if n_q is None else int(n_q)
    ctx = context_for(wl, queue_cap=queue_cap)
    ctx.advance(float(wl.q_t_ms[0]))
    chosen = torch.full((wl.n_scen, N), -1.0, dtype=torch.float64, device=DEV)
    util = torch.full((wl.n_scen, N), -1.0, dtype=torch.float64, device=DEV)
    choice = ctx.route_trace_constrained(
        T(wl.q_prefill[:N], torch.int32), T(wl.q_decode[:N], torch.int32),
        T(wl.q_t_ms[:N], torch.float64), float(wl.q_t_ms[N - 1]), T(tau[:N], torch.float64),
        T(wl.acc[:N], torch.float64), T(wl.cost[:N], torch.float64),
        T(wl.w_cost, torch.float64), chosen_ttft=chosen, utility=util)
    ctx.sync()
    return choice.cpu().numpy(), chosen.cpu().numpy(), util.cpu().numpy(), ctx


def gpu_trace_realized(wl, n_q=None, *, flags=0, tau=None, queue_cap=None, max_seqs_cap=None):
    """Sequential trace (Lagrangian, or Eq. 3 with targets tau) that also reports the
    realised TTFT of every query.  Returns (choice, chosen_ttft, realized, ctx)."""
    import torch
    from paper_2607_18253_amd import context_for

    N = wl.n_q if n_q is None else int(n_q)
    ctx = context_for(wl, flags=flags, queue_cap=queue_cap, max_seqs_cap=max_seqs_cap)
    ctx.advance(float(wl.q_t_ms[0]))
    chosen = torch.full((wl.n_scen, N), -1.0, dtype=torch.float64, device=DEV)
    real = torch.full((wl.n_scen, N), -1.0, dtype=torch.float64, device=DEV)
    args = (T(wl.q_prefill[:N], torch.int32), T(wl.q_decode[:N], torch.int32),
            T(wl.q_t_ms[:N], torch.float64), float(wl.q_t_ms[N - 1]))
    if tau is None:
        choice = ctx.route_trace(*args, T(wl.acc[:N], torch.float64),
                                 T(wl.cost[:N], torch.float64), T(wl.w_cost, torch.float64),
                                 T(wl.w_lat_ms, torch.float64), chosen_ttft=chosen,
                                 realized=real)
    else:
        choice = ctx.route_trace_constrained(*args, T(tau[:N], torch.float64),
                                             T(wl.acc[:N], torch.float64),
                                             T(wl.cost[:N], torch.float64),
                                             T(wl.w_cost, torch.float64), chosen_ttft=chosen,
                                             realized=real)
    ctx.sync()
    return choice.cpu().numpy(), chosen.cpu().numpy(), real.cpu().numpy(), ctx
