"""lar_whatif_noalloc (the what-if estimate and route that allocates nothing, its
working memory in a device array of the library) against the existing entry
points lar_estimate_ttft + lar_route on a context, bit for bit, on two calls in a
row -- the full c3 pool (1024 instances x 512 residents, 4096 queries), then a
smaller pool -- plus its host-side size check and its device-side snapshot check."""

from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from gpu_util import DEV, T, bits  # noqa: E402
from paper_2607_18253_amd import context_for  # noqa: E402
from paper_2607_18253_amd import lar as L  # noqa: E402
from workloads import make_workload  # noqa: E402


def _params(wl):
    rec = L.params_array(wl.a, wl.b, wl.c, wl.d, wl.e, wl.budget, wl.max_seqs, wl.col)
    return torch.as_tensor(rec.view(np.uint8).copy(), device=DEV)


def _noalloc(wl, t_ms, *, context=None, max_resident=None):
    I, Q = wl.n_inst, wl.n_q
    out = dict(ttft=torch.full((Q, I), -1.0, dtype=torch.float64, device=DEV),
               iters=torch.full((Q, I), -7, dtype=torch.int32, device=DEV),
               choice=torch.full((Q,), -7, dtype=torch.int32, device=DEV),
               chosen=torch.full((Q,), -1.0, dtype=torch.float64, device=DEV),
               util=torch.full((Q,), -1.0, dtype=torch.float64, device=DEV),
               status=torch.full((1,), 99, dtype=torch.int32, device=DEV))
    n_res = int(np.max(np.diff(wl.offsets)))
    L.whatif_noalloc(_params(wl), T(wl.offsets, torch.int32), T(wl.rem_prefill, torch.int32),
                     T(wl.rem_decode, torch.int32),
                     T(wl.context if context is None else context, torch.int32),
                     T(wl.clock_ms, torch.float64), T(wl.q_prefill, torch.int32), t_ms,
                     T(wl.acc, torch.float64), T(wl.cost, torch.float64),
                     T(wl.w_cost[:1], torch.float64), T(wl.w_lat_ms[:1], torch.float64),
                     out["ttft"], out["choice"], out["status"],
                     max_seqs_cap=int(np.max(wl.max_seqs)),
                     max_resident=n_res if max_resident is None else max_resident,
                     max_prompt=wl.max_prompt, iters=out["iters"], chosen_ttft=out["chosen"],
                     utility=out["util"])
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def _with_context(wl, t_ms):
    ctx = context_for(wl)
    tt, it = ctx.estimate(T(wl.q_prefill, torch.int32), t_ms)
    chosen = torch.empty((1, wl.n_q), dtype=torch.float64, device=DEV)
    util = torch.empty((1, wl.n_q), dtype=torch.float64, device=DEV)
    ch = ctx.route(tt, T(wl.acc, torch.float64), T(wl.cost, torch.float64),
                   T(wl.w_cost[:1], torch.float64), T(wl.w_lat_ms[:1], torch.float64),
                   chosen_ttft=chosen, utility=util)
    assert ctx.status() == 0
    out = dict(ttft=tt.cpu().numpy()[0], iters=it.cpu().numpy()[0], choice=ch.cpu().numpy()[0],
               chosen=chosen.cpu().numpy()[0], util=util.cpu().numpy()[0])
    ctx.close()
    return out


def _same(a, b):
    assert a["status"][0] == 0
    np.testing.assert_array_equal(bits(a["ttft"]), bits(b["ttft"]))
    np.testing.assert_array_equal(a["iters"], b["iters"])
    np.testing.assert_array_equal(a["choice"], b["choice"])
    np.testing.assert_array_equal(bits(a["chosen"]), bits(b["chosen"]))
    np.testing.assert_array_equal(bits(a["util"]), bits(b["util"]))


def test_noalloc_matches_context_path_twice():
    big = make_workload("c3")
    _same(_noalloc(big, 0.0), _with_context(big, 0.0))
    # a smaller pool and batch second: the array keeps the first call's contents
    small = make_workload("c3", n_inst=100, n_q=300, resident=200, seed=5)
    _same(_noalloc(small, 0.0), _with_context(small, 0.0))


def test_noalloc_size_and_snapshot_checks():
    wl = make_workload("c3", n_inst=20, n_q=16, resident=64, seed=3)
    # working memory beyond the scratch array: refused on the host, nothing enqueued
    with pytest.raises(L.LarError) as ei:
        _noalloc(wl, 0.0, max_resident=1 << 20)
    assert ei.value.code == L.LAR_E_CAPACITY
    # a snapshot breaking the FCFS rules (a running request behind waiting ones):
    # the device reports LAR_E_STATE in the status word
    cx = np.array(wl.context, np.int32)
    lo, hi = int(wl.offsets[4]), int(wl.offsets[5])
    cx[hi - 1] = 7
    assert cx[lo:hi - 1].min() == 0
    out = _noalloc(wl, 0.0, context=cx)
    assert out["status"][0] == L.LAR_E_STATE
    # and the next valid call is clean again
    _same(_noalloc(wl, 0.0), _with_context(wl, 0.0))
