"""GPU parity of the what-if trajectory walk (k_traj: decoding requests as per-batch
finish counts) against the oracle's literal per-pair SFS estimate (Sec. 4.1), bit
for bit, on the states where the walk's bookkeeping changes form:

* decode lengths on both sides of the ring's reach (2048 bins, so last tokens more
  than 1984 batches ahead go to the far list), with and without context terms;
* more far requests than the far list holds (the queue then runs the engine);
* a decode tail longer than the ring (token budget = sequence cap, long prompts);
* several partially prefilled requests (the engine again);
* trajectories that reach the iteration cap.
"""

from __future__ import annotations

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from gpu_util import T, bits  # noqa: E402
from oracle import oracle as O  # noqa: E402
from paper_2607_18253_amd import LarContext  # noqa: E402
from paper_2607_18253_amd import lar as L  # noqa: E402


def _pool(rng, I, M_choices, n_res, rd_draw, budget_extra=(0, 3000), partial_p=0.15,
          d_scale=1e-3):
    M = rng.choice(M_choices, size=I).astype(np.int32)
    B = (M + rng.integers(budget_extra[0], budget_extra[1] + 1, size=I)).astype(np.int32)
    reqs, offs = [], [0]
    for j in range(I):
        n = int(n_res(j))
        n_run = int(min(n, M[j], rng.integers(0, n + 1)))
        run = np.arange(n) < n_run
        rp = np.where(run, np.where(rng.random(n) < 1 - partial_p, 0, rng.integers(1, 300, n)),
                      rng.integers(1, 2500, n))
        cx = np.where(run, rng.integers(1, 4000, n), 0)
        rd = rd_draw(n)
        reqs.append((rp.astype(np.int32), rd.astype(np.int32), cx.astype(np.int32)))
        offs.append(offs[-1] + n)
    coef = rng.random((5, I))
    coef[3] *= d_scale
    coef[4] *= 1e-6
    return M, B, reqs, offs, coef


def _check(M, B, reqs, offs, coef, ps, *, flags=0, max_prompt=20000, max_iters=10_000_000,
           queue_cap=2048):
    I = len(M)
    ctx = LarContext(1, I, max_seqs_cap=int(M.max()), queue_cap=queue_cap,
                     max_prompt=max_prompt, flags=flags, max_iters=max_iters)
    ctx.load_state(a=coef[0], b=coef[1], c=coef[2], d=coef[3], e=coef[4], budget=B, max_seqs=M,
                   col=np.zeros(I, np.int32), offsets=offs,
                   rem_prefill=np.concatenate([r[0] for r in reqs]),
                   rem_decode=np.concatenate([r[1] for r in reqs]),
                   context=np.concatenate([r[2] for r in reqs]), clock_ms=np.zeros(I))
    ps = np.asarray(ps, np.int32)
    tt, it = ctx.estimate(T(ps, torch.int32), 0.0)
    st = ctx.status()
    tt, it = tt.cpu().numpy()[0], it.cpu().numpy()[0]
    capped = 0
    for j in range(I):
        q = O.Queue(O.make_params(*coef[:, j], B[j], M[j]), *reqs[j], 0.0)
        for a, p in enumerate(ps):
            try:
                want, wit = q.estimate(int(p), 1, 0.0, reading=flags, max_iters=max_iters)
            except O.OracleError:
                # past the cap: the trajectory is refused (NaN) or the estimate reports
                # more batches than the cap
                assert np.isnan(tt[a, j]) or it[a, j] > max_iters, (j, p)
                capped += 1
                continue
            assert it[a, j] == wit and bits(tt[a, j]) == bits(want), (j, int(p), tt[a, j], want)
    ctx.close()
    return st, capped


@pytest.mark.parametrize("flags", [0, 1])
@pytest.mark.parametrize("d_scale", [0.0, 1e-3])
def test_walk_far_requests(flags, d_scale):
    """Decode lengths around and far beyond the ring's reach; up to a few dozen far
    requests per queue (within the far list)."""
    rng = np.random.default_rng(21 + flags)

    def rd(n):
        kind = rng.random(n)
        return np.where(kind < 0.6, rng.integers(1, 200, n),
                        np.where(kind < 0.9, rng.integers(1900, 2100, n),
                                 rng.integers(3000, 20000, n)))

    M, B, reqs, offs, coef = _pool(rng, 24, [8, 64, 100, 200], lambda j: rng.integers(0, 120), rd,
                                   d_scale=d_scale)
    st, _ = _check(M, B, reqs, offs, coef, [1, 7, 64, 65, 500, 3000, 19999], flags=flags)
    assert st == 0


def test_walk_far_list_overflow_runs_the_engine():
    """Hundreds of requests beyond the ring's reach in one queue: more than the far
    list holds, so that queue runs the batch engine; the others walk."""
    rng = np.random.default_rng(5)

    def rd(n):
        return np.where(rng.random(n) < 0.8, rng.integers(2100, 9000, n), rng.integers(1, 50, n))

    M, B, reqs, offs, coef = _pool(rng, 6, [300, 512], lambda j: 700 if j < 3 else 40, rd,
                                   budget_extra=(0, 800))
    st, _ = _check(M, B, reqs, offs, coef, [1, 100, 4000])
    assert st == 0


@pytest.mark.parametrize("flags", [0, 1])
def test_walk_tail_longer_than_the_ring(flags):
    """Token budget equal to the sequence cap leaves one prefill token per batch for a
    tail query: its prompt of up to 6000 tokens needs a decode tail of 6000 batches,
    three times around the ring of per-batch counts."""
    rng = np.random.default_rng(8)
    I = 10
    M = np.full(I, 16, np.int32)
    B = M.copy()
    reqs, offs = [], [0]
    for j in range(I):
        n = 40
        rp = np.where(np.arange(n) < 12, 0, rng.integers(1, 30, n))
        cx = np.where(np.arange(n) < 12, rng.integers(1, 100, n), 0)
        rd = rng.integers(1, 5000, n)
        reqs.append((rp.astype(np.int32), rd.astype(np.int32), cx.astype(np.int32)))
        offs.append(offs[-1] + n)
    coef = rng.random((5, I))
    coef[3] *= 1e-3
    coef[4] = 0.0
    st, _ = _check(M, B, reqs, offs, coef, [1, 2, 2047, 2048, 4500, 6000], flags=flags,
                   max_prompt=6000)
    assert st == 0


def test_walk_several_partials_runs_the_engine():
    """Snapshots with two or more partially prefilled requests at the list head."""
    rng = np.random.default_rng(3)

    def rd(n):
        return rng.integers(1, 600, n)

    M, B, reqs, offs, coef = _pool(rng, 16, [4, 16, 64], lambda j: rng.integers(5, 80), rd,
                                   partial_p=0.7)
    assert any(np.sum((r[0] > 0) & (r[2] > 0)) > 1 for r in reqs)
    st, _ = _check(M, B, reqs, offs, coef, [1, 50, 900])
    assert st == 0


def test_walk_iteration_cap():
    """A cap below some queues' trajectories: those entries are refused as the oracle
    refuses them (sticky LAR_E_ITER); the rest are exact."""
    rng = np.random.default_rng(9)

    def rd(n):
        return rng.integers(1, 3000, n)

    M, B, reqs, offs, coef = _pool(rng, 12, [4, 16], lambda j: rng.integers(0, 60), rd,
                                   budget_extra=(0, 200))
    st, capped = _check(M, B, reqs, offs, coef, [1, 300, 5000], max_iters=2500)
    assert capped > 0
    assert st == L.LAR_E_ITER
