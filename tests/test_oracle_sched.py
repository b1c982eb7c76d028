"""Pins of the oracle's scheduler limits (chunk cap, context limit, KV-cache blocks
with recompute preemption), taken from the system appendix's list of what the SFS
simulation follows and Sec. 2 on paged KV caches and chunked prefill.

* hand-worked cases (tests/golden/sched_hand_worked.json);
* reduction: limits that are off, or that never bind, give the pinned default batch
  bit for bit;
* an independent token-at-a-time scheduler with numbered KV blocks and separate
  running / waiting lists (tests/bruteforce_sched.py) on random tiny traces, both
  readings and both objectives, with realised TTFT;
* invariants after every batch; error paths.
"""

import itertools
import json
import os

import numpy as np
import pytest

from oracle import oracle as O
from workloads import make_tiny_workload
from workloads.gen import make_tiny_sched_workload, make_workload
import bruteforce_sched as BF

GOLD = os.path.join(os.path.dirname(__file__), "golden", "sched_hand_worked.json")


def _lim(d):
    return [d["chunk_cap"], d["kv_blocks"], d["block_size"], d["max_ctx"]]


def _queue(coef, B, M, reqs, lim):
    return O.Queue(O.make_params(coef["a"], coef["b"], coef["c"], coef["d"], coef["e"], B, M),
                   [r[0] for r in reqs], [r[1] for r in reqs], [r[2] for r in reqs], 0.0,
                   sched=lim)


def bits(x):
    return np.ascontiguousarray(x, dtype=np.float64).view(np.int64)


# ------------------------------------------------------------------ hand-worked
def test_sched_hand_worked():
    g = json.load(open(GOLD))
    for case in g["cases"]:
        lim = _lim(case["limits"])
        q = _queue(g["coef"], case["budget"], case["max_seqs"], case["requests"], lim)
        tb, ib = q.estimate(case["p"], case["dhat"], case["t"], O.READING_DECODE_BATCH)
        ta, ia = q.estimate(case["p"], case["dhat"], case["t"], O.READING_PREFILL_BATCH)
        assert (tb, ib) == (case["ttft_B"], case["iters_B"]), case["name"]
        assert (ta, ia) == (case["ttft_A"], case["iters_A"]), case["name"]
        # the same through a replay: append the query, step to its first decode
        q.append(case["p"], case["dhat"])
        clk = 0.0
        for _ in range(case["iters_B"]):
            T, _f = q.step()
            clk = clk + T
        assert clk == case["ttft_B"], case["name"]
        assert q.preemptions() == case["preemptions_B"], case["name"]
        # and the brute force agrees
        c = g["coef"]
        bf = BF.BFSchedInstance(c["a"], c["b"], c["c"], c["d"], c["e"], case["budget"],
                                case["max_seqs"], lim, *zip(*case["requests"])
                                if case["requests"] else ((), (), ()))
        assert bf.estimate(case["p"], case["dhat"], case["t"], 0) == (tb, ib), case["name"]
        assert bf.estimate(case["p"], case["dhat"], case["t"], 1) == (ta, ia), case["name"]


def test_sched_hand_worked_batches():
    g = json.load(open(GOLD))
    c = g["coef"]
    for case in g["batch_cases"]:
        lim = _lim(case["limits"])
        q = _queue(c, case["budget"], case["max_seqs"], case["requests"], lim)
        _, f = q.step()
        rp, rd, cx, _, _ = q.state()
        assert list(f) == case["features"], case["name"]
        assert [list(x) for x in zip(rp, rd, cx)] == case["after"], case["name"]
        assert q.preemptions() == case["preemptions"], case["name"]
        bf = BF.BFSchedInstance(c["a"], c["b"], c["c"], c["d"], c["e"], case["budget"],
                                case["max_seqs"], lim, *zip(*case["requests"]))
        _, fb, _ = bf.batch()
        assert list(fb) == case["features"], case["name"]
        assert [list(x) for x in bf.state()] == case["after"], case["name"]


def test_context_limit_cuts_resident_decode():
    g = json.load(open(GOLD))
    case = g["cases"][1]
    q = _queue(g["coef"], case["budget"], case["max_seqs"], case["requests"],
               _lim(case["limits"]))
    rp, rd, cx, _, _ = q.state()
    assert list(rd) == [3]           # 100 predicted decodes cut to 13 - 10


# ------------------------------------------------------------------ reduction
def _trace_pair(wl, **kw):
    r0 = O.trace(wl, full_rows=True, **kw)
    return r0


def _same(r1, r2):
    np.testing.assert_array_equal(r1.choice, r2.choice)
    np.testing.assert_array_equal(bits(r1.ttft_all), bits(r2.ttft_all))
    np.testing.assert_array_equal(r1.iters_all, r2.iters_all)
    np.testing.assert_array_equal(bits(r1.realized), bits(r2.realized))
    for f in ("offsets", "rem_prefill", "rem_decode", "context", "iterations"):
        np.testing.assert_array_equal(getattr(r1, f), getattr(r2, f))
    np.testing.assert_array_equal(bits(r1.clock_ms), bits(r2.clock_ms))


@pytest.mark.parametrize("seed", range(12))
def test_limits_off_or_slack_reduce_to_default(seed):
    """No limit set, or limits that cannot bind (chunk cap >= budget, a KV cache and a
    context limit larger than anything the trace reaches), give the default batch."""
    wl = make_tiny_workload(seed, n_q=30)
    reading = seed % 2
    base = O.trace(wl, full_rows=True, reading=reading)
    wl.sched = np.zeros((wl.n_inst, 4), np.int32)
    _same(base, O.trace(wl, full_rows=True, reading=reading))
    big = 1 << 20
    wl.sched = np.array([[int(wl.budget[j]), big, 4, big] for j in range(wl.n_inst)], np.int32)
    _same(base, O.trace(wl, full_rows=True, reading=reading))


# ------------------------------------------------------------------ brute force
@pytest.mark.parametrize("seed", range(40))
def test_sched_bruteforce_traces(seed):
    wl = make_tiny_sched_workload(seed, n_q=25, max_res=5)
    reading = seed % 2
    tau = None
    if seed % 4 >= 2:      # Eq. 3 with targets inside the estimates' range
        rng = np.random.default_rng(seed)
        tau = rng.uniform(0.0, 40.0, size=wl.n_q)
    real_bf = np.zeros(wl.n_q)
    ch, rows, insts = BF.trace(wl, reading=reading, tau=tau, realized=real_bf)
    r = O.trace(wl, full_rows=True, reading=reading, tau=tau)
    np.testing.assert_array_equal(r.choice, ch)
    np.testing.assert_array_equal(bits(r.ttft_all), bits(rows))
    np.testing.assert_array_equal(bits(r.realized), bits(real_bf))
    for j, x in enumerate(insts):
        lo, hi = r.offsets[j], r.offsets[j + 1]
        got = list(zip(r.rem_prefill[lo:hi], r.rem_decode[lo:hi], r.context[lo:hi]))
        assert got == x.state(), (seed, j)
        assert r.clock_ms[j] == x.clock


def test_sched_bruteforce_exercises_every_limit():
    """The random tiny traces above preempt, cut chunks and end decodes at the
    context limit (counted on the brute force's side)."""
    pre = cut = 0
    for seed in range(40):
        wl = make_tiny_sched_workload(seed, n_q=25, max_res=5)
        _, _, insts = BF.trace(wl, reading=seed % 2)
        pre += sum(x.preemptions for x in insts)
        for j in range(wl.n_inst):
            H, K, S, X = wl.sched[j]
            rp, rd, cx = wl.instance_requests(j)
            cut += int(np.sum(rd > X - (cx + rp)))
    assert pre >= 50 and cut >= 5, (pre, cut)


# ------------------------------------------------------------------ invariants
@pytest.mark.parametrize("seed", range(10))
def test_sched_invariants(seed):
    wl = make_tiny_sched_workload(seed, n_q=1, max_res=6)
    for j in range(wl.n_inst):
        H, K, S, X = (int(v) for v in wl.sched[j])
        q = O.instance_queue(wl, j)
        for p in range(1, 9):
            q.append(p, 3)
        for _ in range(60):
            if q.size() == 0:
                break
            rp0, _, cx0, _, _ = q.state()
            T, (P, D, C, A) = q.step()
            rp, rd, cx, _, _ = q.state()
            running = cx > 0
            assert running.sum() <= wl.max_seqs[j]
            assert P + D <= wl.budget[j]
            if K > 0:
                assert sum(-(-int(c) // S) for c in cx[running]) <= K
            if X > 0:
                assert np.all(cx + rp <= X) and np.all(rd <= X - (cx + rp))
            if H > 0:
                # no request's prefill shrinks by more than the cap in one batch
                n = min(len(rp0), len(rp))
                assert np.all(np.maximum(rp0[:n] - rp[:n], 0) <= H) or len(rp0) != len(rp)


# ------------------------------------------------------------------ errors
def test_sched_errors():
    pr = O.make_params(1, 1, 1, 0, 0, 8, 4)
    with pytest.raises(O.OracleError) as e:
        O.Queue(pr, [0], [3], [5], sched=[0, 4, 2, 0])      # KV cache without a context limit
    assert e.value.code == O.E_ARG
    with pytest.raises(O.OracleError) as e:
        O.Queue(pr, [0], [3], [5], sched=[0, 2, 2, 6])      # 2 blocks of 2 < limit 6
    assert e.value.code == O.E_ARG
    with pytest.raises(O.OracleError) as e:
        O.Queue(pr, [0], [3], [6], sched=[0, 0, 1, 6])      # context at the limit
    assert e.value.code == O.E_STATE
    with pytest.raises(O.OracleError) as e:
        O.Queue(pr, [0, 0], [3, 3], [5, 5], sched=[0, 5, 2, 8])   # 6 blocks held > 5
    assert e.value.code == O.E_STATE
    q = O.Queue(pr, [], [], [], sched=[0, 0, 1, 6])
    with pytest.raises(O.OracleError) as e:
        q.append(6, 1)                                      # no room for a decode
    assert e.value.code == O.E_ARG
    # an instance whose context limit cannot hold the prompt cannot take the query
    assert q.estimate(6, 1, 0.0) == (np.inf, 0)
    with pytest.raises(O.OracleError):
        q.estimate(0, 1, 0.0)                               # a prompt has a token


def _mixed_limit_pool(n_q=40, seed=5):
    """A pool mixing a small context limit (instance 0, the cheapest and most
    accurate) with larger ones; prompts that only the larger instances can hold."""
    wl = make_tiny_sched_workload(seed, n_inst=4, n_q=n_q, max_res=3)
    wl.sched[:, 1] = 0                     # no KV cache (the limit then needs no blocks)
    wl.sched[:, 3] = 64
    wl.sched[0, 3] = 24
    for j in range(4):                    # every resident fits its instance's limit
        rp, rd, cx = wl.instance_requests(j)
        assert len(rp) == 0 or (rp + cx).max() < wl.sched[j, 3]
    wl.acc[:, :] = 0.1
    wl.acc[:, wl.col[0]] = 0.9            # instance 0 wins whenever it can take a query
    rng = np.random.default_rng(seed)
    wl.q_prefill[:] = rng.integers(1, 40, n_q)   # many do not fit instance 0's limit
    wl.max_prompt = 64
    return wl


def test_mixed_context_limits_route():
    """Routing over instances with different context limits: a prompt at or above an
    instance's limit gives it TTFT +inf there and it is never chosen; the choice is
    the argmax over the instances that can take the query (a restatement of Eq. 5
    over the feasible instances, numpy's argmax)."""
    wl = _mixed_limit_pool()
    r = O.trace(wl, full_rows=True)
    assert np.isinf(r.ttft_all[:, 0]).sum() > 5 and np.isfinite(r.ttft_all[:, 1:]).all()
    for i in range(wl.n_q):
        row = r.ttft_all[i]
        u = (wl.acc[i, wl.col] - wl.w_cost[0] * wl.cost[i, wl.col]) - wl.w_lat_ms[0] * row
        u[np.isinf(row)] = -np.inf
        assert r.choice[i] == int(np.argmax(u)), i
        assert np.isfinite(row[r.choice[i]])
    assert (r.choice == 0).sum() > 0 and (r.choice != 0).sum() > 0


def test_query_no_instance_can_take():
    wl = _mixed_limit_pool(n_q=10)
    wl.q_prefill[4] = 64                  # at every instance's context limit
    r = O.trace(wl, n_q=4)
    assert len(r.choice) == 4
    with pytest.raises(O.OracleError) as e:
        O.trace(wl)
    assert e.value.code == O.E_ARG and "query 4" in str(e.value)


def test_c7_limits_bind():
    """The c7 pool: its residents fit the limits, and routing its first queries makes
    the KV cache preempt (counted by the oracle)."""
    wl = make_workload("c7", n_q=300)
    qs = [O.instance_queue(wl, j) for j in range(wl.n_inst)]
    for q in qs:
        q.advance(float(wl.q_t_ms[0]))
    for i in range(wl.n_q):
        p, d, t = int(wl.q_prefill[i]), int(wl.q_decode[i]), float(wl.q_t_ms[i])
        row = np.array([q.estimate(p, d, t)[0] for q in qs])
        u = (wl.acc[i][wl.col] - wl.w_cost[0] * wl.cost[i][wl.col]) - wl.w_lat_ms[0] * row
        qs[int(np.argmax(u))].append(p, d)
        t_next = float(wl.q_t_ms[i + 1]) if i + 1 < wl.n_q else t
        for q in qs:
            q.advance(t_next)
    assert sum(q.preemptions() for q in qs) > 0


# ------------------------------------------------------------------ exhaustive tiny states
def _tiny_states(max_n=3):
    dec = [[0, rd, cx] for rd in (1, 2) for cx in (1, 3)]
    par = [[rp, rd, cx] for rp in (1, 3) for rd in (1, 2) for cx in (1, 3)]
    wai = [[rp, rd, 0] for rp in (1, 3) for rd in (1, 2)]
    run = dec + par
    for n in range(0, max_n + 1):
        for n_run in range(0, n + 1):
            for rs in itertools.product(run, repeat=n_run):
                for ws in itertools.product(wai, repeat=n - n_run):
                    yield [list(x) for x in rs] + [list(x) for x in ws], n_run


# (chunk cap, KV blocks, block size, context limit): none, context limit only, and KV
# caches barely above one request's need at block sizes 1, 2 and 4
_LIMITS = [(0, 0, 1, 0), (0, 0, 1, 9), (1, 7, 1, 7), (2, 4, 2, 8), (0, 3, 4, 10), (2, 0, 1, 0)]


def _sched_cases(stride=1):
    for idx, (reqs, n_run) in enumerate(_tiny_states()):
        if idx % stride:
            continue
        for B, M in [(1, 1), (3, 2), (4, 3)]:
            if n_run > M:
                continue
            for lim in _LIMITS:
                H, K, S, X = lim
                if X and any(r[0] + r[2] >= X for r in reqs):
                    continue
                if K and sum(-(-r[2] // S) for r in reqs if r[2] > 0) > K:
                    continue
                yield reqs, B, M, list(lim)


def _pair(coef, B, M, reqs, lim):
    c = coef
    q = _queue(c, B, M, reqs, lim)
    bf = BF.BFSchedInstance(c["a"], c["b"], c["c"], c["d"], c["e"], B, M, lim,
                            *(zip(*reqs) if reqs else ((), (), ())))
    return q, bf


def test_sched_bruteforce_exhaustive_tiny_states():
    """Every tiny state (<= 3 residents of every kind; one in three of the 3-resident
    ones) under six limit settings against the token-at-a-time scheduler with numbered
    KV blocks: iteration counts and TTFT bits, both readings."""
    coef = dict(a=0.75, b=0.3, c=0.2, d=0.01, e=0.003)
    n_checked = 0
    preempting = 0
    for reqs, B, M, lim in _sched_cases(stride=3):
        q, bf = _pair(coef, B, M, reqs, lim)
        for p in (1, 4):
            if lim[3] and p >= lim[3]:
                continue
            for reading in (0, 1):
                tt, it = q.estimate(p, 1, 0.0, reading)
                w = bf.copy()
                tb, ib = w.estimate(p, 1, 0.0, reading)
                assert (it, tt) == (ib, tb), (reqs, B, M, lim, p, reading)
                n_checked += 1
        probe = bf.copy()
        probe.append(4 if not lim[3] or lim[3] > 4 else 1, 1)
        for _ in range(12):
            if not probe.reqs:
                break
            probe.step()
        preempting += probe.preemptions > 0
    assert n_checked > 20000 and preempting > 500, (n_checked, preempting)


def test_sched_bruteforce_steps_tiny_states():
    """Three replayed batches per tiny state under every limit setting: features, batch
    time and resulting state, against the token-at-a-time scheduler."""
    coef = dict(a=0.75, b=0.3, c=0.2, d=0.01, e=0.003)
    for reqs, B, M, lim in _sched_cases(stride=2):
        q, bf = _pair(coef, B, M, reqs, lim)
        for _ in range(3):
            if not bf.reqs:
                break
            T, f = q.step()
            Tb, fb = bf.step()
            assert (T, f) == (Tb, fb), (reqs, B, M, lim)
            rp, rd, cx, _, _ = q.state()
            assert [list(x) for x in zip(rp, rd, cx)] == [list(x) for x in bf.state()], \
                (reqs, B, M, lim)
