"""Pins of the C oracle against things other than itself.

* hand-worked cases (tests/golden/hand_worked.json);
* closed forms: empty instance, pure-decode backlog, the throughput special case
  (Eq. for the throughput-based estimator with theta = 1/b and zero decode time),
  linearity in (a, b, c) when d = e = 0;
* an independent token-at-a-time scheduler (tests/bruteforce_sched.py), exhaustive
  over tiny states and on random tiny traces;
* numpy's argmax for the route, numpy sorting for the percentiles;
* invariants: token budget, sequence cap, FCFS token conservation, monotonicity.
"""

import dataclasses
import itertools
import json
import math
import os

import numpy as np
import pytest

from oracle import oracle as O
from workloads import make_tiny_workload
import bruteforce_sched as BF

GOLD = os.path.join(os.path.dirname(__file__), "golden", "hand_worked.json")


def _queue(coef, B, M, reqs, clock=0.0):
    rp = [r[0] for r in reqs]
    rd = [r[1] for r in reqs]
    cx = [r[2] for r in reqs]
    return O.Queue(O.make_params(coef["a"], coef["b"], coef["c"], coef["d"], coef["e"], B, M),
                   rp, rd, cx, clock)


def _bf(coef, B, M, reqs, clock=0.0):
    return BF.BFInstance(coef["a"], coef["b"], coef["c"], coef["d"], coef["e"], B, M,
                         [r[0] for r in reqs], [r[1] for r in reqs], [r[2] for r in reqs], clock)


# ------------------------------------------------------------------ hand-worked
def test_hand_worked_estimates():
    g = json.load(open(GOLD))
    for case in g["estimates"]:
        q = _queue(g["coef"], case["budget"], case["max_seqs"], case["requests"], case["clock"])
        if "advance_to" in case:
            q.advance(case["advance_to"])
            assert q.state()[3] == case["clock_after_advance"], case["name"]
        tb, ib = q.estimate(case["p"], case["dhat"], case["t"], O.READING_DECODE_BATCH)
        ta, ia = q.estimate(case["p"], case["dhat"], case["t"], O.READING_PREFILL_BATCH)
        assert (tb, ib) == (case["ttft_B"], case["iters_B"]), case["name"]
        assert (ta, ia) == (case["ttft_A"], case["iters_A"]), case["name"]


def test_hand_worked_routes():
    g = json.load(open(GOLD))
    for case in g["routes"]:
        n = len(case["ttft"])
        m, u = O.route_row(case["ttft"], case["acc"], case["cost"], list(range(n)),
                           case["w_cost"], case["w_lat"])
        assert (m, u) == (case["choice"], case["u"]), case["name"]


# ------------------------------------------------------------------ closed forms
DY = dict(a=1.0, b=0.5, c=0.25, d=0.125, e=0.0625)


@pytest.mark.parametrize("B", [1, 3, 4, 16])
def test_empty_instance_closed_form(B):
    """Empty instance: ceil(p/B) prefill batches of B tokens (last one the rest) at
    contexts 0, B, 2B, ..., then one decode batch at context p."""
    for p in range(1, 5 * B + 3):
        k = -(-p // B)
        prefill = 0.0
        for m in range(1, k + 1):
            ch = B if m < k else p - (k - 1) * B
            prefill += DY["a"] + DY["b"] * ch + DY["e"] * (ch * (m - 1) * B + ch * (ch + 1) / 2)
        decode = DY["a"] + DY["c"] + DY["d"] * p
        q = _queue(DY, B, 1, [])
        assert q.estimate(p, 7, 0.0, O.READING_PREFILL_BATCH) == (prefill, k)
        assert q.estimate(p, 7, 0.0, O.READING_DECODE_BATCH) == (prefill + decode, k + 1)


def test_pure_decode_backlog_closed_form():
    """n decoding sequences that outlive the query's prefill, nothing waiting: the
    query takes B - n tokens per batch, the decode term grows by n each batch."""
    rng = np.random.default_rng(1)
    for _ in range(200):
        B = int(rng.integers(2, 40))
        M = int(rng.integers(2, B + 1))
        n = int(rng.integers(0, M))
        ctx = rng.integers(1, 50, size=n).tolist()
        p = int(rng.integers(1, 4 * B))
        room = B - n
        K = -(-p // room)
        reqs = [[0, K + 2 + int(rng.integers(0, 3)), c] for c in ctx]
        exp, rem, cq = 0.0, p, 0
        for k in range(K):
            ch = min(rem, room)
            T = DY["a"] + DY["b"] * ch + DY["c"] * n + DY["d"] * (sum(ctx) + k * n) \
                + DY["e"] * (ch * cq + ch * (ch + 1) / 2)
            exp += T
            rem -= ch
            cq += ch
        exp_b = exp + DY["a"] + DY["c"] * (n + 1) + DY["d"] * (sum(ctx) + K * n + p)
        q = _queue(DY, B, M, reqs)
        assert q.estimate(p, 1, 0.0, O.READING_PREFILL_BATCH) == (exp, K)
        assert q.estimate(p, 1, 0.0, O.READING_DECODE_BATCH) == (exp_b, K + 1)


def _random_state(rng, B, M, n, pmax=20, dmax=6):
    n_run = int(rng.integers(0, min(n, M) + 1))
    reqs = []
    for r in range(n):
        if r < n_run:
            if rng.random() < 0.5:
                reqs.append([0, int(rng.integers(1, dmax + 1)), int(rng.integers(1, 30))])
            else:
                reqs.append([int(rng.integers(1, pmax)), int(rng.integers(1, dmax + 1)),
                             int(rng.integers(1, 30))])
        else:
            reqs.append([int(rng.integers(1, pmax)), int(rng.integers(1, dmax + 1)), 0])
    return reqs


def test_throughput_special_case():
    """a = c = d = e = 0: every batch costs b*P, and all resident prefill is served
    before the query's last chunk, so TTFT = b*(sum of remaining prefill + p): the
    throughput estimator with prefill throughput 1/b and no decode time."""
    rng = np.random.default_rng(2)
    coef = dict(a=0.0, b=0.375, c=0.0, d=0.0, e=0.0)
    for _ in range(300):
        B = int(rng.integers(1, 30))
        M = int(rng.integers(1, B + 1))
        reqs = _random_state(rng, B, M, int(rng.integers(0, 12)))
        p = int(rng.integers(1, 60))
        q = _queue(coef, B, M, reqs)
        want = 0.375 * (sum(r[0] for r in reqs) + p)
        for reading in (0, 1):
            assert q.estimate(p, 3, 0.0, reading)[0] == want


def test_linearity_when_no_context_terms():
    """d = e = 0: TTFT = a*iters + b*(sum rp + p) + c*(decode tokens), with iters and
    the decode-token count taken from the independent token-at-a-time scheduler."""
    rng = np.random.default_rng(3)
    coef = dict(a=1.0, b=0.5, c=0.25, d=0.0, e=0.0)
    for _ in range(300):
        B = int(rng.integers(1, 20))
        M = int(rng.integers(1, B + 1))
        reqs = _random_state(rng, B, M, int(rng.integers(0, 10)))
        p = int(rng.integers(1, 40))
        tt, it = _queue(coef, B, M, reqs).estimate(p, 2, 0.0)
        _, it_bf, feats = _bf(coef, B, M, reqs).estimate(p, 2, 0.0)
        sumD = sum(f[1] for f in feats)
        assert it == it_bf
        assert tt == 1.0 * it + 0.5 * (sum(r[0] for r in reqs) + p) + 0.25 * sumD


def test_reading_a_b_relation():
    """Reading B runs exactly one more batch than reading A, a decode batch."""
    rng = np.random.default_rng(4)
    for _ in range(300):
        B = int(rng.integers(1, 20))
        M = int(rng.integers(1, B + 1))
        reqs = _random_state(rng, B, M, int(rng.integers(0, 10)))
        p = int(rng.integers(1, 40))
        q = _queue(DY, B, M, reqs)
        ta, ia = q.estimate(p, 2, 0.0, 1)
        tb, ib = q.estimate(p, 2, 0.0, 0)
        assert ib == ia + 1
        _, _, feats = _bf(DY, B, M, reqs).estimate(p, 2, 0.0, 0)
        P, D, Cf, A = feats[-1]
        assert P == 0 and A == 0 and D >= 1
        T = DY["a"] + DY["b"] * P + DY["c"] * D + DY["d"] * Cf + DY["e"] * A
        assert tb == ta + T


def test_monotone_in_prompt():
    rng = np.random.default_rng(5)
    for _ in range(100):
        B = int(rng.integers(1, 20))
        M = int(rng.integers(1, B + 1))
        coef = dict(zip("abcde", rng.random(5)))
        reqs = _random_state(rng, B, M, int(rng.integers(0, 10)))
        q = _queue(coef, B, M, reqs)
        vals = [q.estimate(p, 1, 0.0)[0] for p in range(1, 50)]
        assert all(x <= y for x, y in zip(vals, vals[1:]))


# ------------------------------------------------------------------ brute force
def _tiny_states():
    dec = [[0, rd, cx] for rd in (1, 2) for cx in (1, 3)]
    par = [[rp, rd, cx] for rp in (1, 3) for rd in (1, 2) for cx in (1, 3)]
    wai = [[rp, rd, 0] for rp in (1, 3) for rd in (1, 2)]
    run = dec + par
    for n in range(0, 4):
        for n_run in range(0, n + 1):
            for rs in itertools.product(run, repeat=n_run):
                for ws in itertools.product(wai, repeat=n - n_run):
                    yield [list(x) for x in rs] + [list(x) for x in ws], n_run


def test_bruteforce_exhaustive_tiny_states():
    """Every tiny state (<= 3 residents of every kind) against the token-at-a-time
    scheduler: iteration counts and TTFT bits, both readings."""
    coef = dict(a=0.75, b=0.3, c=0.2, d=0.01, e=0.003)
    BM = [(1, 1), (2, 1), (2, 2), (3, 2), (4, 3), (4, 1)]
    n_checked = 0
    for reqs, n_run in _tiny_states():
        for B, M in BM:
            if n_run > M:
                continue
            q = _queue(coef, B, M, reqs)
            bf = _bf(coef, B, M, reqs)
            for p in (1, 2, 5):
                for reading in (0, 1):
                    tt, it = q.estimate(p, 1, 0.0, reading)
                    tb, ib, _ = bf.estimate(p, 1, 0.0, reading)
                    assert (it, tt) == (ib, tb), (reqs, B, M, p, reading)
                    n_checked += 1
    assert n_checked > 10000


def test_bruteforce_steps_tiny_states():
    """One replayed batch per tiny state: features, batch time and resulting state."""
    coef = dict(a=0.75, b=0.3, c=0.2, d=0.01, e=0.003)
    for reqs, n_run in _tiny_states():
        for B, M in [(1, 1), (2, 2), (4, 3)]:
            if n_run > M:
                continue
            q = _queue(coef, B, M, reqs)
            bf = _bf(coef, B, M, reqs)
            T, f = q.step()
            Tb, fb = bf.step()
            assert (T, f) == (Tb, fb)
            rp, rd, cx, clock, _ = q.state()
            assert [list(x) for x in zip(rp, rd, cx)] == [list(x) for x in bf.state()]
            assert f[0] + f[1] <= B
            assert int(np.sum(cx > 0)) <= M


@pytest.mark.parametrize("seed", range(60))
def test_bruteforce_random_traces(seed):
    """Whole sequential traces (estimate, route, commit, advance) on random tiny
    pools: choices, every TTFT bit and the final state."""
    wl = make_tiny_workload(seed, n_inst=3, max_res=5, n_q=25, dyadic=(seed % 2 == 0),
                            n_scen=1)
    for reading in (0, 1):
        r = O.trace(wl, reading=reading, full_rows=True, queue_cap=10 ** 6)
        real = np.zeros(wl.n_q)
        ch, rows, insts = BF.trace(wl, reading=reading, realized=real)
        np.testing.assert_array_equal(r.choice, ch)
        assert np.array_equal(r.ttft_all.view(np.int64), rows.view(np.int64))
        assert np.array_equal(r.realized.view(np.int64), real.view(np.int64))
        for j, x in enumerate(insts):
            lo, hi = r.offsets[j], r.offsets[j + 1]
            got = list(zip(r.rem_prefill[lo:hi], r.rem_decode[lo:hi], r.context[lo:hi]))
            assert [tuple(int(v) for v in g) for g in got] == x.state()
            assert r.clock_ms[j] == x.clock


# ------------------------------------------------------------------ route / stats
def test_route_matches_numpy_argmax():
    rng = np.random.default_rng(6)
    for _ in range(500):
        I = int(rng.integers(1, 40))
        n_cols = int(rng.integers(1, 5))
        col = rng.integers(0, n_cols, size=I).astype(np.int32)
        # coarse values make exact ties common
        ttft = rng.integers(0, 6, size=I) * 0.5
        acc = rng.integers(0, 4, size=n_cols) / 4.0
        cost = rng.integers(0, 4, size=n_cols) / 4.0
        wc, wlat = float(rng.integers(0, 3)) / 2, float(rng.integers(0, 3)) / 8
        m, u = O.route_row(ttft, acc, cost, col, wc, wlat)
        uu = (acc[col] - wc * cost[col]) - wlat * ttft
        assert m == int(np.argmax(uu))
        assert u == uu[m]


def test_stats_match_numpy():
    rng = np.random.default_rng(7)
    for n in (1, 2, 3, 99, 100, 101, 1000):
        n_cols = 3
        col = np.array([0, 1, 2, 2], np.int32)
        choice = rng.integers(0, 4, size=n).astype(np.int32)
        ttft = rng.random(n) * 100
        acc = rng.random((n, n_cols))
        cost = rng.random((n, n_cols))
        out = O.stats(choice, ttft, acc, cost, col, 0.3)
        a = acc[np.arange(n), col[choice]]
        c = cost[np.arange(n), col[choice]]
        sa = sc = su = 0.0
        for x, y in zip(a, c):
            sa += x
            sc += y
            su += x - 0.3 * y
        s = np.sort(ttft)
        assert out[0] == sa / n and out[1] == sc / n and out[2] == su / n
        assert out[3] == s[math.ceil(0.5 * n) - 1]
        assert out[4] == s[math.ceil(0.99 * n) - 1]


# ------------------------------------------------------------------ replay invariants
def test_advance_conserves_tokens_and_folds_clock():
    rng = np.random.default_rng(8)
    for _ in range(100):
        B = int(rng.integers(1, 20))
        M = int(rng.integers(1, B + 1))
        reqs = _random_state(rng, B, M, int(rng.integers(1, 12)))
        q = _queue(DY, B, M, reqs)
        tot_pre = sum(r[0] for r in reqs)
        tot_dec = sum(r[1] for r in reqs)
        clock, served_p, served_d = 0.0, 0, 0
        while q.size() > 0:
            T, f = q.step()
            clock = clock + T
            served_p += f[0]
            served_d += f[1]
            assert f[0] + f[1] <= B
            assert q.state()[3] == clock
        assert served_p == tot_pre and served_d == tot_dec
        q.advance(clock + 5.0)
        assert q.state()[3] == clock + 5.0           # idle instance jumps to t


def test_error_paths():
    p = O.make_params(1, 1, 1, 0, 0, 4, 2)
    with pytest.raises(O.OracleError) as e:
        O.Queue(p, [0, 1], [1, 1], [0, 3])           # rp == 0 with empty context
    assert e.value.code == O.E_STATE
    with pytest.raises(O.OracleError) as e:
        O.Queue(p, [2, 1], [1, 1], [0, 3])           # running after waiting
    assert e.value.code == O.E_STATE
    with pytest.raises(O.OracleError) as e:
        O.Queue(p, [0, 0, 0], [1, 1, 1], [1, 1, 1])  # more running than M
    assert e.value.code == O.E_STATE
    with pytest.raises(O.OracleError) as e:
        O.Queue(O.make_params(1, 1, 1, 0, 0, 2, 3), [], [], [])   # M > B
    assert e.value.code == O.E_ARG
    q = O.Queue(p, [0], [5], [3])
    with pytest.raises(O.OracleError) as e:
        q.estimate(0, 1, 0.0)
    assert e.value.code == O.E_ARG
    with pytest.raises(O.OracleError) as e:
        q.estimate(1, 1, 10.0)                       # instance not advanced to t
    assert e.value.code == O.E_STATE
    with pytest.raises(O.OracleError) as e:
        q.estimate(100, 1, 0.0, max_iters=3)
    assert e.value.code == O.E_ITER
    q.append(3, 1, queue_cap=1)
    with pytest.raises(O.OracleError) as e:
        q.append(3, 1, queue_cap=1)
    assert e.value.code == O.E_CAPACITY


# ------------------------------------------------------------------ constrained route (Eq. 3)
def test_ttft_target_hand_values():
    """TTFT targets (appendix on TTFT latency assignment), worked by hand:
    p = 1000, u = 3, v = 1: 155 + 3.5 = 158.5, times 1, plus 3 -> 161.5;
    p = 2000, u = 2.5, v = 1: 155 + 7 = 162, plus 2.5 -> 164.5;
    p = 0, u = -100 (outside the drawn range), v = 1: 55 -> clipped up to 150;
    p = 10^6, u = 1, v = 1: 3655 + 1 -> clipped down to 1120;
    p = 0, u = 2, v = 0.5: 77.5 + 2 = 79.5 -> 150."""
    assert O.ttft_target(1000, 3.0, 1.0) == 161.5
    assert O.ttft_target(2000, 2.5, 1.0) == 164.5
    assert O.ttft_target(0, -100.0, 1.0) == 150.0
    assert O.ttft_target(10 ** 6, 1.0, 1.0) == 1120.0
    assert O.ttft_target(0, 2.0, 0.5) == 150.0
    p = np.array([1000, 2000, 0, 10 ** 6], np.int32)
    got = O.ttft_targets(p, [3.0, 2.5, -100.0, 1.0], [1.0, 1.0, 1.0, 1.0])
    assert list(got) == [161.5, 164.5, 150.0, 1120.0]


@pytest.mark.parametrize("p", [0, 1000, 50000])
def test_ttft_target_expectation(p):
    """The paper gives E[tau] ~= 158 + 3.5e-3 * p ms for unclipped targets
    (u ~ U(1, 5) ms, v ~ U(0.98, 1.02)); the sample mean of 200k targets is within
    0.05 ms of it (standard error ~0.005 ms)."""
    rng = np.random.default_rng(11)
    n = 200_000
    tau = O.ttft_targets(np.full(n, p, np.int32), rng.uniform(1, 5, n), rng.uniform(0.98, 1.02, n))
    assert abs(tau.mean() - (158.0 + 3.5e-3 * p)) < 0.05
    assert tau.min() >= 150.0 and tau.max() <= 1120.0


def test_constrained_route_hand_cases():
    """Eq. 3 on hand-made rows (utility = acc - 0.5 * cost, one column per instance):
    utilities [0.9, 0.1, 0.5], TTFT [5, 3, 9]."""
    col = np.array([0, 1, 2], np.int32)
    acc, cost = np.array([1.0, 0.2, 0.75]), np.array([0.2, 0.2, 0.5])
    ttft = np.array([5.0, 3.0, 9.0])
    # only instance 1 meets tau = 4, although instance 0 has the higher utility
    assert O.route_row_constrained(ttft, 4.0, acc, cost, col, 0.5) == 1
    # the target is inclusive: tau = 5 admits instance 0, the best utility
    assert O.route_row_constrained(ttft, 5.0, acc, cost, col, 0.5) == 0
    # everything feasible: plain argmax of the utility
    assert O.route_row_constrained(ttft, 100.0, acc, cost, col, 0.5) == 0
    # nothing feasible: least estimated TTFT
    assert O.route_row_constrained(ttft, 2.0, acc, cost, col, 0.5) == 1
    # ties: equal utilities -> lower index; equal TTFT with nothing feasible -> lower index
    assert O.route_row_constrained(np.array([1.0, 1.0]), 5.0, np.array([0.5, 0.5]),
                                   np.zeros(2), np.array([0, 1], np.int32), 1.0) == 0
    assert O.route_row_constrained(np.array([7.0, 7.0, 8.0]), 5.0, acc, cost, col, 0.5) == 0
    # feasible set {2} only (instance 2 is the slowest but the only one within tau)
    assert O.route_row_constrained(np.array([9.0, 9.5, 4.0]), 5.0, acc, cost, col, 0.5) == 2


def test_constrained_route_special_cases_and_definition():
    """tau = +inf reduces Eq. 3 to the Lagrangian route with delta = 0 (pinned above);
    tau = -inf to numpy's argmin of the TTFT; random rows with coarse values (many
    ties) match the set-based statement of Eq. 3."""
    rng = np.random.default_rng(12)
    for _ in range(500):
        I = int(rng.integers(1, 30))
        n_cols = int(rng.integers(1, 4))
        col = rng.integers(0, n_cols, size=I).astype(np.int32)
        ttft = rng.integers(0, 6, size=I) * 0.5
        acc = rng.integers(0, 4, size=n_cols) / 4.0
        cost = rng.integers(0, 4, size=n_cols) / 4.0
        wc = float(rng.integers(0, 3)) / 2
        m_inf = O.route_row_constrained(ttft, np.inf, acc, cost, col, wc)
        assert m_inf == O.route_row(ttft, acc, cost, col, wc, 0.0)[0]
        assert O.route_row_constrained(ttft, -np.inf, acc, cost, col, wc) == int(np.argmin(ttft))
        tau = float(rng.integers(0, 6)) * 0.5
        util = acc[col] - wc * cost[col]
        assert O.route_row_constrained(ttft, tau, acc, cost, col, wc) == \
            BF._pick_constrained(ttft, util, tau)


def test_ontime_utility_cases():
    """Eq. 4: with every TTFT within its target it is the mean utility of the stats
    (same fold), with none it is 0, and a hand case: utilities [0.5, -0.25, 1.0],
    on time [yes, yes, no] -> (0.5 - 0.25) / 3."""
    rng = np.random.default_rng(13)
    n, n_cols = 257, 3
    col = np.array([0, 1, 2, 2], np.int32)
    choice = rng.integers(0, 4, size=n).astype(np.int32)
    ttft = rng.random(n) * 100
    acc, cost = rng.random((n, n_cols)), rng.random((n, n_cols))
    s = O.stats(choice, ttft, acc, cost, col, 0.3)
    assert O.ontime_utility(choice, ttft, np.full(n, np.inf), acc, cost, col, 0.3) == s[2]
    assert O.ontime_utility(choice, ttft, np.full(n, -np.inf), acc, cost, col, 0.3) == 0.0
    acc3 = np.array([[0.5], [0.0], [1.0]])
    cost3 = np.array([[0.0], [0.25], [0.0]])
    got = O.ontime_utility(np.zeros(3, np.int32), np.array([1.0, 2.0, 3.0]),
                           np.array([1.0, 5.0, 2.5]), acc3, cost3, np.array([0], np.int32), 1.0)
    assert got == (0.5 - 0.25) / 3


@pytest.mark.parametrize("seed", range(24))
def test_bruteforce_constrained_traces(seed):
    """Whole traces under Eq. 3 against the token-at-a-time scheduler with the
    set-based route; targets drawn inside the range of the TTFTs so that both the
    feasible branch and the empty-set fallback occur."""
    wl = make_tiny_workload(200 + seed, n_inst=3, max_res=5, n_q=25, dyadic=(seed % 2 == 0),
                            n_scen=1)
    lam = O.trace(wl, full_rows=True, queue_cap=10 ** 6)
    lo, hi = float(lam.ttft_all.min()), float(lam.ttft_all.max())
    tau = np.random.default_rng(seed).uniform(lo, hi, size=wl.n_q)
    r = O.trace(wl, full_rows=True, queue_cap=10 ** 6, tau=tau)
    real = np.zeros(wl.n_q)
    ch, rows, insts = BF.trace(wl, tau=tau, realized=real)
    np.testing.assert_array_equal(r.choice, ch)
    assert np.array_equal(r.ttft_all.view(np.int64), rows.view(np.int64))
    assert np.array_equal(r.realized.view(np.int64), real.view(np.int64))
    for j, x in enumerate(insts):
        a, b = r.offsets[j], r.offsets[j + 1]
        got = list(zip(r.rem_prefill[a:b], r.rem_decode[a:b], r.context[a:b]))
        assert [tuple(int(v) for v in g) for g in got] == x.state()


# ------------------------------------------------------------------ realised TTFT
def _hand_trace_workload():
    """One empty instance, B = 8, M = 4, T = 1 + 0.5 P + 0.25 D; query 0 (p = 10,
    d = 2) at 0 ms, query 1 (p = 5, d = 1) at 0.5 ms."""
    base = make_tiny_workload(0, n_inst=1, n_q=2)
    return dataclasses.replace(
        base, n_inst=1, a=np.array([1.0]), b=np.array([0.5]), c=np.array([0.25]),
        d=np.zeros(1), e=np.zeros(1), budget=np.array([8], np.int32),
        max_seqs=np.array([4], np.int32), col=np.zeros(1, np.int32),
        offsets=np.zeros(2, np.int32), rem_prefill=np.zeros(0, np.int32),
        rem_decode=np.zeros(0, np.int32), context=np.zeros(0, np.int32),
        clock_ms=np.zeros(1), q_prefill=np.array([10, 5], np.int32),
        q_decode=np.array([2, 1], np.int32), q_t_ms=np.array([0.0, 0.5]),
        acc=np.full((2, 1), 0.5), cost=np.zeros((2, 1)), w_cost=np.zeros(1),
        w_lat_ms=np.zeros(1), queue_cap=8, max_prompt=16)


@pytest.mark.parametrize("reading", [0, 1])
def test_realized_hand_worked(reading):
    """Worked by hand.  Query 0 alone: batches of 8 and 2 prefill tokens (5 and 2 ms)
    and a decode batch (1.25 ms): estimate 8.25 ms (7 ms under reading 1).  The
    replay runs the 8-token batch before query 1 arrives at 0.5 ms (clock 5); query
    1 then shares the next batch: 2 + 5 prefill tokens (4.5 ms, both prefills done
    at 9.5), then both decode (1.5 ms, 11.0).  Query 1's estimate is exact (10.5;
    9.0 under reading 1); query 0's first token comes 2.75 ms (2.5 ms) later than
    its estimate, because of query 1's tokens."""
    wl = _hand_trace_workload()
    r = O.trace(wl, reading=reading, queue_cap=8)
    real = np.zeros(2)
    BF.trace(wl, reading=reading, realized=real)
    if reading == 0:
        assert list(r.ttft_chosen) == [8.25, 10.5]
        assert list(r.realized) == [11.0, 10.5]
    else:
        assert list(r.ttft_chosen) == [7.0, 9.0]
        assert list(r.realized) == [9.5, 9.0]
    assert list(real) == list(r.realized)
    # the trace's own end state is the replay to the last arrival, not the drain
    assert r.clock_ms[0] == 5.0


def _realized_properties(wl, r):
    """A later query only adds tokens to batches (under FCFS it never takes budget or
    a slot ahead of an earlier one), and batch time does not decrease with tokens:
    the realised TTFT is never below the estimate at the choice, and equals it when
    no later query joins the same instance before the first token."""
    N = len(r.choice)
    assert not np.isnan(r.realized).any()
    assert (r.realized >= r.ttft_chosen).all()
    t = wl.q_t_ms[:N]
    for i in range(N):
        later = np.nonzero(r.choice[i + 1:] == r.choice[i])[0]
        if later.size == 0 or t[i + 1 + later[0]] >= t[i] + r.realized[i]:
            assert r.realized[i] == r.ttft_chosen[i], i


@pytest.mark.parametrize("reading", [0, 1])
def test_realized_properties_c1(reading):
    from workloads import make_workload
    wl = make_workload("c1")
    r = O.trace(wl, reading=reading)
    _realized_properties(wl, r)
    assert (r.realized > r.ttft_chosen).sum() > 0   # the case the estimate misses occurs


@pytest.mark.parametrize("seed", range(12))
def test_realized_properties_tiny(seed):
    wl = make_tiny_workload(400 + seed, n_inst=2, max_res=4, n_q=40, mean_gap_ms=1.0,
                            n_scen=1)
    for reading in (0, 1):
        _realized_properties(wl, O.trace(wl, reading=reading, queue_cap=10 ** 6))


# ------------------------------------------------------------------ threads
def _same_trace(a, b):
    for f in ("choice", "ttft_chosen", "util_chosen", "ttft_all", "iters_all", "offsets",
              "rem_prefill", "rem_decode", "context", "clock_ms", "iterations", "realized"):
        x, y = getattr(a, f), getattr(b, f)
        if x is None:
            assert y is None
            continue
        x, y = np.asarray(x), np.asarray(y)
        if x.dtype == np.float64:
            x, y = x.view(np.int64), y.view(np.int64)
        np.testing.assert_array_equal(x, y, err_msg=f)


def test_threaded_oracle_is_bit_identical():
    """The oracle's loops over independent instances (estimates of one query, the
    replays) and over the pairs of a what-if matrix, and scenarios run on threads of
    their own, give exactly the single-threaded results: c1 and c7 in full, c2 and
    c4 prefixes with every TTFT row, c3 what-if rows, c5 scenarios."""
    from workloads import make_workload
    cases = [("c1", None, {}), ("c7", 1500, {}), ("c2", 1500, {}), ("c4", 3, {}),
             ("c2", 400, {"tau": "targets"})]
    try:
        for name, n_q, kw in cases:
            wl = make_workload(name)
            if kw.get("tau") == "targets":
                kw = {"tau": O.ttft_targets(wl.q_prefill, wl.tau_u_ms, wl.tau_v)}
            O.set_threads(1)
            one = O.trace(wl, n_q=n_q, full_rows=True, **kw)
            O.set_threads(4)
            four = O.trace(wl, n_q=n_q, full_rows=True, **kw)
            _same_trace(one, four)
        wl = make_workload("c3")
        rows = [0, 1, int(np.argmax(wl.q_prefill))]
        O.set_threads(1)
        t1, i1 = O.estimate_matrix_all(wl, queries=rows)
        O.set_threads(4)
        t4, i4 = O.estimate_matrix_all(wl, queries=rows)
        np.testing.assert_array_equal(t1.view(np.int64), t4.view(np.int64))
        np.testing.assert_array_equal(i1, i4)
        # the literal per-pair estimate of the Python loop gives the same values
        ref, ref_it = O.estimate_matrix(wl, rows[:1], range(0, wl.n_inst, 97))
        np.testing.assert_array_equal(ref.view(np.int64), t1[:1, ::97].view(np.int64))
        np.testing.assert_array_equal(ref_it, i1[:1, ::97])
    finally:
        O.set_threads(1)
    wl = make_workload("c5", n_q=150)
    seq = O.trace_scenarios(wl, [0, 9, 63], 1)
    par = O.trace_scenarios(wl, [0, 9, 63], 3)
    for a, b in zip(seq, par):
        _same_trace(a, b)
