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
        ch, rows, insts = BF.trace(wl, reading=reading)
        np.testing.assert_array_equal(r.choice, ch)
        assert np.array_equal(r.ttft_all.view(np.int64), rows.view(np.int64))
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
