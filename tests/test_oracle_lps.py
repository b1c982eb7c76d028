"""Pins of the oracle's average-case LPS estimator (Sec. 4.2, Eqs. 10-11; the appendix
on the limited-processor-sharing abstraction, Eqs. 12-13) against what the
mathematics fixes independently of its closed form:

* the textbook M/M/1 mean queueing delay at k = 1;
* the appendix's own series (the stationary distribution times the delay given the
  state seen on arrival), summed term by term;
* the limits the appendix states (k -> infinity gives 0; monotone in k and in load);
* Eq. 13 at c_a^2 = c_s^2 = 1 equals Eq. 12, and at k = 1 is Kingman's G/G/1 form;
* a literal discrete-event simulation of an LPS server within 3 standard errors;
* the TTFT of Eq. 11 in exact rational arithmetic, and, with no queueing, the SFS
  estimate of an empty instance (Sec. 4.1) with the matching coefficients.
"""

from __future__ import annotations

from fractions import Fraction as F

import numpy as np
import pytest

from lps_sim import mean_and_se, simulate_waits
from oracle import oracle as O


def _bits(x):
    return np.float64(x).view(np.int64)


def test_k1_is_the_textbook_mm1_delay():
    """k = 1: W = alpha / (mu (mu - alpha)), the M/M/1 mean delay in queue; with mu a
    power of two both forms are one rounding of the same quotient."""
    rng = np.random.default_rng(0)
    for _ in range(300):
        mu = 2.0 ** int(rng.integers(-8, 4))
        alpha = mu * int(rng.integers(1, 255)) / 256.0
        want = alpha / (mu * (mu - alpha))
        assert _bits(O.lps_wait(alpha, mu, 1)) == _bits(want), (alpha, mu)


@pytest.mark.parametrize("alpha,mu,k", [(0.3, 1.1, 1), (0.7, 1.3, 3), (0.02, 0.025, 7),
                                        (4.9, 5.0, 25), (0.5, 3.0, 2)])
def test_series_of_the_derivation(alpha, mu, k):
    """E[W] = sum_{n >= k} (1 - rho) rho^n (n - k + 1) / mu, summed term by term."""
    rho = alpha / mu
    n = np.arange(k, k + 200000, dtype=np.float64)
    terms = (1.0 - rho) * rho ** n * (n - k + 1) / mu
    s = float(np.sum(terms[::-1]))
    w = O.lps_wait(alpha, mu, k)
    assert abs(w - s) <= 1e-12 * s, (w, s)


def test_limits_and_monotonicity():
    assert O.lps_wait(0.5, 1.0, 5000) == 0.0          # every query enters service at once
    assert O.lps_wait(0.0, 1.0, 3) == 0.0             # no arrivals, no waiting
    ws = [O.lps_wait(0.8, 1.0, k) for k in range(1, 60)]
    assert all(a > b for a, b in zip(ws, ws[1:]))     # geometric decay in k
    ws = [O.lps_wait(a, 1.0, 4) for a in np.linspace(0.05, 0.95, 30)]
    assert all(a < b for a, b in zip(ws, ws[1:]))     # grows with the load
    assert O.lps_wait(0.5, 1.0, 65536) == 0.0
    for bad in [(1.0, 1.0, 2), (1.5, 1.0, 2), (-0.1, 1.0, 2), (0.5, 1.0, 0), (0.5, 1.0, 65537),
                (np.nan, 1.0, 2), (0.5, np.inf, 2)]:
        assert np.isnan(O.lps_wait(*bad)), bad
    assert np.isnan(O.lps_wait(0.5, 1.0, 2, O.LPS_VARIABILITY, -1.0, 1.0))
    assert np.isnan(O.lps_ttft(0.5, 1.0, 2, 0.0, 1.0, 10))     # theta must be positive
    assert np.isnan(O.lps_ttft(0.5, 1.0, 2, 4.0, -1.0, 10))    # decode time >= 0
    assert np.isnan(O.lps_ttft(0.5, 1.0, 2, 4.0, 1.0, 0))      # a prompt has a token


def test_variability_form_reduces():
    """Eq. 13 with c_a^2 = c_s^2 = 1 is Eq. 12; at k = 1 it is Kingman's
    ((c_a^2 + c_s^2) / 2) (rho / (1 - rho)) E[S]; it scales with (c_a^2 + c_s^2) / 2.
    mu a power of two and dyadic alpha keep every step a single rounding of the same
    quotient, so equality is bitwise."""
    rng = np.random.default_rng(1)
    for _ in range(300):
        mu = 2.0 ** int(rng.integers(-6, 3))
        alpha = mu * int(rng.integers(1, 63)) / 64.0
        k = int(rng.integers(1, 12))
        w12 = O.lps_wait(alpha, mu, k)
        assert _bits(O.lps_wait(alpha, mu, k, O.LPS_VARIABILITY, 1.0, 1.0)) == _bits(w12)
        ca2, cs2 = int(rng.integers(0, 9)) / 4.0, int(rng.integers(0, 9)) / 4.0
        rho = alpha / mu
        king = ((ca2 + cs2) / 2.0) * (rho / (1.0 - rho)) * (1.0 / mu)
        assert _bits(O.lps_wait(alpha, mu, 1, O.LPS_VARIABILITY, ca2, cs2)) == _bits(king)
        h = (ca2 + cs2) / 2.0
        assert _bits(O.lps_wait(alpha, mu, k, O.LPS_VARIABILITY, ca2, cs2)) == _bits(h * w12)


@pytest.mark.parametrize("alpha,mu,k,seed", [(0.6, 1.0, 1, 3), (0.75, 1.0, 2, 4),
                                             (0.7, 1.0, 4, 12), (0.3, 0.5, 3, 21)])
def test_discrete_event_simulation(alpha, mu, k, seed):
    """A literal event-by-event LPS server (tests/lps_sim.py) agrees with Eq. 12
    within 3 standard errors (batch means over 200k arrivals)."""
    m, se = mean_and_se(simulate_waits(alpha, mu, k, 200_000, seed), 5000)
    w = O.lps_wait(alpha, mu, k)
    assert abs(m - w) <= 3 * se, (m, se, w)


def test_ttft_exact_and_against_sfs_empty_instance():
    rng = np.random.default_rng(2)
    for _ in range(200):
        mu = 2.0 ** int(rng.integers(-6, 3))
        alpha = mu * int(rng.integers(1, 63)) / 64.0
        k = int(rng.integers(1, 8))
        theta = 2.0 ** int(rng.integers(-3, 6))
        t_dec = int(rng.integers(0, 64)) / 8.0
        p = int(rng.integers(1, 5000))
        w = O.lps_wait(alpha, mu, k)
        exact = F(w) + F(p) / F(theta) + F(t_dec)
        got = O.lps_ttft(alpha, mu, k, theta, t_dec, p)
        assert got == float(exact) or abs(F(got) - exact) <= abs(exact) * F(2) ** -52
        assert _bits(got) == _bits((w + p / theta) + t_dec)
    # no queueing (k large): prefill at throughput theta = 1/b plus one decode batch of
    # time c is the SFS estimate of an empty instance with a = d = e = 0 (reading: the
    # first token comes in the decode batch after the prefill), prompts within budget
    for b_exp, c, p in [(-6, 0.75, 100), (-3, 2.5, 2048), (-9, 0.125, 1)]:
        b = 2.0 ** b_exp
        par = O.make_params(0.0, b, c, 0.0, 0.0, 4096, 64)
        sfs, _ = O.Queue(par, [], [], []).estimate(p, 1, 0.0)
        lps = O.lps_ttft(0.25, 1.0, 5000, 1.0 / b, c, p)
        assert _bits(lps) == _bits(sfs), (lps, sfs)


def test_matrix_is_the_pairwise_estimate():
    rng = np.random.default_rng(3)
    I, Q = 7, 11
    prm = dict(alpha=rng.random(I) * 0.5, mu=0.6 + rng.random(I), k=rng.integers(1, 30, I),
               ca2=rng.random(I) * 2, cs2=rng.random(I) * 2, theta=1 + rng.random(I) * 20,
               t_dec=rng.random(I) * 30)
    p = rng.integers(1, 4000, Q)
    for mode in (O.LPS_POISSON, O.LPS_VARIABILITY):
        m = O.lps_matrix(prm, p, mode)
        for i in range(Q):
            for j in range(I):
                want = O.lps_ttft(prm["alpha"][j], prm["mu"][j], prm["k"][j], prm["theta"][j],
                                  prm["t_dec"][j], p[i], mode, prm["ca2"][j], prm["cs2"][j])
                assert _bits(m[i, j]) == _bits(want)
