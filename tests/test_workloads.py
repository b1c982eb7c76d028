"""Input generators: the MMPP-2 arrival process (appendix on correlated query
arrivals) against the paper's table of rates and its stated long-run behaviour."""

import json
import os

import numpy as np
import pytest

from workloads import make_workload
from workloads.gen import mmpp2_arrivals_ms, mmpp2_rates

GOLD = os.path.join(os.path.dirname(__file__), "golden", "mmpp2_rates.json")


def test_mmpp2_rates_match_paper_table():
    g = json.load(open(GOLD))
    for row in g["rows"]:
        low, high = mmpp2_rates(row["mean_qps"], row["r"], g["p_high"])
        assert round(low, 2) == row["low"] and round(high, 2) == row["high"], row


@pytest.mark.parametrize("r", [3.0, 6.0])
def test_mmpp2_long_run_rate_and_burstiness(r):
    """Long-run mean rate (it comes out right only with the 20 % of time in the high
    state that the transition rates 0.1 and 0.4 per second imply) and over-dispersed
    counts (index of dispersion of 1-s counts well above the Poisson value 1)."""
    mean = 7.0
    t = mmpp2_arrivals_ms(np.random.default_rng(5), 200_000, mean, r, 0.2, 0.1, 0.4) / 1000.0
    assert np.all(np.diff(t) >= 0)
    rate = len(t) / t[-1]
    assert abs(rate - mean) / mean < 0.03, rate
    counts = np.bincount(t.astype(np.int64))
    assert counts.var() / counts.mean() > 2.0
    # a Poisson path of the same mean is not over-dispersed
    p = np.cumsum(np.random.default_rng(6).exponential(1 / mean, 200_000))
    pc = np.bincount(p.astype(np.int64))
    assert 0.8 < pc.var() / pc.mean() < 1.2


def test_bursty_config_keeps_the_poisson_twins_queries():
    a = make_workload("c2", n_q=2000)
    b = make_workload("c6", n_q=2000)
    np.testing.assert_array_equal(a.q_prefill, b.q_prefill)
    np.testing.assert_array_equal(a.acc, b.acc)
    assert not np.array_equal(a.q_t_ms, b.q_t_ms)
    assert np.all(np.diff(b.q_t_ms) >= 0)
