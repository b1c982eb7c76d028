"""A literal discrete-event simulation of a limited-processor-sharing server
(appendix on the LPS abstraction): Poisson arrivals at rate alpha; each query
brings an exponential amount of work with mean 1 (one query's worth); the server
processes mu work per ms in total, shared equally by at most k active queries; the
other queries wait in FCFS order and enter the active set, one per completion, as
soon as fewer than k are active.  A query's queueing delay is the time from its
arrival to its entry into the active set.

Independent of the closed forms it checks: it follows the system's definition event
by event, with each active query's remaining work tracked explicitly (it does not
use the birth-death argument of the derivation)."""

from __future__ import annotations

import numpy as np


def simulate_waits(alpha: float, mu: float, k: int, n_arrivals: int, seed: int) -> np.ndarray:
    """Queueing delays (ms) of the first n_arrivals queries, starting empty."""
    rng = np.random.default_rng(seed)
    arrive = np.cumsum(rng.exponential(1.0 / alpha, n_arrivals))
    work = rng.exponential(1.0, n_arrivals)
    waits = np.full(n_arrivals, np.nan)
    active = []               # remaining work of the active queries
    waiting = []              # FCFS: indices of waiting queries
    head = 0
    now = 0.0
    i = 0                     # next arriving query
    while i < n_arrivals or active:
        n_a = len(active)
        t_done = now + min(active) * n_a / mu if n_a else np.inf
        if i < n_arrivals and arrive[i] <= t_done:
            if n_a:
                served = (arrive[i] - now) * mu / n_a
                active = [r - served for r in active]
            now = arrive[i]
            if len(active) < k:
                active.append(work[i])
                waits[i] = 0.0
            else:
                waiting.append(i)
            i += 1
        else:
            served = (t_done - now) * mu / n_a
            m = min(range(n_a), key=active.__getitem__)
            active = [r - served for r in active]
            active.pop(m)
            now = t_done
            if head < len(waiting):
                q = waiting[head]
                head += 1
                waits[q] = now - arrive[q]
                active.append(work[q])
    return waits


def mean_and_se(waits: np.ndarray, warmup: int, n_batches: int = 20):
    """Mean delay after a warm-up and its standard error by batch means."""
    w = waits[warmup:]
    b = len(w) // n_batches
    means = w[:b * n_batches].reshape(n_batches, b).mean(axis=1)
    return float(means.mean()), float(means.std(ddof=1) / np.sqrt(n_batches))
