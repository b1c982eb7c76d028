"""Seeded input generation (numpy PCG64).  Draws inputs only; computes no results.

Draw order for a config (one ``np.random.default_rng(seed)`` stream):
  1. instances, instance-major; per instance: prompt lengths [R], predicted
     remaining decode lengths [R], extra decoded tokens g [R];
  2. queries: inter-arrival times [N] (when the config has an arrival rate),
     prompt lengths [N], predicted decode lengths [N];
  3. accuracy predictions;
  4. cost predictions (only the uniform layout draws; the token-price layout is a
     deterministic function of the query lengths).
Two more streams draw the per-query variables of the TTFT targets (appendix on
TTFT latency assignment): ``default_rng([seed, 1])`` u ~ U(1, 5) ms and
``default_rng([seed, 2])`` v ~ U(0.98, 1.02), [N] each.  A config with MMPP-2
arrivals (appendix on correlated query arrivals) still draws the Poisson gaps of
step 2 and replaces the arrival times by an MMPP-2 path drawn from
``default_rng([seed, 3])``, so its queries are those of the Poisson twin.  The targets themselves are computed by the
library and by the oracle, not here.

Initial resident queue of an instance, in arrival (FCFS) order:
  * the first n_dec = min(R // 2, M - 1) requests are decoding:
    remaining prefill 0, context = prompt + g;
  * the next one is a partially prefilled running request:
    context = prompt // 2, remaining prefill = prompt - prompt // 2;
  * the rest are waiting: context 0, remaining prefill = prompt.
Every request carries its drawn remaining decode length (>= 1).
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from .configs import get_config


@dataclass
class Workload:
    name: str
    n_scen: int
    n_inst: int
    # per-instance parameters
    a: np.ndarray
    b: np.ndarray
    c: np.ndarray
    d: np.ndarray
    e: np.ndarray
    budget: np.ndarray        # int32 [I]
    max_seqs: np.ndarray      # int32 [I]
    col: np.ndarray           # int32 [I]: acc/cost column of each instance
    # snapshot, CSR over instances, FCFS order inside an instance
    offsets: np.ndarray       # int32 [I+1]
    rem_prefill: np.ndarray   # int32 [n_req]
    rem_decode: np.ndarray    # int32 [n_req]
    context: np.ndarray       # int32 [n_req]
    clock_ms: np.ndarray      # float64 [I]
    # query trace
    q_prefill: np.ndarray     # int32 [N]
    q_decode: np.ndarray      # int32 [N]
    q_t_ms: np.ndarray        # float64 [N]
    # predictions, [N][n_cols]
    acc: np.ndarray
    cost: np.ndarray
    # routing weights per scenario
    w_cost: np.ndarray        # float64 [Z]   (lambda)
    w_lat_ms: np.ndarray      # float64 [Z]   (delta per ms = delta_per_s / 1000)
    # draws of the TTFT targets, [N]
    tau_u_ms: np.ndarray
    tau_v: np.ndarray
    queue_cap: int
    max_prompt: int
    meta: dict = field(default_factory=dict)
    # scheduler limits per instance, int32 [I][4]: chunk cap, KV blocks, block size,
    # context limit (0 = none); None: the default batch with no limits
    sched: np.ndarray | None = None

    @property
    def n_q(self) -> int:
        return int(self.q_prefill.shape[0])

    @property
    def n_cols(self) -> int:
        return int(self.acc.shape[1])

    def instance_requests(self, j: int):
        lo, hi = int(self.offsets[j]), int(self.offsets[j + 1])
        return (self.rem_prefill[lo:hi], self.rem_decode[lo:hi], self.context[lo:hi])


def _draw_target_vars(seed, n):
    u = np.random.default_rng([int(seed), 1]).uniform(1.0, 5.0, size=n)
    v = np.random.default_rng([int(seed), 2]).uniform(0.98, 1.02, size=n)
    return np.ascontiguousarray(u), np.ascontiguousarray(v)


def mmpp2_rates(mean_rate, r, p_high):
    """Low- and high-state rates of a two-state Markov-modulated Poisson process with
    long-run mean rate ``mean_rate``, rate ratio r = high/low and high-state time
    fraction p_high (appendix on correlated query arrivals)."""
    low = mean_rate / ((1.0 - p_high) + p_high * r)
    return low, r * low


def mmpp2_arrivals_ms(rng, n, mean_rate, r, p_high, z_lh, z_hl):
    """n arrival times (ms, from t = 0) of an MMPP-2: a latent two-state Markov chain
    (transition rates z_lh and z_hl per second, started from its stationary law)
    modulating Poisson arrivals at the low or high rate.  Competing exponential
    clocks: the next event is an arrival with probability rate / (rate + switch)."""
    low, high = mmpp2_rates(mean_rate, r, p_high)
    state = 1 if rng.random() < z_lh / (z_lh + z_hl) else 0
    t = 0.0
    out = np.empty(n)
    k = 0
    while k < n:
        lam = high if state else low
        sw = z_hl if state else z_lh
        t += rng.exponential(1.0 / (lam + sw))
        if rng.random() < lam / (lam + sw):
            out[k] = t
            k += 1
        else:
            state = 1 - state
    return 1000.0 * out


def _draw_prompts(rng, spec, size):
    kind = spec[0]
    if kind == "uniform":
        lo, hi = spec[1], spec[2]
        return rng.integers(lo, hi + 1, size=size).astype(np.int32)
    if kind == "lognormal":
        mu, sigma, lo, hi = spec[1:]
        x = np.rint(rng.lognormal(mu, sigma, size=size))
        return np.clip(x, lo, hi).astype(np.int32)
    raise ValueError(f"unknown prompt distribution {kind!r}")


def _initial_queue(prompts, decodes, extra, max_seqs):
    R = prompts.shape[0]
    n_dec = min(R // 2, max_seqs - 1)
    rp = np.empty(R, np.int32)
    cx = np.empty(R, np.int32)
    rp[:n_dec] = 0
    cx[:n_dec] = prompts[:n_dec] + extra[:n_dec]
    if R > n_dec:
        p = int(prompts[n_dec])
        half = p // 2
        cx[n_dec] = half
        rp[n_dec] = p - half
    rp[n_dec + 1:] = prompts[n_dec + 1:]
    cx[n_dec + 1:] = 0
    return rp, decodes.astype(np.int32), cx


def make_workload(name: str, *, n_q: int | None = None, n_inst: int | None = None,
                  resident: int | None = None, n_scen: int | None = None,
                  seed: int | None = None, queue_cap: int | None = None) -> Workload:
    """Draw the workload of config ``name``; the keyword arguments shrink it for tests."""
    cfg = get_config(name)
    if n_inst is not None and n_inst != cfg["n_inst"]:
        n_types = len(cfg["types"])
        cfg["type_of_inst"] = [j * n_types // n_inst for j in range(n_inst)]
        cfg["n_inst"] = n_inst
    if n_q is not None:
        cfg["n_q"] = n_q
    if resident is not None:
        cfg["resident"] = resident
    if n_scen is not None:
        cfg["weights"] = cfg["weights"][:n_scen]
        cfg["n_scen"] = n_scen
    if seed is not None:
        cfg["seed"] = seed
    if queue_cap is not None:
        cfg["queue_cap"] = queue_cap
    return _build(cfg)


def _build(cfg: dict) -> Workload:
    rng = np.random.default_rng(cfg["seed"])
    I, R, N = cfg["n_inst"], cfg["resident"], cfg["n_q"]
    types = cfg["types"]
    tof = np.asarray(cfg["type_of_inst"], np.int32)
    M = cfg["max_seqs"]
    p_dec = 1.0 / cfg["decode_mean"]

    offsets = np.zeros(I + 1, np.int32)
    rps, rds, cxs = [], [], []
    for j in range(I):
        prompts = _draw_prompts(rng, cfg["prompt"], R)
        decodes = rng.geometric(p_dec, size=R)
        extra = rng.integers(0, 256, size=R)
        rp, rd, cx = _initial_queue(prompts, decodes, extra, M)
        rps.append(rp), rds.append(rd), cxs.append(cx)
        offsets[j + 1] = offsets[j] + R

    if cfg["rate_per_s"] is not None:
        inter = rng.exponential(1.0 / cfg["rate_per_s"], size=N)
        t_ms = 1000.0 * np.cumsum(inter)
        arr = cfg.get("arrivals", ("poisson",))
        if arr[0] == "mmpp2":   # drawn from a stream of its own: other draws unchanged
            t_ms = mmpp2_arrivals_ms(np.random.default_rng([int(cfg["seed"]), 3]), N,
                                     cfg["rate_per_s"], *arr[1:])
        elif arr[0] != "poisson":
            raise ValueError(arr)
    else:
        t_ms = np.zeros(N)
    q_prefill = _draw_prompts(rng, cfg["prompt"], N)
    q_decode = rng.geometric(p_dec, size=N).astype(np.int32)

    if cfg["acc"] == "per_type":
        acc = rng.random((N, len(types)))
        col = tof.copy()
    elif cfg["acc"] == "per_instance":
        acc = rng.random((N, I))
        col = np.arange(I, dtype=np.int32)
    else:
        raise ValueError(cfg["acc"])

    if cfg["cost"] == "tokens_x_price":
        if cfg["acc"] != "per_type":
            raise ValueError("token-price cost is defined per model type")
        prices = np.array([t["price"] for t in types])
        raw = (q_prefill.astype(np.float64) + q_decode)[:, None] * prices[None, :]
        cost = raw / raw.max() if N else raw
    elif cfg["cost"] == "uniform":
        cost = rng.random(acc.shape)
    else:
        raise ValueError(cfg["cost"])

    w = np.asarray(cfg["weights"], np.float64).reshape(-1, 2)
    tau_u, tau_v = _draw_target_vars(cfg["seed"], N)
    sched = None
    if cfg.get("sched") is not None:
        lim = cfg["sched"]
        sched = np.tile(np.array([lim["chunk_cap"], lim["kv_blocks"], lim["block_size"],
                                  lim["max_ctx"]], np.int32), (I, 1))
    return Workload(
        name=cfg["name"], n_scen=int(w.shape[0]), n_inst=I,
        a=np.array([types[t]["a"] for t in tof]), b=np.array([types[t]["b"] for t in tof]),
        c=np.array([types[t]["c"] for t in tof]), d=np.array([types[t]["d"] for t in tof]),
        e=np.array([types[t]["e"] for t in tof]),
        budget=np.full(I, cfg["budget"], np.int32), max_seqs=np.full(I, M, np.int32),
        col=col.astype(np.int32),
        offsets=offsets,
        rem_prefill=np.concatenate(rps) if rps else np.zeros(0, np.int32),
        rem_decode=np.concatenate(rds) if rds else np.zeros(0, np.int32),
        context=np.concatenate(cxs) if cxs else np.zeros(0, np.int32),
        clock_ms=np.zeros(I),
        q_prefill=q_prefill, q_decode=q_decode, q_t_ms=t_ms,
        acc=np.ascontiguousarray(acc), cost=np.ascontiguousarray(cost),
        w_cost=np.ascontiguousarray(w[:, 0]), w_lat_ms=np.ascontiguousarray(w[:, 1] / 1000.0),
        tau_u_ms=tau_u, tau_v=tau_v,
        queue_cap=int(cfg["queue_cap"]), max_prompt=int(cfg["max_prompt"]),
        meta=cfg, sched=sched,
    )


def make_tiny_workload(seed: int, *, n_inst: int = 3, max_res: int = 4, budget=(1, 8),
                       max_seqs=(1, 4), prompt=(1, 12), decode=(1, 5), n_q: int = 20,
                       mean_gap_ms: float = 3.0, n_scen: int = 1, coef_scale: float = 1.0,
                       dyadic: bool = False) -> Workload:
    """Small random pools for exhaustive and property checks.

    Every resident request is decoding, partially prefilled or waiting, in a valid
    FCFS order (running before waiting, at most M running).  With ``dyadic`` the
    coefficients are small dyadic rationals, so every binary64 sum of batch times in
    a short trace is exact.
    """
    rng = np.random.default_rng(seed)
    I = n_inst
    B = rng.integers(budget[0], budget[1] + 1, size=I).astype(np.int32)
    M = np.minimum(rng.integers(max_seqs[0], max_seqs[1] + 1, size=I), B).astype(np.int32)
    if dyadic:
        def coef():
            return rng.integers(0, 9, size=I) / 8.0 * coef_scale
    else:
        def coef():
            return rng.random(I) * coef_scale
    a, b, c, d, e = coef(), coef(), coef(), coef(), coef()
    offsets = np.zeros(I + 1, np.int32)
    rps, rds, cxs = [], [], []
    for j in range(I):
        n = int(rng.integers(0, max_res + 1))
        n_run = int(rng.integers(0, min(n, int(M[j])) + 1))
        rp = np.zeros(n, np.int32)
        rd = rng.integers(decode[0], decode[1] + 1, size=n).astype(np.int32)
        cx = np.zeros(n, np.int32)
        for r in range(n):
            if r < n_run:
                if rng.random() < 0.6:   # decoding
                    cx[r] = rng.integers(1, prompt[1] + 4)
                else:                     # partially prefilled
                    cx[r] = rng.integers(1, prompt[1] + 1)
                    rp[r] = rng.integers(1, prompt[1] + 1)
            else:
                rp[r] = rng.integers(prompt[0], prompt[1] + 1)
        rps.append(rp), rds.append(rd), cxs.append(cx)
        offsets[j + 1] = offsets[j] + n
    gaps = rng.exponential(mean_gap_ms, size=n_q)
    t_ms = np.cumsum(gaps)
    q_prefill = rng.integers(prompt[0], prompt[1] + 1, size=n_q).astype(np.int32)
    q_decode = rng.integers(decode[0], decode[1] + 1, size=n_q).astype(np.int32)
    n_cols = 2
    col = rng.integers(0, n_cols, size=I).astype(np.int32)
    if dyadic:
        acc = rng.integers(0, 64, size=(n_q, n_cols)) / 64.0
        cost = rng.integers(0, 64, size=(n_q, n_cols)) / 64.0
        w_cost = rng.integers(0, 8, size=n_scen) / 8.0
        w_lat = rng.integers(0, 8, size=n_scen) / 1024.0
    else:
        acc = rng.random((n_q, n_cols))
        cost = rng.random((n_q, n_cols))
        w_cost = rng.random(n_scen)
        w_lat = rng.random(n_scen) / 1000.0
    return Workload(
        name=f"tiny{seed}", n_scen=n_scen, n_inst=I, a=a, b=b, c=c, d=d, e=e,
        budget=B, max_seqs=M, col=col, offsets=offsets,
        rem_prefill=np.concatenate(rps) if rps else np.zeros(0, np.int32),
        rem_decode=np.concatenate(rds) if rds else np.zeros(0, np.int32),
        context=np.concatenate(cxs) if cxs else np.zeros(0, np.int32),
        clock_ms=np.zeros(I), q_prefill=q_prefill, q_decode=q_decode, q_t_ms=t_ms,
        acc=acc, cost=cost, w_cost=w_cost, w_lat_ms=w_lat,
        tau_u_ms=_draw_target_vars(seed, n_q)[0], tau_v=_draw_target_vars(seed, n_q)[1],
        queue_cap=max_res + n_q + 1, max_prompt=int(prompt[1]),
        meta=dict(kind="tiny", seed=seed),
    )


def make_tiny_sched_workload(seed: int, **kw) -> Workload:
    """A tiny random pool (as ``make_tiny_workload``) with random scheduler limits that
    its residents fit: a chunk cap (or none), a context limit a little above the
    longest resident or query, and (mostly) a KV cache of power-of-two blocks only a
    little larger than one request can need, so that preemption is frequent."""
    wl = make_tiny_workload(seed, **kw)
    rng = np.random.default_rng([int(seed), 7])
    I = wl.n_inst
    sched = np.zeros((I, 4), np.int32)
    for j in range(I):
        rp, rd, cx = wl.instance_requests(j)
        longest = int((rp + cx).max()) if len(rp) else 0
        X = max(longest + 1, wl.max_prompt + 1) + int(rng.integers(0, 6))
        S = int(rng.choice([1, 2, 4]))
        held = int(sum(-(-int(c) // S) for c in cx if c > 0))
        K = 0
        if rng.random() < 0.8:
            K = max(-(-X // S), held) + int(rng.integers(0, 4))
        H = 0 if rng.random() < 0.3 else int(rng.integers(1, 6))
        sched[j] = (H, K, S, X)
    wl.sched = sched
    wl.name = f"tinysched{seed}"
    return wl


def lps_params(wl: Workload, seed: int = 0) -> dict:
    """Per-instance parameters of the average-case LPS estimator (Sec. 4.2), derived
    from each instance's batch-time model and drawn from a stream of their own (rates
    per ms, times in ms):
      prefill throughput theta = B / (a + b B), a batch that is all prefill;
      mean decode batch time  t_dec = a + c M/2, half the sequence cap decoding;
      capacity mu = M / ((a + c M) * mean decode length), queries per ms completed
        by full decode batches;
      load rho ~ U(0.05, 0.98), arrival rate alpha = rho * mu;
      parallelism k ~ U{1..64} (the paper observes about 25 on its engine);
      squared coefficients of variation ca2 ~ U(0.5, 2), cs2 ~ U(0.5, 3)."""
    rng = np.random.default_rng([seed, 0x1F5])
    I = wl.n_inst
    a, b, c = (np.asarray(x, np.float64) for x in (wl.a, wl.b, wl.c))
    B = np.asarray(wl.budget, np.float64)
    M = np.asarray(wl.max_seqs, np.float64)
    dbar = float(wl.meta.get("decode_mean", 256))
    theta = B / (a + b * B)
    t_dec = a + c * (M / 2.0)
    mu = M / ((a + c * M) * dbar)
    rho = rng.uniform(0.05, 0.98, I)
    return dict(alpha=rho * mu, mu=mu, k=rng.integers(1, 65, I).astype(np.int32),
                ca2=rng.uniform(0.5, 2.0, I), cs2=rng.uniform(0.5, 3.0, I), theta=theta,
                t_dec=t_dec)
