"""The synthetic workloads, with every constant pinned.

Each entry fixes the instance pool (model types and their batch-time
coefficients, token budget B, sequence cap M), the initial resident queue depth R,
the prompt and decode length distributions, the query trace, the accuracy / cost
prediction layout, and the routing weights.  Batch-time coefficients are in ms and
follow the token-batch processing-time model of Sec. 4.1 (Eq. for the batch
processing time): T = a + b*prefill_tokens + c*decode_seqs + d*decode_context
+ e*prefill_attention.  The paper's own form has b = c = beta_1, d = beta_2,
e = beta_3.

Workload sizes span the prompt (about 10..1e4 tokens) and response (about
1e2..1e3 tokens) ranges the paper reports in its appendix on token length
distributions; the paper's datasets are not used.
"""

from __future__ import annotations

import copy

# (a, b, c) of the "1x" model type; the pool configs scale it by s in {1, 2, 4, 8}.
_BASE_ABC = (5.0, 0.02, 0.3)


def _scaled_types(d: float = 0.0):
    out = []
    for s in (1, 2, 4, 8):
        out.append(dict(a=_BASE_ABC[0] * s, b=_BASE_ABC[1] * s, c=_BASE_ABC[2] * s,
                        d=d, e=0.0, price=float(s)))
    return out


def _grid_weights():
    """8 x 8 log grid of (lambda, delta) in [0.01, 10]; scenario s = 8*k_lambda + k_delta."""
    vals = [10.0 ** (-2.0 + 3.0 * k / 7.0) for k in range(8)]
    return [(vals[kl], vals[kd]) for kl in range(8) for kd in range(8)]


CONFIGS = {
    "c1": dict(
        title="tiny routing trace",
        n_inst=4, n_scen=1,
        types=[dict(a=5.0, b=0.02, c=0.3, d=0.0, e=0.0, price=1.0),
               dict(a=12.0, b=0.06, c=0.8, d=0.0, e=0.0, price=5.0)],
        type_of_inst=[0, 0, 1, 1],
        budget=2048, max_seqs=64, resident=16,
        prompt=("uniform", 64, 2048), decode_mean=256,
        n_q=1000, rate_per_s=20.0,
        acc="per_type", cost="tokens_x_price",
        weights=[(0.5, 1.0)],
        queue_cap=4096, max_prompt=2048, seed=0,
    ),
    "c2": dict(
        title="medium pool, sequential routing",
        n_inst=32, n_scen=1,
        types=_scaled_types(),
        type_of_inst=[j // 8 for j in range(32)],
        budget=4096, max_seqs=256, resident=256,
        prompt=("lognormal", 6.5, 1.0, 16, 32768), decode_mean=384,
        n_q=100_000, rate_per_s=50.0,
        acc="per_type", cost="tokens_x_price",
        weights=[(0.5, 1.0)],
        queue_cap=8192, max_prompt=32768, seed=0,
    ),
    "c3": dict(
        title="batched what-if estimation",
        n_inst=1024, n_scen=1,
        types=_scaled_types(),
        type_of_inst=[j // 256 for j in range(1024)],
        budget=4096, max_seqs=256, resident=512,
        prompt=("lognormal", 6.5, 1.0, 16, 32768), decode_mean=384,
        n_q=4096, rate_per_s=None,
        acc="per_instance", cost="uniform",
        weights=[(0.5, 0.01)],
        queue_cap=1024, max_prompt=32768, seed=0,
    ),
    "c4": dict(
        title="long-context chunked prefill",
        n_inst=256, n_scen=1,
        types=_scaled_types(d=1e-5),
        type_of_inst=[j // 64 for j in range(256)],
        budget=8192, max_seqs=512, resident=1024,
        prompt=("lognormal", 8.0, 1.5, 32, 131072), decode_mean=1024,
        n_q=50_000, rate_per_s=100.0,
        acc="per_type", cost="tokens_x_price",
        weights=[(0.5, 0.01)],
        queue_cap=8192, max_prompt=131072, seed=0,
    ),
    "c6": dict(
        title="medium pool, bursty MMPP-2 arrivals",
        n_inst=32, n_scen=1,
        types=_scaled_types(),
        type_of_inst=[j // 8 for j in range(32)],
        budget=4096, max_seqs=256, resident=256,
        prompt=("lognormal", 6.5, 1.0, 16, 32768), decode_mean=384,
        n_q=100_000, rate_per_s=50.0,
        # two-state Markov-modulated Poisson arrivals (appendix on correlated query
        # arrivals): rate ratio r = 6, high-state fraction 0.2, transition rates
        # L->H 0.1/s and H->L 0.4/s, long-run mean rate_per_s
        arrivals=("mmpp2", 6.0, 0.2, 0.1, 0.4),
        acc="per_type", cost="tokens_x_price",
        weights=[(0.5, 1.0)],
        queue_cap=8192, max_prompt=32768, seed=0,
    ),
    "c7": dict(
        title="medium pool under KV-cache, chunk and context limits",
        n_inst=32, n_scen=1,
        types=_scaled_types(),
        type_of_inst=[j // 8 for j in range(32)],
        budget=4096, max_seqs=256, resident=256,
        # prompts clipped so that every resident (prompt + up to 255 decoded tokens)
        # is below the context limit
        prompt=("lognormal", 6.5, 1.0, 16, 7936), decode_mean=384,
        n_q=100_000, rate_per_s=50.0,
        # scheduler limits of a paged-KV engine (Sec. 2; appendix on the system):
        # 512-token prefill chunks per request, 16-token KV blocks, 8192-token context
        # limit, 18432 blocks (294,912 tokens) per instance: the residents hold
        # 9.7k-11.8k blocks at the start, so admissions and preemptions are bound by
        # the KV cache until the initial backlog drains
        sched=dict(chunk_cap=512, kv_blocks=18432, block_size=16, max_ctx=8192),
        acc="per_type", cost="tokens_x_price",
        weights=[(0.5, 1.0)],
        queue_cap=8192, max_prompt=7936, seed=0,
    ),
    "c5": dict(
        title="utility-weight sweep",
        n_inst=64, n_scen=64,
        types=_scaled_types(),
        type_of_inst=[j // 16 for j in range(64)],
        budget=4096, max_seqs=256, resident=256,
        prompt=("lognormal", 6.5, 1.0, 16, 32768), decode_mean=384,
        n_q=100_000, rate_per_s=100.0,
        acc="per_type", cost="tokens_x_price",
        weights=_grid_weights(),
        queue_cap=8192, max_prompt=32768, seed=0,
    ),
}


def config_names():
    return list(CONFIGS)


def get_config(name: str, **overrides) -> dict:
    """Return a deep copy of a config, with top-level fields overridden."""
    cfg = copy.deepcopy(CONFIGS[name])
    cfg["name"] = name
    for k, v in overrides.items():
        if k not in cfg:
            raise KeyError(f"unknown config field {k!r}")
        cfg[k] = v
    return cfg
