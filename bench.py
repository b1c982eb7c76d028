#!/usr/bin/env python
"""Benchmark of the SFS TTFT estimator + latency-aware router on one MI355X.

A step is one pass of the whole hot path over one synthetic workload, all inputs
resident in HBM before the timed region:
  re-install the instance snapshot (device-to-device), replay the instances to the
  first arrival, then route every query of the trace in order -- SFS estimate at
  every instance, Lagrangian utility + argmax, commit + replay to the next arrival
  -- and finally the per-scenario summary (mean accuracy / cost / utility, p50 and
  p99 TTFT).

Prints ONE JSON line.  ``value`` = TTFT estimates per second (scenarios x queries x
instances per step / step time); routed queries per second are reported next to it.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "TTFT estimates/sec (query x instance) and routed queries/sec on 1 MI355X"
# fp64 operations of one simulated batch: the batch time (4 multiplies, 4 adds)
# plus the fold into the clock / TTFT sum (1 add).
FLOPS_PER_BATCH = 9
PEAK = {"fp64_vector_tflops": 78.6, "hbm_gbs": 8000.0}


def _parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="c2", choices=["c1", "c2", "c4", "c5"])
    ap.add_argument("--n-q", type=int, default=None, help="shorten the trace (testing only)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="budget of the CPU-oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    return ap.parse_args()


def cpu_baseline(wl, budget_s):
    """The plain C oracle, single-threaded, on a prefix of the same trace."""
    from oracle import oracle as orc
    n = 16
    while True:
        t0 = time.perf_counter()
        orc.trace(wl, scenario=0, n_q=n, final_state=False)
        dt = time.perf_counter() - t0
        if dt >= budget_s / 4 or n >= wl.n_q:
            break
        n = min(wl.n_q, int(n * max(2.0, budget_s / 4 / max(dt, 1e-3))))
    est = n * wl.n_inst
    return {"value": est / dt, "unit": "TTFT estimates/s", "cores": 1, "kind": "oracle",
            "sample": f"scenario 0, first {n} queries of the trace ({est} estimates, "
                      f"{dt:.2f} s single-threaded)",
            "routed_queries_per_s": n / dt}


def main():
    args = _parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the sharded design is described, not built)", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2607_18253_amd import context_for
    from workloads import make_workload

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = make_workload(args.workload, n_q=args.n_q)
    Z, I, N = wl.n_scen, wl.n_inst, wl.n_q

    def T(a, dt):
        return torch.as_tensor(np.ascontiguousarray(a), dtype=dt, device=dev)

    qp, qd, qt = T(wl.q_prefill, torch.int32), T(wl.q_decode, torch.int32), T(wl.q_t_ms, torch.float64)
    acc, cost = T(wl.acc, torch.float64), T(wl.cost, torch.float64)
    wc, wlat = T(wl.w_cost, torch.float64), T(wl.w_lat_ms, torch.float64)
    choice = torch.empty((Z, N), dtype=torch.int32, device=dev)
    chosen = torch.empty((Z, N), dtype=torch.float64, device=dev)
    util = torch.empty((Z, N), dtype=torch.float64, device=dev)
    stats = torch.empty((Z, 5), dtype=torch.float64, device=dev)
    ctx = context_for(wl)
    stream = ctx.stream
    t_first, t_last = float(wl.q_t_ms[0]), float(wl.q_t_ms[-1])

    def step():
        ctx.reload_state()
        ctx.advance(t_first)
        ctx.route_trace(qp, qd, qt, t_last, acc, cost, wc, wlat, choice=choice,
                        chosen_ttft=chosen, utility=util)
        ctx.stats(choice, chosen, acc, cost, wc, out=stats)

    for _ in range(args.warmup):
        step()
    ctx.sync()
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ctx.sync()
    gpu_ms = ev0.elapsed_time(ev1)
    ms_per_step = wall * 1000.0 / args.steps
    est_per_step = Z * N * I
    value = est_per_step / (ms_per_step / 1000.0)

    line = {
        "metric": METRIC, "value": value, "unit": "TTFT estimates/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {wl.meta['title']}", "scenarios": Z,
                   "instances": I, "queries": N, "resident_per_instance": wl.meta["resident"],
                   "token_budget": int(wl.budget[0]), "max_seqs": int(wl.max_seqs[0]),
                   "parallelism": "1 GPU"},
        "routed_queries_per_s": Z * N / (ms_per_step / 1000.0),
        "gpu_event_ms_per_step": gpu_ms / args.steps,
        "stats_scenario0": stats[0].tolist(),
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(line), flush=True)
    ctx.close()


if __name__ == "__main__":
    main()
