#!/usr/bin/env python
"""Benchmark of the SFS TTFT estimator + latency-aware router on one MI355X.

A step is one pass of the whole hot path over one synthetic workload, all inputs
resident in HBM before the timed region.  For the sequential-routing workloads
(default: the 32-instance medium pool, 100k queries):
  re-install the instance snapshot (device to device), replay the instances to the
  first arrival, route every query of the trace in order -- SFS estimate at every
  instance, Lagrangian utility + argmax, commit + replay to the next arrival -- in
  one persistent kernel, then the per-scenario summary (mean accuracy / cost /
  utility, p50 and p99 TTFT).
For the batched what-if workload (c3): one estimate call for 4096 queries x 1024
instances followed by the row argmax.  The c7 pool runs the sequential trace under
scheduler limits (chunk cap, context limit, KV-cache blocks with preemption).

Prints ONE JSON line.  ``value`` = TTFT estimates per second (scenarios x queries x
instances per step / step time); routed queries per second are reported next to it.
``roofline`` covers the dominant kernel, timed with HIP events on the context's
stream; its algorithmic work is counted in simulated token batches (each one is a
batch time -- 4 multiplies, 4 adds -- plus one add folding it into the clock or the
TTFT sum: 9 fp64 operations), the batch counts coming from the oracle's replay of
the same trace.
"""

from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "TTFT estimates/sec (query x instance) and routed queries/sec on 1 MI355X"
FLOPS_PER_BATCH = 9                 # 4 mul + 4 add (batch time) + 1 add (fold)
FP64_VECTOR_PEAK_TFLOPS = 78.6      # MI355X dense fp64 vector
HBM_PEAK_GBS = 8000.0


def _parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="c2",
                    choices=["c1", "c2", "c3", "c4", "c5", "c6", "c7"])
    ap.add_argument("--n-q", type=int, default=None, help="shorten the trace (testing only)")
    ap.add_argument("--objective", default="lagrangian", choices=["lagrangian", "constrained"],
                    help="route by the Lagrangian objective or by Eq. 3 with the paper's "
                         "per-query TTFT targets (sequential workloads)")
    ap.add_argument("--realized", action="store_true",
                    help="also track each query's realised TTFT in the replay (always on "
                         "under --objective constrained, whose OnTimeUtility counts it)")
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="time budget of the CPU-oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", action="store_true",
                    help="run one plain 256 MiB device copy first (counter calibration)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="turn two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of "
                         "'bench.py --copy-probe --steps 1 --warmup 0' into the traffic record")
    return ap.parse_args()


COPY_PROBE_BYTES = 256 << 20
_CSRC = "paper_2607_18253_amd/csrc/"
KERNEL_SOURCES = tuple(_CSRC + f for f in ("sfs_kernels.hip", "sfs_device.h", "sfs_route.h"))
LIMIT_KERNEL_SOURCES = tuple(_CSRC + f for f in ("sfs_limits.hip", "sfs_limits.h", "sfs_device.h",
                                                 "sfs_route.h"))


def kernel_source_hash(workload=None):
    """Hash of the sources of the workload's trace kernel (a measured traffic figure
    is reported only while they are unchanged)."""
    h = hashlib.sha256()
    for f in (LIMIT_KERNEL_SOURCES if workload == "c7" else KERNEL_SOURCES):
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_path(workload):
    return os.path.join(ROOT, "profiles", f"traffic_{workload}.json")


def summarize_pmc(fetch_csv, write_csv, workload):
    """HBM bytes per launch of the dominant kernel from two counter runs, each scaled
    by what the same counter reads for the plain device copy of known size."""
    def per_kernel(path, counter):
        vals = {}
        with open(path) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] != counter:
                    continue
                key = (r["Kernel_Name"], r.get("Dispatch_Id", r.get("Correlation_Id", "")))
                vals[key] = vals.get(key, 0.0) + float(r["Counter_Value"])
        return vals

    out = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        v = per_kernel(path, counter)
        copy = [x for (k, _), x in v.items() if "copy" in k.lower() or "elementwise" in k.lower()]
        dom = [x for (k, _), x in v.items() if dominant_kernel(workload) in k]
        if not copy or not dom:
            raise SystemExit(f"{path}: no copy-probe or {dominant_kernel(workload)} dispatch")
        factor = max(copy) * 1024.0 / COPY_PROBE_BYTES   # KiB counted per true byte
        out[counter] = {"kib_per_launch": sum(dom) / len(dom), "copy_probe_kib": max(copy),
                        "scale": factor, "bytes_per_launch": sum(dom) / len(dom) * 1024.0 / factor}
    rec = {"workload": workload, "kernel": dominant_kernel(workload), "source_hash": kernel_source_hash(workload),
           "fetch": out["FETCH_SIZE"], "write": out["WRITE_SIZE"],
           "bytes_per_launch": out["FETCH_SIZE"]["bytes_per_launch"]
           + out["WRITE_SIZE"]["bytes_per_launch"]}
    with open(traffic_path(workload), "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec))


def load_traffic(workload):
    """Measured HBM bytes per launch, or None when absent or taken on other sources."""
    try:
        with open(traffic_path(workload)) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    if rec.get("source_hash") != kernel_source_hash(workload):
        return None
    return rec["bytes_per_launch"]


def dominant_kernel(workload):
    if workload == "c3":
        return "k_traj"
    return "k_ltrace" if workload == "c7" else "k_trace_cl"


def oracle_sample(wl, budget_s, tau=None):
    """The plain C oracle, single-threaded, on a prefix of the same trace (scenario 0).

    Returns the CPU baseline record and the oracle's count of simulated batches over
    that prefix (estimate batches + replayed batches); the prefix grows from 4 queries
    until it takes about a third of the budget."""
    from oracle import oracle as orc
    n = min(wl.n_q, 4)
    while True:
        t0 = time.perf_counter()
        r = orc.trace(wl, scenario=0, n_q=n, full_rows=True, final_state=True, tau=tau)
        dt = time.perf_counter() - t0
        if n >= wl.n_q or dt >= budget_s / 3:
            break
        n = min(wl.n_q, int(n * max(2.0, budget_s / 3 / max(dt, 1e-3))))
    est = n * wl.n_inst
    batches = int(r.iters_all.astype(np.int64).sum() + r.iterations.sum())
    rec = {"value": est / dt, "unit": "TTFT estimates/s", "cores": 1, "kind": "oracle",
           "sample": f"scenario 0, first {n} of {wl.n_q} queries ({est} estimates + the "
                     f"replay; {dt:.2f} s single-threaded)",
           "routed_queries_per_s": n / dt}
    return rec, n, batches, r


def whatif_oracle_sample(wl, budget_s):
    from oracle import oracle as orc
    rng = np.random.default_rng(1)
    n, t_used, batches = 0, 0.0, 0
    qs = {}
    pairs = []
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < budget_s:
        i, j = int(rng.integers(wl.n_q)), int(rng.integers(wl.n_inst))
        if j not in qs:
            qs[j] = orc.instance_queue(wl, j)
        tt, it = qs[j].estimate(int(wl.q_prefill[i]), 1, 0.0)
        pairs.append((i, j, tt))
        batches += it
        n += 1
    dt = time.perf_counter() - t0
    return {"value": n / dt, "unit": "TTFT estimates/s", "cores": 1, "kind": "oracle",
            "sample": f"{n} random (query, instance) pairs, literal per-pair SFS "
                      f"({dt:.1f} s single-threaded)"}, batches / max(n, 1), pairs


def host_cpu():
    """The host's CPU model and the threads available to this process."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for ln in fh:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        threads = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        threads = os.cpu_count() or 0
    return model, threads


def parity_record(got, want, what):
    """Bit-level comparison of GPU results with the oracle's on the same sample."""
    got = np.ascontiguousarray(got, np.float64)
    want = np.ascontiguousarray(want, np.float64)
    rel = np.abs(got - want) / np.maximum(np.abs(want), 1e-300)
    return {"compared": what, "n": int(got.size),
            "ttft_bits_equal": bool(np.array_equal(got.view(np.int64), want.view(np.int64))),
            "max_rel_ttft_err": float(rel.max()) if got.size else 0.0}


import numpy as np  # noqa: E402


def main():
    args = _parse()
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, args.workload)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the multi-GPU sharding is a design, not a built path)", file=sys.stderr)
        sys.exit(2)
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
    whatif = args.workload == "c3"
    constrained = args.objective == "constrained" and not whatif
    t_first, t_last = float(wl.q_t_ms[0]), float(wl.q_t_ms[-1])
    tau = None
    if constrained:   # the paper's per-query TTFT targets, computed once on the GPU
        tau = ctx.ttft_targets(qp, T(wl.tau_u_ms, torch.float64), T(wl.tau_v, torch.float64))
        ontime = torch.empty(Z, dtype=torch.float64, device=dev)
    track = (constrained or args.realized) and not whatif
    real = torch.empty((Z, N), dtype=torch.float64, device=dev) if track else None
    if whatif:
        ttft = torch.empty((Z, N, I), dtype=torch.float64, device=dev)
    kev = []   # (start, end) events around the dominant kernel of each timed step
    if args.copy_probe:
        src = torch.ones(COPY_PROBE_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    def step(record=False):
        if whatif:
            if record:
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
            ctx.estimate(qp, 0.0, ttft=ttft, want_iters=False)
            if record:
                e1.record(stream)
                kev.append((e0, e1))
            ctx.route(ttft, acc, cost, wc, wlat, choice=choice, chosen_ttft=chosen, utility=util)
            return
        ctx.reload_state()
        ctx.advance(t_first)
        if record:
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
        if constrained:
            ctx.route_trace_constrained(qp, qd, qt, t_last, tau, acc, cost, wc, choice=choice,
                                        chosen_ttft=chosen, utility=util, realized=real)
        else:
            ctx.route_trace(qp, qd, qt, t_last, acc, cost, wc, wlat, choice=choice,
                            chosen_ttft=chosen, utility=util, realized=real)
        if record:
            e1.record(stream)
            kev.append((e0, e1))
        ctx.stats(choice, chosen, acc, cost, wc, out=stats)
        if constrained:
            ctx.ontime_utility(choice, real, tau, acc, cost, wc, out=ontime)

    for _ in range(args.warmup):
        step()
    ctx.sync()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(record=True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ctx.sync()
    ms_per_step = wall * 1000.0 / args.steps
    kernel_ms = sum(a.elapsed_time(b) for a, b in kev) / len(kev)
    value = Z * N * I / (ms_per_step / 1000.0)

    line = {
        "metric": METRIC, "value": value, "unit": "TTFT estimates/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {wl.meta['title']}", "scenarios": Z,
                   "instances": I, "queries": N, "resident_per_instance": wl.meta["resident"],
                   "token_budget": int(wl.budget[0]), "max_seqs": int(wl.max_seqs[0]),
                   "objective": "eq3-constrained" if constrained else
                   ("what-if" if whatif else "lagrangian"),
                   "parallelism": "1 GPU"},
        "routed_queries_per_s": Z * N / (ms_per_step / 1000.0),
    }
    if whatif:
        line["roofline_kernel"] = "k_traj + k_est (lar_estimate_ttft)"
    else:
        line["roofline_kernel"] = (
            "k_ltrace (lar_route_trace under scheduler limits, one launch per step)"
            if wl.sched is not None else "k_trace_cl (lar_route_trace, one launch per step)")
        line["stats_scenario0"] = stats[0].tolist()
        if constrained:
            line["ontime_utility_scenario0"] = float(ontime[0])
        if track:
            # the replay's first-token times against the estimates at the choice
            # (the comparison of Fig. 2), scenario 0
            e0, r0 = chosen[0].cpu().numpy(), real[0].cpu().numpy()
            line["realized_vs_estimated_scenario0"] = {
                "mean_estimated_ms": float(e0.mean()), "mean_realized_ms": float(r0.mean()),
                "frac_realized_later": float((r0 > e0).mean()),
                "max_gap_ms": float((r0 - e0).max())}
        line["config"]["realized_tracking"] = bool(track)
        if wl.sched is not None:
            H, K, S, X = (int(v) for v in wl.sched[0])
            line["config"]["scheduler_limits"] = {"chunk_cap": H, "kv_blocks": K,
                                                  "block_size": S, "max_ctx": X}
    line["kernel_ms"] = kernel_ms

    roof = None
    if not whatif:
        # simulated batches of the last step, counted by the trace itself (estimates)
        # and by the instances' replay counters; equal to the oracle's count of the
        # same trace (checked by the GPU tests)
        est_batches = ctx.trace_work()
        replay = [int(ctx.read_state(z)["iterations"].sum()) for z in range(Z)]
        batches = int(est_batches.sum()) + int(sum(replay))
        flops = FLOPS_PER_BATCH * batches
        achieved = flops / (kernel_ms / 1000.0) / 1e12
        roof = {"bound": "alu", "achieved": achieved, "peak": FP64_VECTOR_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": achieved / FP64_VECTOR_PEAK_TFLOPS,
                "traffic": None if track else load_traffic(args.workload),
                "note": f"{batches} simulated token batches per step over {Z} scenario(s) "
                        f"({int(est_batches.sum())} behind the estimates, {int(sum(replay))} "
                        "replayed) x 9 fp64 ops each; sequential trace, latency-bound"
                        + ("; the batches run after the last arrival for realised TTFTs "
                           "are not counted" if track else "")}
        line["batches_per_step"] = batches
    if not args.no_cpu_baseline:
        model, threads = host_cpu()
        if whatif:
            rec, batches_per_pair, pairs = whatif_oracle_sample(wl, args.cpu_seconds)
            rec["cpu_model"], rec["host_threads"] = model, threads
            line["cpu_baseline"] = rec
            tt = ttft[0].cpu().numpy()
            line["parity_vs_oracle"] = parity_record(
                [tt[i, j] for i, j, _ in pairs], [x for _, _, x in pairs],
                "TTFT of the oracle's sampled (query, instance) pairs, scenario 0")
            # HBM-bound output: the fp64 TTFT matrix written once, plus per-query and
            # per-instance inputs (negligible); algorithmic bytes per estimate = 8
            achieved = Z * N * I * 8 / (kernel_ms / 1000.0) / 1e9
            roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": achieved / HBM_PEAK_GBS, "traffic": load_traffic(args.workload),
                    "note": "algorithmic bytes = 8 B of TTFT output per (query, instance); "
                            f"a literal per-pair SFS would simulate {batches_per_pair:.0f} "
                            "batches per pair"}
        else:
            rec, n, obatches, ref = oracle_sample(
                wl, args.cpu_seconds, tau=None if tau is None else tau.cpu().numpy())
            rec["cpu_model"], rec["host_threads"] = model, threads
            line["cpu_baseline"] = rec
            if n == N and Z == 1:
                rec["oracle_batches"] = obatches
            # the last timed step's results against the oracle's on the same prefix
            par = parity_record(chosen[0, :n].cpu().numpy(), ref.ttft_chosen,
                                f"chosen TTFT of queries 0..{n - 1}, scenario 0")
            par["mismatched_choices"] = int((choice[0, :n].cpu().numpy() != ref.choice).sum())
            line["parity_vs_oracle"] = par
    line["roofline"] = roof
    print(json.dumps(line), flush=True)
    ctx.close()


if __name__ == "__main__":
    main()
