#!/usr/bin/env python
"""Benchmark of the SFS TTFT estimator + latency-aware router on one MI355X.

Default: the headline workload c5 (utility-weight sweep: 64 routing scenarios x 100k
queries x 64 instances, 409.6 M TTFT estimates per step), with sub-records for c1
(tiny trace), c2 (medium pool), c3 (batched what-if) and c4 (long-context pool) in
the same JSON line.  ``--workload cX`` runs one workload alone as the headline.

A step is one pass of the whole hot path over one synthetic workload, all inputs
resident in HBM before the timed region:
  sequential workloads (c1, c2, c4, c5; c6, c7): re-install the instance snapshot
  (device to device), replay the instances to the first arrival, route every query
  of the trace in order -- SFS estimate at every instance, utility + argmax, commit +
  replay to the next arrival -- in one persistent kernel, then the per-scenario
  summary (mean accuracy / cost / utility, p50 and p99 TTFT);
  c3: one estimate call for 4096 queries x 1024 instances, then the row argmax.
The device error word is checked after every timed step of a sequential workload
(a step starts by re-installing the snapshot, which clears it) and once after the
what-if steps (which never clear it); any error fails the run.

Per workload: ``value`` = TTFT estimates per second (scenarios x queries x instances
per step / step time), routed queries per second, the dominant kernel's time from
HIP events on the context's stream, and two roofline fractions of that kernel from
the algorithmic work per query step (bytes that must move; VALU wave64 instructions
of the shared-trajectory method), against 8 TB/s of HBM and 614.4 G wave64 VALU
instructions/s (256 CUs x 4 SIMDs x 2.4 GHz / 4 cycles per wave64 instruction).
Counter-measured HBM bytes and VALU instructions of the same kernel, when recorded
under profiles/ for the current kernel sources, are reported beside them.  The CPU
baseline is the plain oracle on a bounded sample of the same workload, on one core
and on all the host's cores.  Parity: the last timed step against the oracle's
sample, and, where full-size expected values exist (tests/golden), against them.
"""

from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
GOLDEN = os.path.join(ROOT, "tests", "golden")

METRIC = "TTFT estimates/sec (query x instance) and routed queries/sec on 1 MI355X"
HBM_PEAK_GBS = 8000.0
VALU_PEAK_GINSTR = 256 * 4 * 2.4 / 4        # G wave64 VALU instructions per second
SUITE = ("c1", "c2", "c3", "c3_lps", "c4")  # sub-records of the default run
SUB_STEPS = {"c1": 20, "c2": 5, "c3": 20, "c3_lps": 20, "c4": 5, "c5": 5, "c6": 5, "c7": 3}

# Algorithmic work per query step, per scenario (the shared-trajectory method):
#  bytes: every instance's running slots (M requests x 12 B: remaining prefill,
#    remaining decode, context) plus its 8-byte TTFT estimate;
#  VALU: every instance replays about one batch (M slot updates) and the chosen
#    instance re-walks its backlog to the admission point (l_a batches of M slot
#    updates); a 64-slot pass costs about 40 wave64 instructions.
# l_a = batches before a new query's admission (back-of-envelope per workload).
ADMISSION_BATCHES = {"c1": 4, "c2": 37, "c4": 1000, "c5": 37, "c6": 37, "c7": 37}
WAVE_INSTR_PER_64_SLOTS = 40


def _parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default=None,
                    choices=["c1", "c2", "c3", "c3_lps", "c4", "c5", "c6", "c7"],
                    help="one workload alone (default: c5 with sub-records c1-c4); c3_lps "
                         "is c3's what-if with the average-case LPS estimator (Sec. 4.2)")
    ap.add_argument("--n-q", type=int, default=None, help="shorten the trace (testing only)")
    ap.add_argument("--objective", default="lagrangian", choices=["lagrangian", "constrained"],
                    help="route by the Lagrangian objective or by Eq. 3 with the paper's "
                         "per-query TTFT targets (sequential workloads)")
    ap.add_argument("--realized", action="store_true",
                    help="also track each query's realised TTFT in the replay (always on "
                         "under --objective constrained, whose OnTimeUtility counts it)")
    ap.add_argument("--cpu-seconds", type=float, default=6.0,
                    help="time budget of each CPU-oracle sample (one core; all cores)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-suite", action="store_true", help="headline workload only")
    ap.add_argument("--copy-probe", action="store_true",
                    help="run one plain 256 MiB device copy first (counter calibration)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="turn two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of "
                         "'bench.py --workload cX --copy-probe --steps 1 --warmup 0 "
                         "--no-cpu-baseline --no-suite' into the traffic record")
    ap.add_argument("--summarize-valu", metavar="COUNTER_CSV",
                    help="turn a rocprofv3 --pmc SQ_WAVES SQ_INSTS_VALU SQ_INSTS_SALU run "
                         "of the same command into the VALU record")
    return ap.parse_args()


# ------------------------------------------------------------------ counter records
COPY_PROBE_BYTES = 256 << 20
_CSRC = "paper_2607_18253_amd/csrc/"
KERNEL_SOURCES = tuple(_CSRC + f for f in ("sfs_kernels.hip", "sfs_device.h", "sfs_route.h",
                                           "sfs_launch.h", "sfs_walk.h"))
LPS_KERNEL_SOURCES = tuple(_CSRC + f for f in ("sfs_lps.hip", "sfs_kernels.hip", "sfs_route.h"))
LIMIT_KERNEL_SOURCES = tuple(_CSRC + f for f in ("sfs_limits.hip", "sfs_limits.h", "sfs_device.h",
                                                 "sfs_route.h", "sfs_launch.h"))


def kernel_source_hash(workload=None):
    """Hash of the sources of the workload's kernels (a counter record is reported
    only while they are unchanged)."""
    h = hashlib.sha256()
    srcs = {"c7": LIMIT_KERNEL_SOURCES, "c3_lps": LPS_KERNEL_SOURCES}.get(workload, KERNEL_SOURCES)
    for f in srcs:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def dominant_kernels(workload):
    """Kernel-name fragments of the timed region's dominant kernel(s)."""
    if workload == "c3":
        return ("k_traj", "k_est", "k_route")
    if workload == "c3_lps":
        return ("k_lps_wait", "k_lps_est", "k_route")
    return ("k_ltrace",) if workload == "c7" else ("k_trace_cl",)


def _record_path(kind, workload):
    return os.path.join(ROOT, "profiles", f"{kind}_{workload}.json")


def _rows(path, counter):
    with open(path) as fh:
        for r in csv.DictReader(fh):
            if r["Counter_Name"] == counter:
                yield r


def summarize_pmc(fetch_csv, write_csv, workload):
    """HBM bytes per launch of the dominant kernels from two counter runs, each scaled
    by what the same counter reads for the plain device copy of known size."""
    out = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        copy, dom = [], {}
        for r in _rows(path, counter):
            k, v = r["Kernel_Name"], float(r["Counter_Value"])
            if "copy" in k.lower() or "elementwise" in k.lower():
                copy.append(v)
            elif any(d in k for d in dominant_kernels(workload)):
                dom[r["Dispatch_Id"]] = dom.get(r["Dispatch_Id"], 0.0) + v
        if not copy or not dom:
            raise SystemExit(f"{path}: no copy-probe or {dominant_kernels(workload)} dispatch")
        factor = max(copy) * 1024.0 / COPY_PROBE_BYTES   # KiB counted per true byte
        kib = sum(dom.values()) / (len(dom) / len(dominant_kernels(workload)))
        out[counter] = {"kib_per_step": kib, "copy_probe_kib": max(copy), "scale": factor,
                        "bytes_per_step": kib * 1024.0 / factor}
    rec = {"workload": workload, "kernels": list(dominant_kernels(workload)),
           "source_hash": kernel_source_hash(workload), "fetch": out["FETCH_SIZE"],
           "write": out["WRITE_SIZE"],
           "bytes_per_step": out["FETCH_SIZE"]["bytes_per_step"]
           + out["WRITE_SIZE"]["bytes_per_step"]}
    with open(_record_path("traffic", workload), "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec))


def summarize_valu(path, workload):
    """VALU / SALU wave64 instructions and duration per step of the dominant kernels
    from one counter run; issue utilisation = VALU instructions / (duration x peak)."""
    vals, span = {}, {}
    for counter in ("SQ_INSTS_VALU", "SQ_INSTS_SALU", "SQ_WAVES"):
        for r in _rows(path, counter):
            if not any(d in r["Kernel_Name"] for d in dominant_kernels(workload)):
                continue
            vals[counter] = vals.get(counter, 0.0) + float(r["Counter_Value"])
            span[r["Dispatch_Id"]] = (int(r["Start_Timestamp"]), int(r["End_Timestamp"]))
    if not span:
        raise SystemExit(f"{path}: no {dominant_kernels(workload)} dispatch")
    steps = len(span) / len(dominant_kernels(workload))
    ns = sum(e - s for s, e in span.values()) / steps
    per = {k: v / steps for k, v in vals.items()}
    rec = {"workload": workload, "kernels": list(dominant_kernels(workload)),
           "source_hash": kernel_source_hash(workload), "valu_instr_per_step": per["SQ_INSTS_VALU"],
           "salu_instr_per_step": per.get("SQ_INSTS_SALU"), "waves_per_step": per.get("SQ_WAVES"),
           "kernel_ns_in_counter_run": ns,
           "valu_issue_util": per["SQ_INSTS_VALU"] / (ns * VALU_PEAK_GINSTR)}
    with open(_record_path("valu", workload), "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec))


def load_record(kind, workload):
    """A counter record under profiles/, or None when absent or taken on other sources."""
    try:
        with open(_record_path(kind, workload)) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    return rec if rec.get("source_hash") == kernel_source_hash(workload) else None


# ------------------------------------------------------------------ algorithmic work
def algorithmic_work(name, wl):
    """(bytes, wave64 VALU instructions) the method must move / issue per step."""
    Z, I, N = wl.n_scen, wl.n_inst, wl.n_q
    M = int(np.max(wl.max_seqs))
    if name == "c3_lps":
        # parameters per instance (56 B), prompts, acc + cost, TTFT written and read back
        # by the route; the wait per instance and one division, two adds per pair
        nbytes = I * 56 + N * 4 + 2 * N * wl.n_cols * 8 + 2 * N * I * 8
        return nbytes, N * I / 64 * 20
    if name == "c3":
        R = int(np.max(np.diff(wl.offsets)))
        nbytes = I * R * 12 + 2 * N * wl.n_cols * 8 + N * I * 8   # state, acc + cost, TTFT
        slot_updates = I * 385 * M                                # background to admission
        return nbytes, slot_updates / 64 * WAVE_INSTR_PER_64_SLOTS
    per_q_bytes = I * (M * 12 + 8)
    per_q_slots = I * M + ADMISSION_BATCHES[name] * M
    return (Z * N * per_q_bytes,
            Z * N * per_q_slots / 64 * WAVE_INSTR_PER_64_SLOTS)


def rooflines(name, wl, kernel_ms):
    nbytes, winstr = algorithmic_work(name, wl)
    s = kernel_ms / 1000.0
    gbs = nbytes / s / 1e9
    gin = winstr / s / 1e9
    traffic = load_record("traffic", name)
    valu = load_record("valu", name)
    alu = {"bound": "alu", "achieved": gin, "peak": VALU_PEAK_GINSTR,
           "unit": "G wave64 VALU instr/s", "frac": gin / VALU_PEAK_GINSTR,
           "work_per_step": winstr,
           "traffic": traffic["bytes_per_step"] if traffic else None}
    hbm = {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
           "frac": gbs / HBM_PEAK_GBS, "bytes_per_step": nbytes,
           "traffic": traffic["bytes_per_step"] if traffic else None}
    counters = None
    if traffic or valu:
        counters = {"source": "builder counter runs under profiles/ (kernel source hash "
                              f"{kernel_source_hash(name)})"}
        if traffic:
            counters["hbm_bytes_per_step"] = traffic["bytes_per_step"]
            counters["hbm_gbs"] = traffic["bytes_per_step"] / s / 1e9
        if valu:
            counters["valu_instr_per_step"] = valu["valu_instr_per_step"]
            counters["valu_issue_util"] = valu["valu_issue_util"]
    return alu, hbm, counters


# ------------------------------------------------------------------ CPU oracle
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
        threads = os.cpu_count() or 1
    return model, threads


def _grow(run, budget_s, n_max, n0=4):
    """Run run(n) on growing prefixes until one takes about a third of the budget."""
    n = min(n_max, n0)
    while True:
        t0 = time.perf_counter()
        out = run(n)
        dt = time.perf_counter() - t0
        if n >= n_max or dt >= budget_s / 3:
            return n, dt, out
        n = min(n_max, int(n * max(2.0, budget_s / 3 / max(dt, 1e-3))))


def cpu_baselines(name, wl, budget_s, threads, tau=None):
    """The oracle, single-threaded and on every host thread, on bounded samples of
    the workload.  Returns (record, single-thread trace result or what-if pairs)."""
    from oracle import oracle as orc
    model, _ = host_cpu()
    if name == "c3_lps":
        from workloads.gen import lps_params
        prm = lps_params(wl)
        rows = np.random.default_rng(1).permutation(wl.n_q)
        n1, dt1, _ = _grow(lambda k: orc.lps_matrix(prm, wl.q_prefill[rows[:k]]), budget_s,
                           wl.n_q, n0=8)
        n, dt, _ = _grow(lambda k: orc.lps_matrix(prm, wl.q_prefill[rows[:k]], n_threads=threads),
                         budget_s, wl.n_q, n0=8)
        one = {"value": n1 * wl.n_inst / dt1, "cores": 1,
               "sample": f"{n1} random whole rows (x {wl.n_inst} instances) ({dt1:.2f} s)"}
        allc = {"value": n * wl.n_inst / dt, "cores": threads,
                "sample": f"{n} random whole rows (x {wl.n_inst} instances), rows split over "
                          f"{threads} threads ({dt:.2f} s)"}
        return _baseline(allc, one, model, threads), orc.lps_matrix(prm, wl.q_prefill,
                                                                    n_threads=threads)
    if name == "c3":
        rng = np.random.default_rng(1)
        qs, pairs = {}, []
        orc.set_threads(1)
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < budget_s:
            i, j = int(rng.integers(wl.n_q)), int(rng.integers(wl.n_inst))
            if j not in qs:
                qs[j] = orc.instance_queue(wl, j)
            tt, _ = qs[j].estimate(int(wl.q_prefill[i]), int(wl.q_decode[i]), 0.0)
            pairs.append((i, j, tt))
        dt1 = time.perf_counter() - t0
        one = {"value": len(pairs) / dt1, "cores": 1,
               "sample": f"{len(pairs)} random (query, instance) pairs, literal per-pair SFS "
                         f"({dt1:.1f} s)"}
        orc.set_threads(threads)
        rows = rng.choice(wl.n_q, size=wl.n_q, replace=False)
        n, dt, _ = _grow(lambda k: orc.estimate_matrix_all(wl, queries=rows[:k]), budget_s,
                         wl.n_q, n0=1)
        orc.set_threads(1)
        allc = {"value": n * wl.n_inst / dt, "cores": threads,
                "sample": f"{n} random whole rows (x {wl.n_inst} instances), one thread per "
                          f"(query, instance) pair ({dt:.1f} s)"}
        return _baseline(allc, one, model, threads), pairs
    orc.set_threads(1)
    n1, dt1, ref = _grow(lambda k: orc.trace(wl, scenario=0, n_q=k, tau=tau), budget_s, wl.n_q)
    one = {"value": n1 * wl.n_inst / dt1, "cores": 1,
           "sample": f"scenario 0, first {n1} of {wl.n_q} queries ({n1 * wl.n_inst} "
                     f"estimates + the replay; {dt1:.2f} s)",
           "routed_queries_per_s": n1 / dt1}
    if wl.n_scen > 1:   # independent scenarios, one per thread
        zs = list(range(min(threads, wl.n_scen)))
        n, dt, _ = _grow(lambda k: orc.trace_scenarios(wl, zs, len(zs), n_q=k, tau=tau),
                         budget_s, wl.n_q)
        est = len(zs) * n * wl.n_inst
        how = f"scenarios 0..{len(zs) - 1} on one thread each"
    else:               # the instances of each query in parallel
        orc.set_threads(threads)
        n, dt, _ = _grow(lambda k: orc.trace(wl, scenario=0, n_q=k, tau=tau), budget_s, wl.n_q)
        orc.set_threads(1)
        est = n * wl.n_inst
        how = f"scenario 0, the estimates and replays of the {wl.n_inst} instances in parallel"
    allc = {"value": est / dt, "cores": threads,
            "sample": f"{how}, first {n} of {wl.n_q} queries ({est} estimates + the replay; "
                      f"{dt:.2f} s)", "routed_queries_per_s": est / wl.n_inst / dt}
    return _baseline(allc, one, model, threads), (n1, ref)


def _baseline(allc, one, model, threads):
    rec = {"value": allc["value"], "unit": "TTFT estimates/s", "cores": allc["cores"],
           "kind": "oracle", "sample": allc["sample"]}
    if "routed_queries_per_s" in allc:
        rec["routed_queries_per_s"] = allc["routed_queries_per_s"]
    rec["single_core"] = {"value": one["value"], "unit": "TTFT estimates/s", "cores": 1,
                          "sample": one["sample"]}
    if "routed_queries_per_s" in one:
        rec["single_core"]["routed_queries_per_s"] = one["routed_queries_per_s"]
    rec["cpu_model"], rec["host_threads"] = model, threads
    return rec


# ------------------------------------------------------------------ parity
def _digest(a):
    sys.path.insert(0, GOLDEN)
    from digests import digest
    return digest(a)


def golden_parity(name, wl, ctx, out):
    """The timed step's results against the oracle's full-size expected values."""
    path = os.path.join(GOLDEN, f"fullsize_{name}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        g = json.load(fh)
    sys.path.insert(0, GOLDEN)
    from digests import digest, state_digest
    if name == "c3" and g["rows"] == wl.n_q and g["instances"] == wl.n_inst:
        tt = out["ttft"][0]
        B = g["block_rows"]
        bad = sum(digest(tt[b * B:(b + 1) * B]) != d for b, d in enumerate(g["ttft_blocks"]))
        return {"compared": f"every TTFT bit of the {wl.n_q} x {wl.n_inst} matrix and every "
                            "row's choice, against the oracle's stored digests",
                "mismatched_row_blocks": int(bad),
                "choices_equal": digest(out["choice"][0].astype(np.int32)) == g["choice"]}
    if name == "c5" and g["queries"] == wl.n_q:
        bad = []
        for z, want in enumerate(g["per_scenario"]):
            s = ctx.read_state(z)
            ok = (digest(out["choice"][z].astype(np.int32)) == want["choice"]
                  and digest(out["chosen"][z]) == want["ttft"]
                  and digest(out["util"][z]) == want["utility"]
                  and state_digest(s["offsets"], s["rem_prefill"], s["rem_decode"], s["context"],
                                   s["clock_ms"], s["iterations"]) == want["state"])
            if not ok:
                bad.append(z)
        return {"compared": f"all {wl.n_scen} scenarios x {wl.n_q} queries: every choice, "
                            "chosen-TTFT and utility bit and the final states, against the "
                            "oracle's stored digests", "mismatched_scenarios": bad}
    if name == "c4" and g["blocks"] and g["blocks"][-1]["end"] == wl.n_q:
        bad = [k for k, b in enumerate(g["blocks"])
               if digest(out["choice"][0, b["first"]:b["end"]].astype(np.int32)) != b["choice"]
               or digest(out["chosen"][0, b["first"]:b["end"]]) != b["ttft"]]
        s = ctx.read_state(0)
        st_ok = state_digest(s["offsets"], s["rem_prefill"], s["rem_decode"], s["context"],
                             s["clock_ms"], s["iterations"]) == g["blocks"][-1]["state"]
        return {"compared": f"all {wl.n_q} queries: every choice and chosen-TTFT bit and the "
                            "final state, against the oracle's stored digests",
                "mismatched_query_blocks": bad, "final_state_equal": bool(st_ok)}
    return None


def sample_parity(name, out, sample):
    if name == "c3_lps":   # the whole matrix, computed by the oracle
        got, want = out["ttft"][0], sample
        return {"compared": f"every TTFT bit of the {got.shape[0]} x {got.shape[1]} LPS matrix",
                "n": int(got.size),
                "ttft_bits_equal": bool(np.array_equal(got.view(np.int64), want.view(np.int64)))}
    if name == "c3":
        tt = out["ttft"][0]
        got = np.array([tt[i, j] for i, j, _ in sample])
        want = np.array([x for _, _, x in sample])
        what = "TTFT of the oracle's sampled (query, instance) pairs"
    else:
        n, ref = sample
        got, want = out["chosen"][0, :n], ref.ttft_chosen
        what = f"choice and chosen TTFT of queries 0..{n - 1}, scenario 0"
    got, want = np.ascontiguousarray(got, np.float64), np.ascontiguousarray(want, np.float64)
    rel = np.abs(got - want) / np.maximum(np.abs(want), 1e-300)
    rec = {"compared": what, "n": int(got.size),
           "ttft_bits_equal": bool(np.array_equal(got.view(np.int64), want.view(np.int64))),
           "max_rel_ttft_err": float(rel.max()) if got.size else 0.0}
    if name != "c3":
        n, ref = sample
        rec["mismatched_choices"] = int((out["choice"][0, :n] != ref.choice).sum())
    return rec


# ------------------------------------------------------------------ one workload
def run_workload(name, args, steps, warmup, want_cpu):
    import torch

    from paper_2607_18253_amd import context_for
    from workloads import make_workload

    dev = torch.device("cuda:0")
    lps = name == "c3_lps"
    wl = make_workload("c3" if lps else name, n_q=args.n_q)
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
    whatif = name in ("c3", "c3_lps")
    if lps:
        from paper_2607_18253_amd import lar as L
        from workloads.gen import lps_params
        prm = lps_params(wl)
        lps_dev = torch.as_tensor(L.lps_params_array(prm["alpha"], prm["mu"], prm["theta"],
                                                     prm["t_dec"], prm["k"], prm["ca2"],
                                                     prm["cs2"]).view(np.uint8).copy(),
                                  device=dev)
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
    kev = []   # (start, end) events around the dominant kernels of each timed step

    def step(record=False):
        if record:
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
        if whatif:
            if record:
                e0.record(stream)
            if lps:
                ctx.estimate_lps(lps_dev, qp, L.LPS_POISSON, ttft=ttft)
            else:
                ctx.estimate(qp, 0.0, ttft=ttft, want_iters=False)
            ctx.route(ttft, acc, cost, wc, wlat, choice=choice, chosen_ttft=chosen, utility=util)
            if record:
                e1.record(stream)
                kev.append((e0, e1))
            return
        ctx.reload_state()
        ctx.advance(t_first)
        if record:
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

    def check(where):
        st = ctx.status()
        if st != 0:
            raise SystemExit(f"bench.py: device error {st} in {name} ({where})")

    for _ in range(warmup):
        step()
        if not whatif:
            check("warmup step")
    check("warmup")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(steps):
        step(record=True)
        if not whatif:
            check(f"timed step {k}")   # the next step's snapshot re-install clears it
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    check("timed steps")
    ms_per_step = wall * 1000.0 / steps
    kernel_ms = sum(a.elapsed_time(b) for a, b in kev) / len(kev)

    rec = {
        "metric": METRIC, "value": Z * N * I / (ms_per_step / 1000.0), "unit": "TTFT estimates/s",
        "steps": steps, "warmup": warmup, "ms_per_step": ms_per_step,
        "config": {"workload": (f"{name}: {wl.meta['title']} with the average-case LPS "
                                "estimator (Sec. 4.2)") if lps else f"{name}: {wl.meta['title']}",
                   "scenarios": Z, "instances": I,
                   "queries": N, "resident_per_instance": wl.meta["resident"],
                   "token_budget": int(wl.budget[0]), "max_seqs": int(wl.max_seqs[0]),
                   "objective": "eq3-constrained" if constrained else
                   ("what-if" if whatif else "lagrangian")},
        "routed_queries_per_s": Z * N / (ms_per_step / 1000.0),
        "kernel": ("k_lps_wait + k_lps_est + k_route (lar_estimate_lps + lar_route)" if lps else
                   "k_traj + k_est + k_route (lar_estimate_ttft + lar_route)" if whatif else
                   ("k_ltrace (lar_route_trace under scheduler limits)" if wl.sched is not None
                    else "k_trace_cl (lar_route_trace, one launch per step)")),
        "kernel_ms": kernel_ms,
    }
    if not whatif:
        rec["config"]["realized_tracking"] = bool(track)
        rec["stats_scenario0"] = stats[0].tolist()
        est_batches = ctx.trace_work()
        replay = [int(ctx.read_state(z)["iterations"].sum()) for z in range(Z)]
        rec["simulated_batches_per_step"] = {
            "behind_the_estimates": int(est_batches.sum()), "replayed": int(sum(replay)),
            "note": "batches a literal per-pair SFS would simulate (the frontier cache "
                    "simulates far fewer); not used for the roofline"}
        if constrained:
            rec["ontime_utility_scenario0"] = float(ontime[0])
        if track:
            e0, r0 = chosen[0].cpu().numpy(), real[0].cpu().numpy()
            rec["realized_vs_estimated_scenario0"] = {
                "mean_estimated_ms": float(e0.mean()), "mean_realized_ms": float(r0.mean()),
                "frac_realized_later": float((r0 > e0).mean()),
                "max_gap_ms": float((r0 - e0).max())}
        if wl.sched is not None:
            H, K, S, X = (int(v) for v in wl.sched[0])
            rec["config"]["scheduler_limits"] = {"chunk_cap": H, "kv_blocks": K,
                                                 "block_size": S, "max_ctx": X}
    alu, hbm, counters = rooflines(name, wl, kernel_ms)
    rec["roofline"] = alu
    rec["roofline_hbm"] = hbm
    if counters:
        rec["counters"] = counters
    out = {"choice": choice.cpu().numpy(), "chosen": chosen.cpu().numpy(),
           "util": util.cpu().numpy()}
    if whatif:
        out["ttft"] = ttft.cpu().numpy()
    gp = golden_parity(name, wl, ctx, out) if not constrained and not track else None
    if want_cpu:
        _, threads = host_cpu()
        base, sample = cpu_baselines(name, wl, args.cpu_seconds, threads,
                                     tau=None if tau is None else tau.cpu().numpy())
        rec["cpu_baseline"] = base
        rec["parity_vs_oracle"] = sample_parity(name, out, sample)
    if gp:
        rec.setdefault("parity_vs_oracle", {})["full_size"] = gp
    ctx.close()
    return rec


def main():
    args = _parse()
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, args.workload or "c5")
        return
    if args.summarize_valu:
        summarize_valu(args.summarize_valu, args.workload or "c5")
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the multi-GPU sharding is a design, not a built path)", file=sys.stderr)
        sys.exit(2)
    import torch
    torch.cuda.set_device(0)
    if args.copy_probe:
        src = torch.ones(COPY_PROBE_BYTES // 4, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    head = args.workload or "c5"
    want_cpu = not args.no_cpu_baseline
    rec = run_workload(head, args, args.steps, args.warmup, want_cpu)
    line = {"metric": METRIC, "value": rec["value"], "unit": rec["unit"], "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": rec["ms_per_step"],
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64",
            "data": "synthetic", "config": dict(rec["config"], parallelism="1 GPU")}
    for k, v in rec.items():
        if k not in line and k not in ("metric", "steps", "warmup"):
            line[k] = v
    if args.workload is None and not args.no_suite:
        line["sub_records"] = {}
        for name in SUITE:
            s = min(args.steps, SUB_STEPS[name])
            line["sub_records"][name] = run_workload(name, args, s, min(args.warmup, 1),
                                                     want_cpu)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
