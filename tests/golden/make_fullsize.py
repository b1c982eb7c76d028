"""Write the full-size expected values of the c3, c4 and c5 workloads.

Calls only the oracle (``oracle/``) and the seeded input generators
(``workloads/``).  The results are stored as SHA-256 digests (first 32 hex digits)
of their little-endian bytes -- float64 values by their bit patterns -- so that a GPU
test can compare every value without the file holding them:

* c3 (batched what-if, Sec. 4.1): the 4096 x 1024 TTFT and batch-count matrices in
  blocks of 16 rows, and the route of every row (Lagrangian objective with the
  utility of Eq. 2): choices and the Eq. 2 utility at the choice.
* c4 (long-context trace, 256 instances): the trace from the original snapshot in
  blocks of 1000 queries -- choices, chosen TTFT and utility per block, the batches
  behind the block's estimates, and the state of every instance after the block.
  The oracle runs block by block from its own state after the previous block; the
  blocks chain exactly (advancing to one arrival and then to the next runs the
  same batches as advancing to the later one), so block k's state is the state of
  one trace over the first k blocks whose last query is the end of block k.  The
  file is rewritten after every block, so a run stopped early leaves a shorter,
  valid prefix.
* c5 (weight sweep): every scenario's whole trace -- choices, chosen TTFT, utility,
  per-scenario stats, final state and the batches behind its estimates.

Usage: python tests/golden/make_fullsize.py c3|c4|c5 [--threads N] [--c4-blocks K]
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

sys.path.insert(0, HERE)

from digests import digest, state_digest  # noqa: E402
from oracle import oracle as O  # noqa: E402
from workloads import make_workload  # noqa: E402

C3_BLOCK = 16
C4_BLOCK = 1000


def out_path(name):
    return os.path.join(HERE, f"fullsize_{name}.json")


def write(name, doc):
    tmp = out_path(name) + ".tmp"
    with open(tmp, "w") as f:
        json.dump(doc, f, indent=1)
        f.write("\n")
    os.replace(tmp, out_path(name))


def make_c3():
    wl = make_workload("c3")
    t0 = time.time()
    ttft, iters = O.estimate_matrix_all(wl, t_ms=0.0)
    el = time.time() - t0
    choice = np.zeros(wl.n_q, np.int32)
    util = np.zeros(wl.n_q)
    for i in range(wl.n_q):
        m, _ = O.route_row(ttft[i], wl.acc[i], wl.cost[i], wl.col, wl.w_cost[0],
                           wl.w_lat_ms[0])
        choice[i] = m
        pen = wl.w_cost[0] * wl.cost[i, wl.col[m]]
        util[i] = wl.acc[i, wl.col[m]] - pen
    nb = wl.n_q // C3_BLOCK
    doc = dict(
        workload="c3", rows=wl.n_q, instances=wl.n_inst, block_rows=C3_BLOCK,
        ttft_blocks=[digest(ttft[b * C3_BLOCK:(b + 1) * C3_BLOCK]) for b in range(nb)],
        iters_blocks=[digest(iters[b * C3_BLOCK:(b + 1) * C3_BLOCK]) for b in range(nb)],
        ttft_all=digest(ttft), iters_all=digest(iters), iters_total=int(iters.sum(dtype=np.int64)),
        choice=digest(choice), utility=digest(util),
        oracle_seconds=round(el, 1), oracle_threads=O.get_threads())
    write("c3", doc)


def make_c4(max_blocks):
    wl = make_workload("c4")
    N = wl.n_q
    nblk = min(max_blocks, (N + C4_BLOCK - 1) // C4_BLOCK)
    doc = dict(workload="c4", queries=N, block_queries=C4_BLOCK, blocks=[],
               oracle_threads=O.get_threads())
    cur = wl
    iters_cum = np.zeros(wl.n_inst, np.int64)
    t_start = time.time()
    for b in range(nblk):
        lo, hi = b * C4_BLOCK, min(N, (b + 1) * C4_BLOCK)
        sl = slice(lo, hi)
        part = _replace_queries(cur, wl, sl)
        t0 = time.time()
        r = O.trace(part, queue_cap=wl.queue_cap, full_rows=True)
        iters_cum += r.iterations
        doc["blocks"].append(dict(
            first=lo, end=hi, choice=digest(r.choice), ttft=digest(r.ttft_chosen),
            utility=digest(r.util_chosen), estimate_batches=int(r.iters_all.sum(dtype=np.int64)),
            state=state_digest(r.offsets, r.rem_prefill, r.rem_decode, r.context, r.clock_ms,
                               iters_cum),
            seconds=round(time.time() - t0, 1)))
        doc["oracle_seconds"] = round(time.time() - t_start, 1)
        write("c4", doc)
        print(f"c4 block {b} queries {lo}..{hi - 1} {time.time() - t0:.1f} s", flush=True)
        cur = _with_state(cur, r)


def _replace_queries(cur, wl, sl):
    import dataclasses
    return dataclasses.replace(
        cur, q_prefill=wl.q_prefill[sl], q_decode=wl.q_decode[sl],
        q_t_ms=wl.q_t_ms[sl], acc=wl.acc[sl], cost=wl.cost[sl], tau_u_ms=wl.tau_u_ms[sl],
        tau_v=wl.tau_v[sl])


def _with_state(cur, r):
    import dataclasses
    return dataclasses.replace(cur, offsets=r.offsets, rem_prefill=r.rem_prefill,
                               rem_decode=r.rem_decode, context=r.context, clock_ms=r.clock_ms)


def make_c5(n_threads):
    wl = make_workload("c5")
    O.set_threads(1)
    t0 = time.time()
    res = O.trace_scenarios(wl, list(range(wl.n_scen)), n_threads, full_rows=True)
    el = time.time() - t0
    scen = []
    for z, r in enumerate(res):
        st = O.stats(r.choice, r.ttft_chosen, wl.acc, wl.cost, wl.col, wl.w_cost[z])
        scen.append(dict(
            choice=digest(r.choice), ttft=digest(r.ttft_chosen), utility=digest(r.util_chosen),
            stats_bits=[format(int(v), "016x") for v in np.asarray(st).view(np.uint64)],
            state=state_digest(r.offsets, r.rem_prefill, r.rem_decode, r.context, r.clock_ms,
                               r.iterations),
            estimate_batches=int(r.iters_all.sum(dtype=np.int64))))
    write("c5", dict(workload="c5", scenarios=wl.n_scen, queries=wl.n_q, per_scenario=scen,
                     oracle_seconds=round(el, 1), oracle_threads=n_threads))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("which", choices=["c3", "c4", "c5"])
    ap.add_argument("--threads", type=int, default=os.cpu_count() or 1)
    ap.add_argument("--c4-blocks", type=int, default=50)
    a = ap.parse_args()
    if a.which == "c3":
        O.set_threads(a.threads)
        make_c3()
    elif a.which == "c4":
        O.set_threads(a.threads)
        make_c4(a.c4_blocks)
    else:
        make_c5(a.threads)


if __name__ == "__main__":
    main()
