"""The trace's own count of simulated batches (lar_trace_work + the replay's
iterations) against the oracle's count of the same trace, so that the throughput
accounting of every config rests on a count checked here."""

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from gpu_util import gpu_trace  # noqa: E402
from oracle import oracle as O  # noqa: E402
from workloads import make_tiny_workload, make_workload  # noqa: E402


@pytest.mark.parametrize("name,n_q", [("c1", 1000), ("c2", 3000), ("tiny", 40), ("tiny_long", 30)])
def test_trace_work_matches_oracle(name, n_q):
    if name == "tiny":
        wl = make_tiny_workload(7, n_inst=5, max_res=6, n_q=n_q, n_scen=2)
    elif name == "tiny_long":   # more than 64 tail batches: the HBM-state kernel
        wl = make_tiny_workload(101, n_inst=6, max_res=8, n_q=n_q, prompt=(1, 300),
                                budget=(1, 6), max_seqs=(1, 3), n_scen=2)
    else:
        wl = make_workload(name, n_q=n_q)
    choice, chosen, util, ctx = gpu_trace(wl, queue_cap=10 ** 4)
    work = ctx.trace_work()
    for z in range(wl.n_scen):
        ref = O.trace(wl, scenario=z, full_rows=True, queue_cap=10 ** 4)
        assert int(work[z]) == int(ref.iters_all.astype(np.int64).sum()), z
        st = ctx.read_state(z)
        assert int(st["iterations"].sum()) == int(ref.iterations.sum())
    ctx.close()
