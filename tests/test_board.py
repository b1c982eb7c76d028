"""Snapshot board (appendix on the system: query workload snapshots and robustness
to incomplete snapshots): host-side seqlock per instance.  CPU only."""

import os
import threading

import numpy as np
import pytest

LIB = os.path.join(os.path.dirname(__file__), "..", "paper_2607_18253_amd", "liblar.so")
if not os.path.exists(LIB):
    pytest.skip("liblar.so not built (run __graft_entry__.build())", allow_module_level=True)

from paper_2607_18253_amd.lar import LAR_E_ARG, LAR_E_CAPACITY, LAR_E_STATE, LarError, \
    SnapshotBoard  # noqa: E402


def test_publish_collect_roundtrip_and_cache():
    b = SnapshotBoard(3, 8)
    with pytest.raises(LarError) as e:
        b.collect()          # no instance has published yet
    assert e.value.code == LAR_E_STATE
    b.publish(0, [0, 5], [3, 4], [7, 0], 1.5)
    b.publish(1, [], [], [], 2.0)
    with pytest.raises(LarError) as e:
        b.collect()          # instance 2 still missing
    assert e.value.code == LAR_E_STATE
    b.publish(2, [2], [1], [0], 3.25)
    s = b.collect()
    assert list(s["offsets"]) == [0, 2, 2, 3]
    assert list(s["rem_prefill"]) == [0, 5, 2]
    assert list(s["rem_decode"]) == [3, 4, 1]
    assert list(s["context"]) == [7, 0, 0]
    assert list(s["clock_ms"]) == [1.5, 2.0, 3.25]
    # instances 0 and 1 were copied into the cache by the failing collect already
    assert list(s["fresh"]) == [0, 0, 1]
    v1 = s["versions"].copy()
    s = b.collect()          # nothing new: cached copies, not fresh
    assert list(s["fresh"]) == [0, 0, 0]
    assert np.array_equal(s["versions"], v1)
    b.publish(1, [9], [9], [0], 4.0)
    s = b.collect()
    assert list(s["fresh"]) == [0, 1, 0]
    assert s["versions"][1] > v1[1]
    assert list(s["offsets"]) == [0, 2, 3, 4]
    with pytest.raises(LarError) as e:
        b.collect(cap=3)
    assert e.value.code == LAR_E_CAPACITY
    with pytest.raises(LarError) as e:
        b.publish(3, [1], [1], [0], 0.0)
    assert e.value.code == LAR_E_ARG
    with pytest.raises(LarError) as e:
        b.publish(0, np.zeros(9), np.ones(9), np.zeros(9), 0.0)   # over max_requests
    assert e.value.code == LAR_E_ARG
    b.close()


def _snapshot(v, j, big):
    n = big + (v % 97)
    i = np.arange(n, dtype=np.int64)
    rp = ((v + i) % 1000).astype(np.int32)
    rd = ((v * 3 + j + i) % 777 + 1).astype(np.int32)
    cx = ((v * 7 + i) % 555).astype(np.int32)
    return rp, rd, cx, float(v)


def test_concurrent_publishers_never_yield_torn_snapshots():
    """Two publisher threads rewrite large snapshots as fast as they can while the
    router collects; every snapshot it accepts must be one whole publication
    (all fields derived from one version number), versions never go back, and the
    router must both take fresh copies and, while an update is in progress, fall
    back to its cached one."""
    big, n_inst = 20000, 2
    b = SnapshotBoard(n_inst, big + 100)
    for j in range(n_inst):
        b.publish(j, *_snapshot(0, j, big))
    stop = threading.Event()

    def writer(j):
        v = 1
        while not stop.is_set():
            b.publish(j, *_snapshot(v, j, big))
            v += 1

    ts = [threading.Thread(target=writer, args=(j,)) for j in range(n_inst)]
    for t in ts:
        t.start()
    last = [-1.0] * n_inst
    fresh = stale = 0
    try:
        for _ in range(3000):
            s = b.collect()
            for j in range(n_inst):
                lo, hi = s["offsets"][j], s["offsets"][j + 1]
                v = int(s["clock_ms"][j])
                rp, rd, cx, _ = _snapshot(v, j, big)
                assert hi - lo == len(rp), (j, v)
                assert np.array_equal(s["rem_prefill"][lo:hi], rp)
                assert np.array_equal(s["rem_decode"][lo:hi], rd)
                assert np.array_equal(s["context"][lo:hi], cx)
                assert v >= last[j]
                last[j] = v
                fresh += int(s["fresh"][j])
                stale += 1 - int(s["fresh"][j])
    finally:
        stop.set()
        for t in ts:
            t.join()
    assert fresh > 100 and stale > 0, (fresh, stale)
    b.close()
