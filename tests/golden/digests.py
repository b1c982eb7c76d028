"""Digests of stored expected values: SHA-256 (first 32 hex digits) of arrays'
little-endian bytes, float64 values by their bit patterns.  Shared by the script
that writes the full-size expected values from the oracle and by the GPU tests that
compare the HIP path with them; no arithmetic of the method is here."""

from __future__ import annotations

import hashlib

import numpy as np


def digest(*arrays) -> str:
    h = hashlib.sha256()
    for a in arrays:
        a = np.ascontiguousarray(a)
        h.update(a.astype(a.dtype.newbyteorder("<"), copy=False).tobytes())
    return h.hexdigest()[:32]


def state_digest(offsets, rp, rd, cx, clock, iterations) -> str:
    """One instance pool's state as lar_read_state gives it: CSR offsets, the resident
    requests (remaining prefill, remaining decode, context), clocks, batches replayed."""
    return digest(np.asarray(offsets, np.int32), np.asarray(rp, np.int32),
                  np.asarray(rd, np.int32), np.asarray(cx, np.int32),
                  np.asarray(clock, np.float64), np.asarray(iterations, np.int64))
