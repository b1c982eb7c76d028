"""MI355X (gfx950) SFS TTFT estimator and latency-aware router.

The work runs in the HIP kernels of ``liblar.so`` behind the C ABI declared in
include/lar.h; ``paper_2607_18253_amd.lar`` is its Python binding.
"""

from .lar import (EXPORTED, FIRST_TOKEN_DECODE_BATCH, FIRST_TOKEN_PREFILL_BATCH, LarContext,
                  LarError, SnapshotBoard, context_for, load_library)

__all__ = ["EXPORTED", "FIRST_TOKEN_DECODE_BATCH", "FIRST_TOKEN_PREFILL_BATCH", "LarContext",
           "LarError", "SnapshotBoard", "context_for", "load_library"]
