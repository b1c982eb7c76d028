"""Build the HIP library ``liblar.so`` in-tree for gfx950 with hipcc.

Every floating-point operation in the kernels is a separate binary64
round-to-nearest-even operation: -ffp-contract=off (no fused multiply-add), no
fast-math.  Packed FP32 instructions are disabled for all device code.
"""

from __future__ import annotations

import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "liblar.so")
SOURCES = [os.path.join(CSRC, "sfs_kernels.hip"), os.path.join(CSRC, "sfs_limits.hip"),
           os.path.join(CSRC, "sfs_lps.hip"),
           os.path.join(CSRC, "lar_api.cpp"), os.path.join(CSRC, "lar_noalloc.hip"),
           os.path.join(CSRC, "lar_board.cpp")]
HEADERS = [os.path.join(CSRC, "sfs_device.h"), os.path.join(CSRC, "sfs_launch.h"),
           os.path.join(CSRC, "sfs_limits.h"), os.path.join(CSRC, "sfs_route.h"), os.path.join(CSRC, "sfs_walk.h"),
           os.path.join(ROOT, "include", "lar.h")]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def command(out: str = LIB, extra=()) -> list:
    return [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
            "-ffp-contract=off", "-fno-fast-math",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wall", "-Wno-unused-result", f"-I{os.path.join(ROOT, 'include')}",
            *extra, "-o", out, *SOURCES]


def stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(s) > t for s in SOURCES + HEADERS)


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = command(tmp)
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
