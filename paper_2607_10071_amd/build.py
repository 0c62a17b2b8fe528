"""Build the gfx950 HIP library in-tree.

    python -m paper_2607_10071_amd.build

Produces ``paper_2607_10071_amd/libflashbev.so`` (the fused Sampling-VT
forward and backward behind the C ABI of ``include/flashbev.h``, and FlashSCA
behind ``include/flashsca.h``) and
``libflashbev_membench.so`` (the memory-ceiling micro-benchmarks of
``include/flashbev_membench.h`` that bench.py uses).
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
INCLUDE = os.path.join(ROOT, "include")
SRC = os.path.join(HERE, "csrc", "flashbev.hip")
SCA_SRC = os.path.join(HERE, "csrc", "flashsca.hip")
LIB = os.path.join(HERE, "libflashbev.so")
# memory-ceiling micro-benchmarks used by bench.py (not part of the operator)
MEMBENCH_SRC = os.path.join(HERE, "csrc", "membench.hip")
MEMBENCH_LIB = os.path.join(HERE, "libflashbev_membench.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    # float32 coordinate recipe: every product and sum rounded on its own
    "-ffp-contract=off",
    # no packed-FP32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fPIC",
    "-shared",
    "-Wall",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    cand = os.path.join(rocm, "bin", "hipcc")
    return cand if os.path.exists(cand) else "hipcc"


def _compile(srcs, lib: str, verbose: bool) -> str:
    tmp = lib + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, f"-I{INCLUDE}", *srcs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"hipcc failed with status {r.returncode}")
    os.replace(tmp, lib)
    return lib


def build(verbose: bool = False) -> str:
    """Compile the operator library and the micro-benchmark library."""
    _compile([MEMBENCH_SRC], MEMBENCH_LIB, verbose)
    return _compile([SRC, SCA_SRC], LIB, verbose)


if __name__ == "__main__":
    build(verbose=True)
