"""Build the gfx950 HIP library in-tree.

    python -m paper_2607_10071_amd.build

Produces ``paper_2607_10071_amd/libflashbev.so`` (the fused Sampling-VT
forward and backward behind the C ABI of ``include/flashbev.h``, and FlashSCA
behind ``include/flashsca.h``) and
``libflashbev_membench.so`` (the memory-ceiling micro-benchmarks of
``include/flashbev_membench.h`` that bench.py uses) and
``libflashbev_phases.so`` (the same operator library with the forward's
phase clock compiled in, ``include/flashbev_phases.h``, for
``python -m paper_2607_10071_amd.phases``).  The three compile in parallel.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
INCLUDE = os.path.join(ROOT, "include")
SRC = os.path.join(HERE, "csrc", "flashbev.hip")
SCA_SRC = os.path.join(HERE, "csrc", "flashsca.hip")
LIB = os.path.join(HERE, "libflashbev.so")
# memory-ceiling micro-benchmarks used by bench.py (not part of the operator)
MEMBENCH_SRC = os.path.join(HERE, "csrc", "membench.hip")
MEMBENCH_LIB = os.path.join(HERE, "libflashbev_membench.so")
# the operator library with the forward's phase clock (measurement tool)
PHASES_LIB = os.path.join(HERE, "libflashbev_phases.so")
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


def _compile(srcs, lib: str, verbose: bool, extra=()) -> str:
    tmp = lib + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, *extra, f"-I{INCLUDE}", *srcs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"hipcc failed with status {r.returncode}")
    os.replace(tmp, lib)
    return lib


# a C++ program that drives the forward through the C ABI alone (plain HIP
# memory and streams); the GPU tests run it (test infrastructure)
C_ABI_SRC = os.path.join(ROOT, "tests", "c_abi_forward.cpp")
C_ABI_EXE = os.path.join(ROOT, "tests", "c_abi_forward")


def _build_c_abi_program(verbose: bool) -> str:
    tmp = C_ABI_EXE + ".tmp"
    cmd = [hipcc(), "-O2", "-std=c++17", "-Wall", f"-I{INCLUDE}", C_ABI_SRC, "-o", tmp,
           f"-L{HERE}", "-lflashbev", "-Wl,-rpath,$ORIGIN/../paper_2607_10071_amd"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"hipcc failed with status {r.returncode}")
    os.replace(tmp, C_ABI_EXE)
    return C_ABI_EXE


def build(verbose: bool = False) -> str:
    """Compile the operator library, the micro-benchmark library and the
    C-ABI test program."""
    with ThreadPoolExecutor(max_workers=3) as ex:
        jobs = [ex.submit(_compile, [MEMBENCH_SRC], MEMBENCH_LIB, verbose),
                ex.submit(_compile, [SRC, SCA_SRC], LIB, verbose),
                ex.submit(_compile, [SRC, SCA_SRC], PHASES_LIB, verbose,
                          ("-DFLASHBEV_PHASE_CLOCK",))]
        lib = jobs[1].result()
        for j in jobs:
            j.result()
    _build_c_abi_program(verbose)
    return lib


if __name__ == "__main__":
    build(verbose=True)
