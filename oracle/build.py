"""Build the CPU oracle shared library (test infrastructure only).

    python -m oracle.build

Compiles ``flashbev_oracle.c`` (Eq. 1 and its backward) and
``flashsca_oracle.c`` (FlashSCA) with gcc into ``liboracle.so`` next to them.
No fast-math and no floating-point contraction: the oracle's float32
coordinate recipe rounds every product and sum on its own.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "flashbev_oracle.c")
SCA_SRC = os.path.join(HERE, "flashsca_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

CFLAGS = ["-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
          "-fPIC", "-shared", "-Wall", "-Wextra"]


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = ["gcc", *CFLAGS, SRC, SCA_SRC, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
