"""Build the oracle's plain-C helper (test infrastructure only)."""

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "vq_ref.c")
LIB = os.path.join(HERE, "_vq_ref.so")


def build(verbose: bool = False) -> str:
    cmd = ["gcc", "-O3", "-mavx2", "-fopenmp", "-ffp-contract=off", "-shared", "-fPIC",
           "-o", LIB + ".tmp", SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


def ensure_built() -> str:
    if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        build()
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
