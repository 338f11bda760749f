"""Compile the FP64 oracle (test infrastructure) into oracle/liboracle_exact.so."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "exact_attn.c")
LIB = os.path.join(HERE, "liboracle_exact.so")


def build(verbose: bool = False) -> str:
    # Portable x86-64 code (no -march=native): the library is built in one
    # container and may run on another machine's host CPU.
    cmd = ["gcc", "-O3", "-mavx2", "-mfma", "-fopenmp", "-fPIC", "-shared",
           "-std=c11", "-Wall", "-Wextra", "-o", LIB + ".tmp", SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
