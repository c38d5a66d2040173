"""Compile the C part of the oracle (test infrastructure) with gcc.

The oracle is plain C99 + OpenMP, built without fast-math and with
-ffp-contract=off so every result is bitwise reproducible.  Only the test
suite, the smoke check and the benchmark's CPU-baseline leg load it.
"""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "lrc_oracle.c")
LIB = os.path.join(HERE, "liblrc_oracle.so")


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-std=c99", "-O3", "-fno-fast-math", "-ffp-contract=off",
           "-fno-math-errno", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-Wno-unused-parameter", SRC, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
