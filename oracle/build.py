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


SAN_LIB = os.path.join(os.path.dirname(HERE), "_build", "san", "liblrc_oracle.so")
CLANG = "/opt/rocm/llvm/bin/clang"


def build(verbose: bool = False, sanitize: bool = False) -> str:
    """gcc build of the oracle; with sanitize=True an AddressSanitizer +
    UndefinedBehaviorSanitizer build by clang (the runtime the sanitized HIP
    library uses too), without OpenMP, to _build/san/liblrc_oracle.so (load it
    with LRC_ORACLE_LIBRARY and the clang ASan runtime preloaded)."""
    lib = SAN_LIB if sanitize else LIB
    os.makedirs(os.path.dirname(lib), exist_ok=True)
    tmp = lib + ".tmp"
    if sanitize:
        cmd = [CLANG, "-std=c99", "-O1", "-g", "-fno-fast-math", "-ffp-contract=off", "-fno-math-errno",
               "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
               "-shared-libasan", "-fPIC", "-shared", "-Wall", "-Wextra", "-Wno-unused-parameter", SRC, "-o", tmp,
               "-lm"]
    else:
        cmd = ["gcc", "-std=c99", "-O3", "-fno-fast-math", "-ffp-contract=off",
               "-fno-math-errno", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
               "-Wno-unused-parameter", SRC, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose=True))
