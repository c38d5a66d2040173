"""Build the HIP library liblrc.so in-tree for gfx950 with hipcc.

Usage: python -m paper_2607_12969_amd.build   (or call build()).
Every HIP source is compiled with packed-FP32 instructions disabled (their
results are not trusted on the test machines); the host compiler warns that
it does not know that target feature, which is harmless.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "liblrc.so")
SOURCES = ["apply.hip", "tt.hip", "reduce.hip", "quant.hip", "gauge.hip", "quality.hip", "factor.hip", "ceiling.hip",
           "lrc_api.cpp"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def flags():
    return ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            # keep matrix-core accumulators in ordinary VGPRs: the default AGPR
            # form copies every loop-carried accumulator out and back each
            # iteration, which halves the FP64 matrix-core rate
            "-mllvm", "-amdgpu-mfma-vgpr-form=1",
            "-I", os.path.join(ROOT, "include"), "-I", CSRC]


# AddressSanitizer and UndefinedBehaviorSanitizer for the host code only (the
# device code is built as usual): each -fsanitize= sits behind -Xarch_host.
SAN_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
SAN_DIR = os.path.join(ROOT, "_build", "san")


def build(verbose: bool = False, jobs: int = 4, sanitize: bool = False) -> str:
    """Compile liblrc.so in-tree; with sanitize=True a host-sanitized copy
    goes to _build/san/liblrc.so instead (load it with LRC_LIBRARY and the
    clang ASan runtime preloaded)."""
    objdir = SAN_DIR if sanitize else os.path.join(ROOT, "_build")
    os.makedirs(objdir, exist_ok=True)
    procs, objs = [], []
    for src in SOURCES:
        obj = os.path.join(objdir, src + ".o")
        objs.append(obj)
        lang = ["-x", "hip"] if src.endswith(".cpp") else []
        cmd = [HIPCC] + flags() + (SAN_HOST if sanitize else []) + lang + ["-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stderr=subprocess.PIPE, stdout=subprocess.PIPE, text=True)))
        if len(procs) >= jobs:
            _wait(procs.pop(0), verbose)
    while procs:
        _wait(procs.pop(0), verbose)
    lib = os.path.join(SAN_DIR, "liblrc.so") if sanitize else LIB
    tmp = lib + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    if sanitize:
        cmd += ["-fsanitize=address,undefined", "-shared-libasan"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)
    return lib


def _wait(item, verbose):
    src, p = item
    out, err = p.communicate()
    lines = [ln for ln in (err or "").splitlines() if "packed-fp32-ops" not in ln]
    if p.returncode != 0:
        sys.stderr.write("\n".join(lines) + "\n")
        raise RuntimeError(f"hipcc failed on {src}")
    if verbose and lines:
        sys.stderr.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
