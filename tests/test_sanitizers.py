"""The host code under AddressSanitizer and UndefinedBehaviorSanitizer (no
GPU needed): the C ABI layer's argument checks and planning (lrc_api.cpp and
the host side of the kernel sources, built with -fsanitize behind
-Xarch_host, device code unchanged) and the oracle's C loops (clang, the same
sanitizer runtime, OpenMP off) run the host, binding, parity-helper and
oracle tests in a child process with the clang ASan runtime preloaded; any
report fails the run.  The two paper-table reproductions are left out here
(100 s single-threaded under the sanitizers); they run unsanitized in
test_oracle_certificate.py."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
RUNTIME = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))


@pytest.mark.skipif(not RUNTIME, reason="clang ASan runtime not installed")
def test_host_code_clean_under_asan_and_ubsan():
    from oracle import build as oracle_build
    from paper_2607_12969_amd import build as lib_build
    lib = lib_build.build(sanitize=True)
    olib = oracle_build.build(sanitize=True)
    env = dict(os.environ)
    env.update(LD_PRELOAD=RUNTIME[-1], ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", LRC_LIBRARY=lib, LRC_ORACLE_LIBRARY=olib)
    files = ["tests/test_abi_host.py", "tests/test_binding_host.py", "tests/test_parity_host.py",
             "tests/test_oracle_rounding.py", "tests/test_oracle_linalg.py", "tests/test_oracle_quality.py",
             "tests/test_oracle_factor.py", "tests/test_oracle_certificate.py"]
    cmd = [sys.executable, "-m", "pytest", *files, "-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider",
           "-k", "not table_reproduced", "-o", "addopts="]
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in tail and "runtime error:" not in tail, tail
    # the children really loaded the sanitized builds
    probe = subprocess.run([sys.executable, "-c",
                            "from paper_2607_12969_amd import lrc; import oracle as O; O._load(); lrc.lib();"
                            "print(open('/proc/self/maps').read())"],
                           cwd=ROOT, env=env, capture_output=True, text=True, timeout=120)
    assert lib in probe.stdout and olib in probe.stdout, probe.stderr[-2000:]
