"""The CPU suite again on builds instrumented by AddressSanitizer and
UndefinedBehaviorSanitizer: the library's host code (argument checks,
instance tables, the host Route-Plan planner) and the float64 reference.
Any report fails the run (CPU only; the GPU code is not instrumented)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ASAN_RT = "/opt/rocm/lib/llvm/lib/clang/22/lib/linux/libclang_rt.asan-x86_64.so"


def test_cpu_suite_under_sanitizers(tmp_path):
    from oracle import oracle
    from paper_2502_06798_amd import binding, build_lib
    if not os.path.exists(ASAN_RT):
        pytest.skip("no clang sanitizer runtime in this image")
    if not os.path.exists(binding.LIB_PATH) or not os.path.isdir(build_lib.BUILD):
        pytest.skip("libapc.so not built")
    d = str(tmp_path)
    lib = build_lib.build_sanitized(d)
    olib = oracle.build(sanitize_dir=d)
    env = dict(os.environ, LD_PRELOAD=ASAN_RT, APC_LIB=lib, APC_ORACLE_LIB=olib,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "tests", "-m", "not gpu", "-x", "-q", "-p", "no:cacheprovider",
                        "--deselect", "tests/test_sanitized_host.py::test_cpu_suite_under_sanitizers"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-3000:]
    assert r.returncode == 0, tail
    assert "passed" in r.stdout and "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, tail
