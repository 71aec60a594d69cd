"""The host code of libdpool under AddressSanitizer and UndefinedBehaviorSanitizer.

Builds libdpool_asan.so (every source's host code instrumented; the device
code as usual) and runs the host-side tests against it in a child process:
the router's bit-exact runs, the pool allocator, the cost model, the
adaptive threshold and the host validation of every device entry point.  Any
sanitizer report aborts the child and fails this test.  CPU only.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLANG = "/opt/rocm/llvm/bin/clang"


def test_host_code_is_clean_under_asan_and_ubsan():
    if not os.path.exists(CLANG) or not os.path.exists(os.path.join(ROOT, "paper_2604_08075_amd",
                                                                    "build_sanitize.py")):
        pytest.skip("the sanitizer build needs ROCm's clang and build_sanitize.py")
    from paper_2604_08075_amd import build_sanitize
    lib = build_sanitize.build()
    rt = subprocess.run([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                        text=True).stdout.strip()
    env = dict(os.environ, DPOOL_LIB=lib, LD_PRELOAD=rt, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    tests = ["tests/test_host_lib.py", "tests/test_oracle_adapt.py", "tests/test_oracle_cost.py",
             "tests/test_oracle_pool_route.py"]
    r = subprocess.run([sys.executable, "-m", "pytest", *tests, "-m", "not gpu", "-q", "-x", "-p", "no:cacheprovider"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    tail = "\n".join((r.stdout + r.stderr).splitlines()[-30:])
    assert r.returncode == 0, tail
    assert "passed" in r.stdout and "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr
