"""Host-sanitizer build of libdpool, for the CPU tests only.

Compiles every source of the library with AddressSanitizer and
UndefinedBehaviorSanitizer on its host code - the pool, the router, the cost
model and the host-side validation and planning of every device entry point
- into libdpool_asan.so beside libdpool.so.  Device code of the HIP sources
is compiled as usual, without sanitizers.  Nothing on a GPU loads this
library.

  python -m paper_2604_08075_amd.build_sanitize
  DPOOL_LIB=$PWD/paper_2604_08075_amd/libdpool_asan.so \\
  LD_PRELOAD=$(/opt/rocm/llvm/bin/clang -print-file-name=libclang_rt.asan-x86_64.so) \\
  ASAN_OPTIONS=detect_leaks=0:abort_on_error=1 UBSAN_OPTIONS=halt_on_error=1:print_stacktrace=1 \\
  python -m pytest tests -m "not gpu" -q -p no:cacheprovider
"""
from __future__ import annotations

import os
import subprocess
import sys

from .build import ARCH, CSRC, HIP_SOURCES, HOST_SOURCES, INCLUDE, PKG, hipcc

LIB = os.path.join(PKG, "libdpool_asan.so")
CLANG = "/opt/rocm/llvm/bin/clang++"
SAN = ["address", "undefined"]
HOST_SAN = [f"-fsanitize={s}" for s in SAN] + ["-fno-omit-frame-pointer", "-fno-sanitize-recover=all"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build step failed ({r.returncode}): {' '.join(cmd)}\n{msg}")
    if msg.strip():
        print(msg, file=sys.stderr)


def build() -> str:
    out_dir = os.path.join(PKG, "_build", "asan")
    os.makedirs(out_dir, exist_ok=True)
    objs = []
    for src in HOST_SOURCES:
        obj = os.path.join(out_dir, src + ".o")
        _run([CLANG, "-O1", "-g", "-std=c++17", "-fPIC", "-ffp-contract=off", *HOST_SAN, "-I", INCLUDE, "-I", CSRC,
              "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    hc = hipcc()
    # every sanitizer flag applies to the host pass only
    hip_san = [x for f in HOST_SAN for x in ("-Xarch_host", f)]
    for src in HIP_SOURCES:
        obj = os.path.join(out_dir, src + ".o")
        _run([hc, "-O1", "-g", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Xclang", "-target-feature",
              "-Xclang", "-packed-fp32-ops", *hip_san, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, src),
              "-o", obj])
        objs.append(obj)
    tmp = LIB + ".tmp"
    _run([hc, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-shared-libsan", *hip_san, *objs, "-o", tmp])
    os.replace(tmp, LIB)
    print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build()
