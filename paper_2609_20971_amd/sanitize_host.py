"""Host AddressSanitizer + UndefinedBehaviorSanitizer build of the C ABI's host
code (argument validation, stride and batch resolution, size helpers, the
debug switch), and a run of the ABI tests against it.

The instrumentation covers the host side of api.hip only (every sanitizer flag
goes through -Xarch_host); the kernels are linked from the normal build.  The
ABI tests launch nothing, so this runs without a GPU.

Usage: python -m paper_2609_20971_amd.sanitize_host
"""

from __future__ import annotations

import glob
import os
import subprocess
import sys

from . import build as _build

SAN_DIR = os.path.join(_build.BUILD_DIR, "asan")
SAN_LIB = os.path.join(SAN_DIR, "librbs_host_asan.so")
_HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]


def asan_runtime() -> str:
    found = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not found:
        raise RuntimeError("the ASan runtime of the ROCm compiler was not found")
    return found[-1]


def build_sanitized() -> str:
    objs = [os.path.join(_build.BUILD_DIR, s.replace(".hip", ".o")) for s in _build.SOURCES if s != "api.hip"]
    if not all(os.path.exists(o) for o in objs):
        _build.build()
    os.makedirs(SAN_DIR, exist_ok=True)
    api_o = os.path.join(SAN_DIR, "api.o")
    flags = [f for f in _build.FLAGS if f != "-O3"] + ["-O1", "-g"] + _HOST_SAN
    _build._run([_build.HIPCC, *flags, "-c", os.path.join(_build.CSRC, "api.hip"), "-o", api_o])
    _build._run([_build.HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *_HOST_SAN, "-Xarch_host",
                 "-shared-libasan", api_o, *objs, "-o", SAN_LIB])
    return SAN_LIB


def run_abi_tests() -> int:
    env = dict(os.environ)
    env.update(LD_PRELOAD=asan_runtime(), ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", RBS_LIB_PATH=SAN_LIB)
    tests = os.path.join(_build.ROOT, "tests", "test_abi.py")
    return subprocess.run([sys.executable, "-m", "pytest", tests, "-x", "-q", "-p", "no:cacheprovider"],
                          cwd=_build.ROOT, env=env).returncode


if __name__ == "__main__":
    print(build_sanitized())
    sys.exit(run_abi_tests())
