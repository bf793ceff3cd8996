"""The CPU test suite under AddressSanitizer and UndefinedBehaviorSanitizer.

Builds oracle.c and the host code of libsfda.so (argument validation, size arithmetic,
workspace bookkeeping, the C ABI) with ASan and UBSan into a temporary directory, then runs
`pytest -m "not gpu"` in a child process that preloads clang's sanitizer runtime and loads
those builds instead of the in-tree ones (SFDA_LIBRARY, SFDA_ORACLE_LIB).  Any sanitizer
report ends the child with an error.  Needs no GPU:

    python tests/run_sanitized.py [extra pytest arguments]
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def asan_runtime() -> str:
    found = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not found:
        raise RuntimeError("clang's ASan runtime (libclang_rt.asan-x86_64.so) was not found")
    return found[-1]


def main(argv) -> int:
    import oracle
    from paper_2607_11897_amd import build as hip_build
    with tempfile.TemporaryDirectory(prefix="sfda_san_") as tmp:
        lib = hip_build.build(verbose=False, sanitize=True, out=os.path.join(tmp, "libsfda.so"))
        olib = oracle.build(verbose=False, sanitize=True, out=os.path.join(tmp, "liboracle.so"))
        env = dict(os.environ)
        env.update({
            "SFDA_LIBRARY": lib,
            "SFDA_ORACLE_LIB": olib,
            "LD_PRELOAD": asan_runtime(),
            # the interpreter itself is not instrumented: its allocations are not leaks
            "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1:halt_on_error=1",
            "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
        })
        cmd = [sys.executable, "-m", "pytest", os.path.join(ROOT, "tests"), "-x", "-q", "-m", "not gpu",
               "-p", "no:cacheprovider"] + list(argv)
        print("sanitized builds:", lib, olib, flush=True)
        return subprocess.call(cmd, env=env, cwd=ROOT)


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
