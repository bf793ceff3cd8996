"""Build libsfda.so (HIP, gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libsfda.so")
POISON_LIB = os.path.join(HERE, "libsfda_poison.so")
SOURCES = ["sfda_api.hip", "sfda_chunk.hip", "sfda_chunk_grad.hip", "sfda_chunk_bf16.hip", "sfda_segments.hip",
           "sfda_step.hip"]
ARCH = "gfx950"


# host code checked by AddressSanitizer and UndefinedBehaviorSanitizer (device code is
# compiled as usual); the sanitizer runtime must be preloaded into the loading process
SANITIZE_FLAGS = ["-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-omit-frame-pointer",
                  "-Xarch_host", "-fno-sanitize-recover=undefined"]


def build(verbose: bool = True, sanitize: bool = False, out: str = LIB, poison: bool = False) -> str:
    """Compile every HIP source for gfx950 into one shared library (always recompiles).
    sanitize adds ASan/UBSan instrumentation of the host code; poison builds the LDS-poison
    debug variant (SFDA_LDS_POISON: the kernels fill their LDS operand areas with NaN
    before each chunk or step rewrites them, so a stale read shows up as NaN); out is the
    library path."""
    cmd = [
        "hipcc", f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
        "-Wall", "-Wno-unused-variable",
        # packed fp32 instructions are kept out of the generated code
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-I", os.path.join(ROOT, "include"),
        "-o", out + ".tmp",
    ] + (SANITIZE_FLAGS if sanitize else []) + (["-DSFDA_LDS_POISON"] if poison else []) + \
        [os.path.join(CSRC, s) for s in SOURCES]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    msgs = "\n".join(l for l in (res.stdout + res.stderr).splitlines()
                     if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + msgs)
    if verbose and msgs.strip():
        print(msgs)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
