"""Build libsdblock.so (the HIP kernels and their C ABI) for gfx950 with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "sd_block.hip")
LIB = os.path.join(PKG, "libsdblock.so")
# the benchmark's streaming-read ceiling kernel (not part of the library's ABI)
BENCH_SRC = os.path.join(PKG, "csrc", "bench_read.hip")
BENCH_LIB = os.path.join(PKG, "libsdbench.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Wall", "-Wno-unused-function",
    # keep the compiler from emitting packed fp32 VALU ops
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _hipcc(src: str, out: str, extra=()) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tmp = out + ".tmp"
    cmd = [hipcc, *HIPCC_FLAGS, *extra, "-I", os.path.join(ROOT, "include"), "-o", tmp, src]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def build(out: str = LIB, extra=()) -> str:
    """libsdblock.so, and libsdbench.so beside it when building the default library."""
    _hipcc(SRC, out, extra)
    if out == LIB:
        _hipcc(BENCH_SRC, BENCH_LIB, extra)
    return out


if __name__ == "__main__":
    print(build(extra=sys.argv[1:]))
