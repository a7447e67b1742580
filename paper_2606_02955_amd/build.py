"""Build the HIP libraries in-tree for gfx950 (hipcc, no JIT).

libfdllm.so is the commit selector (include/fdllm.h); libfdllm_bench.so is
the read-only HBM stream used as the bandwidth reference in reports
(include/fdllm_bench.h).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "fdllm.hip")
LOOP_SRC = os.path.join(PKG, "csrc", "loop.hip")
LMHEAD_SRC = os.path.join(PKG, "csrc", "lmhead.hip")
STATIC_SRC = os.path.join(PKG, "csrc", "decode_static.hip")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libfdllm.so")
BENCH_SRC = os.path.join(PKG, "csrc", "stream_read.hip")
BENCH_LIB = os.path.join(PKG, "libfdllm_bench.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    # packed-FP32 VALU forms stay disabled on this target
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # logits are finite by contract: max/min need no NaN quieting.  (Not
    # -mno-amdgpu-ieee: the device library keeps IEEE mode, and its work-item
    # and workgroup id functions would then stay out-of-line calls.)
    "-Xarch_device", "-fno-honor-nans",
    "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libfdllm.so)")


def _compile(srcs, lib: str, verbose: bool, extra=()) -> str:
    tmp = lib + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, *extra, "-I", INCLUDE, *srcs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed with status {res.returncode} on {srcs}")
    os.replace(tmp, lib)
    return lib


def build(verbose: bool = False, extra=()) -> str:
    """Compile libfdllm.so and libfdllm_bench.so (always recompiles both)."""
    _compile([BENCH_SRC], BENCH_LIB, verbose)
    return _compile([SRC, LMHEAD_SRC, LOOP_SRC, STATIC_SRC], LIB, verbose, extra)


if __name__ == "__main__":
    print(build(verbose=True))
