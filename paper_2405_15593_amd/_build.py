"""Builds libmicroadam.so (HIP for gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIBRARY = os.path.join(PKG, "libmicroadam.so")
SOURCES = [os.path.join(CSRC, f) for f in ("microadam_kernels.hip", "microadam_api.cpp")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # one rounding per written operation: results that decide integers
    # (EF codes, Top-K) must not depend on FMA contraction
    "-ffp-contract=off",
    # no packed FP32 instructions in generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # device code: min/max without IEEE NaN quieting, so that they fuse with
    # lane permutes (gradients are taken to be finite)
    "-Xarch_device", "-fno-honor-nans", "-Xarch_device", "-mno-amdgpu-ieee",
    "-Wall", "-Wno-unused-function",
    "-I", INCLUDE, "-I", CSRC,
    "-Wl,-rpath,/opt/rocm/lib",
]


def build(verbose: bool = False) -> str:
    """Compiles every HIP/C++ source of the library; always rebuilds."""
    tmp = LIBRARY + ".tmp"
    cmd = [HIPCC, *FLAGS, "-x", "hip", SOURCES[0], "-x", "hip", SOURCES[1], "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{res.stderr[-6000:]}")
    os.replace(tmp, LIBRARY)
    return LIBRARY


if __name__ == "__main__":
    print(build(verbose=True))
