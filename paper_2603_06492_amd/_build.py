"""Builds libnoble.so (the HIP kernels and the C ABI) in-tree for gfx950."""

from __future__ import annotations

import os
import shutil
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libnoble.so")
SOURCES = ["noble_api.hip"]
HEADERS = ["noble_act.hpp", "noble_init.hpp", "noble_kernels.hpp", "noble_tiles.hpp", "noble_gemm.hpp", "noble_gemm_dma.hpp", "noble_skinny.hpp"]

HIP_FLAGS = [
    "-O3",
    "-std=c++20",
    "--offload-arch=gfx950",
    "-fPIC",
    "-shared",
    "-munsafe-fp-atomics",
    # no packed-FP32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libnoble)")


def build(verbose: bool = False) -> str:
    """Compile libnoble.so; always recompiles.  Returns the library path."""
    tmp = LIB + ".tmp"
    cmd = [hipcc(), *HIP_FLAGS, "-I", INCLUDE, "-I", CSRC,
           *[os.path.join(CSRC, s) for s in SOURCES], "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
