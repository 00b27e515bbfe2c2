"""Build liberase.so in-tree with hipcc for gfx950.

    python -m paper_2608_18469_amd.build

Compiles the HIP kernels and the C-ABI dispatcher into one shared library
next to this file.  Packed-FP32 instructions are disabled for all device code.
MFMA accumulators are allocated in the architectural VGPRs: with the default
heuristic (accumulation registers) the register allocator permutes the
accumulators between the unrolled halves of the GEMM main loops and repairs
the permutation with register copies that wait on MFMA results.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "liberase.so")
SOURCES = [os.path.join(HERE, "csrc", f) for f in ("kernels.hip", "embed.hip", "transformer.hip", "erase_api.cpp", "tf_api.cpp")]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found; the HIP library cannot be built")


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-mllvm", "-amdgpu-mfma-vgpr-form", "-fvisibility=hidden",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc"),
           *SOURCES, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops' is not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
