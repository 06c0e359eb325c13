"""Build libsaf.so in-tree with hipcc for gfx950.

Usage: ``python -m paper_2609_34650_amd.build``.  Always recompiles.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libsaf.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-shared",
    "-fPIC",
    "-fvisibility=hidden",
    # No packed-fp32 VALU instructions in any kernel.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA accumulators in ordinary VGPRs: the softmax works on them directly,
    # with no copies between AGPRs and VGPRs.
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    # Schedule for instruction-level parallelism (LDS reads issued well ahead
    # of the MFMAs that consume them) rather than for the smallest register
    # count: every kernel runs at two wavefronts per SIMD either way.
    "-mllvm", "-amdgpu-sched-strategy=max-ilp",
    "-Wall",
    "-Wno-unused-function",
]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; libsaf.so needs ROCm's hipcc")
    return path


def build(verbose: bool = False) -> str:
    """Compile ``csrc/saf_api.hip`` (which includes every kernel) into
    ``libsaf.so`` next to this file; returns its path."""
    src = os.path.join(CSRC, "saf_api.hip")
    tmp = LIB + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, "-I", INCLUDE, "-I", CSRC, src, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    out = (res.stdout or "") + (res.stderr or "")
    # hipcc's host pass does not know the packed-fp32 feature; that warning is expected.
    noise = "'-packed-fp32-ops' is not a recognized feature for this target"
    lines = [ln for ln in out.splitlines() if noise not in ln and "(ignoring feature)" not in ln]
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(lines))
    if verbose and lines:
        print("\n".join(lines))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
