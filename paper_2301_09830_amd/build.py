"""Build liboptcc.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2301_09830_amd.build        # or build() from Python

The library is a single translation unit (csrc/api.hip includes the kernel
templates).  Packed-fp32 VALU instructions are disabled for the device code.
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
LIB = os.path.join(PKG, "liboptcc.so")
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build liboptcc)")


def compile_command(out: str = LIB) -> list:
    return [
        hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
        "-ffp-contract=off",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-Wno-unused-result",
        "-I", INCLUDE, "-I", CSRC,
        os.path.join(CSRC, "api.hip"),
        "-o", out,
    ]


def build(verbose: bool = False) -> str:
    """Compile liboptcc.so for gfx950 next to this file; returns its path."""
    tmp = LIB + ".tmp"
    cmd = compile_command(tmp)
    proc = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    errlines = [ln for ln in proc.stderr.splitlines() if noise not in ln]
    if proc.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + "\n".join(errlines))
    if verbose and errlines:
        print("\n".join(errlines), file=sys.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
