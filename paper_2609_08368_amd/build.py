"""Compile librlattn.so (HIP for gfx950) in-tree with hipcc.

Usage: ``python -m paper_2609_08368_amd.build`` (``__graft_entry__.build()`` calls it).
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "librlattn.so")
ARCH = os.environ.get("RL_ATTN_ARCH", "gfx950")

SOURCES = ["decode.hip", "extend.hip", "append.hip", "diag.hip", "scratch.hip", "rl_attn_host.cpp"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build librlattn.so)")


def build(verbose: bool = False) -> str:
    """Compile every HIP source into librlattn.so next to this file; returns its path."""
    out_tmp = LIB + ".tmp"
    cmd = [
        hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
        # packed FP32 instructions stay off: ordinary float code only
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        # device code: scores are never NaN unless the inputs are (a NaN still
        # reaches the output through the exponent), so fmaxf needs no NaN-quieting
        # canonicalisation; the host code keeps full NaN semantics
        "-Xarch_device", "-fno-honor-nans",
        "-I", os.path.join(ROOT, "include"), "-I", CSRC,
        "-Wall", "-Wno-unused-result",
        *[os.path.join(CSRC, s) for s in SOURCES],
        "-o", out_tmp,
    ]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    msgs = "\n".join(l for l in (res.stdout + res.stderr).splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{msgs}")
    if verbose and msgs.strip():
        print(msgs, file=sys.stderr)
    os.replace(out_tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
