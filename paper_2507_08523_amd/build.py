"""Builds libilpc.so (host prefix cache + gfx950 kernels) in-tree with hipcc.

    python -m paper_2507_08523_amd.build

Every HIP translation unit is compiled for gfx950 only, with packed-fp32 VALU
instructions disabled (``-target-feature -packed-fp32-ops``; the host pass
warns that it does not know the feature, which is harmless).
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libilpc.so")
SOURCES = [os.path.join(PKG, "csrc", "prefix_cache.cpp"), os.path.join(PKG, "csrc", "pair_table.cpp"),
           os.path.join(PKG, "csrc", "schedule.cpp"),
           os.path.join(PKG, "csrc", "paged_attn.hip"), os.path.join(PKG, "csrc", "rope_append.hip"),
           os.path.join(PKG, "csrc", "decode_attn.hip"),
           os.path.join(PKG, "csrc", "attn_noalloc.hip")]
ARCH = "gfx950"


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def build(verbose: bool = False) -> str:
    """Compile the library (always recompiles) and return its path."""
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Wall", "-Wno-unused-result", "-I", os.path.join(ROOT, "include"),
           *SOURCES, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    msgs = [ln for ln in (res.stdout + res.stderr).splitlines() if noise not in ln]
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs), file=sys.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
