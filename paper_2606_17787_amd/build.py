"""Builds the HIP library in-tree for gfx950.

    python -m paper_2606_17787_amd.build

compiles csrc/lumen_kv_ckpt.hip (device kernels and their host entry
points) and the host-only csrc/lumen_page_tags.cpp (page tags),
csrc/lumen_sched.cpp (placement and recovery scheduling) and
csrc/lumen_progress.cpp (checkpoint progress) with hipcc into
paper_2606_17787_amd/liblumen_kv_ckpt.so (position-independent, C ABI from
include/lumen_kv_ckpt.h, lumen_page_tags.h, lumen_sched.h and
lumen_progress.h).
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "lumen_kv_ckpt.hip")
SRC_TAGS = os.path.join(PKG, "csrc", "lumen_page_tags.cpp")
SRC_SCHED = os.path.join(PKG, "csrc", "lumen_sched.cpp")
SRC_PROGRESS = os.path.join(PKG, "csrc", "lumen_progress.cpp")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "liblumen_kv_ckpt.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Wall", "-Werror",
    # no packed-FP32 instructions in any device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def build(out: str = LIB, extra_flags=(), verbose: bool = False) -> str:
    hipcc = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    cmd = [hipcc, *HIPCC_FLAGS, *extra_flags, "-I", INCLUDE, SRC, SRC_TAGS,
           SRC_SCHED, SRC_PROGRESS, "-o", out]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "'-packed-fp32-ops' is not a recognized feature for this target"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
