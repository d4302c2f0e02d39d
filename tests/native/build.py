"""Builds tests/native/abi_conformance (a plain HIP host program that drives
the C ABI and checks it against the C oracle) next to its source.  Called
by __graft_entry__.build() after the library and the oracle are built, so
that the GPU test only runs it.

    python tests/native/build.py
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "abi_conformance.cpp")
OUT = os.path.join(HERE, "abi_conformance")


def build(verbose: bool = False) -> str:
    hipcc = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin",
                         "hipcc")
    cmd = [hipcc, "-std=c++17", "-O2", "-Wall", "-Werror",
           "-I", os.path.join(ROOT, "include"), SRC,
           "-L", os.path.join(ROOT, "paper_2606_17787_amd"),
           "-llumen_kv_ckpt", "-L", os.path.join(ROOT, "oracle"),
           "-llumen_oracle",
           "-Wl,-rpath,$ORIGIN/../../paper_2606_17787_amd:$ORIGIN/../../oracle",
           "-o", OUT]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"abi_conformance build failed:\n{res.stderr}")
    return OUT


if __name__ == "__main__":
    print(build(verbose=True))
