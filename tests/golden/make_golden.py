"""Writes the stored expected values under tests/golden/.

Run from the repository root:  python tests/golden/make_golden.py

It calls only the seeded input generators and the CPU oracle, never the GPU
library.  The files it writes are:

* workload_fingerprints.txt -- SHA-256 of every workload's generated metadata
  (context lengths, ranges, block tables).  A change means the generator or
  numpy's PCG64 stream changed, and every stored value below is suspect.
* oracle_digests.txt -- SHA-256 of the oracle's checkpoint bytes for the tiny
  workload (full pack) and for the first two steps of a reduced Llama-3-8B
  decode workload, each over a pool of seeded random 16-bit patterns.
"""
import hashlib
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
from paper_2606_17787_amd import workloads as W  # noqa: E402


def oracle_digests():
    out = {}
    w = W.c1_tiny()
    pool = W.random_bits(np.random.default_rng(1000), w.shape.pool_elems(w.num_blocks))
    st, ck = oracle.pack(w.shape, w.num_blocks, pool, w.block_tables,
                         w.starts[0], w.ends[0])
    assert st == 0
    out["tiny.pack"] = hashlib.sha256(ck.tobytes()).hexdigest()
    dst = W.random_bits(np.random.default_rng(1001), w.shape.pool_elems(w.dst_num_blocks))
    assert oracle.unpack(w.shape, w.dst_num_blocks, dst, w.dst_block_tables,
                         w.starts[0], w.ends[0], ck) == 0
    out["tiny.unpack_pool"] = hashlib.sha256(dst.tobytes()).hexdigest()

    w = W.c2_llama8b(num_reqs=6, steps=2, median=200, clip_hi=400)
    pool = W.random_bits(np.random.default_rng(2000), w.shape.pool_elems(w.num_blocks))
    for k in range(w.num_steps):
        st, ck = oracle.pack(w.shape, w.num_blocks, pool, w.block_tables,
                             w.starts[k], w.ends[k])
        assert st == 0
        out[f"llama3-8b-decode-small.step{k}"] = hashlib.sha256(ck.tobytes()).hexdigest()
    return out


def main():
    with open(os.path.join(HERE, "workload_fingerprints.txt"), "w") as f:
        for name, make in W.WORKLOADS.items():
            f.write(f"{name} {make().fingerprint()}\n")
    with open(os.path.join(HERE, "oracle_digests.txt"), "w") as f:
        for k, v in oracle_digests().items():
            f.write(f"{k} {v}\n")


if __name__ == "__main__":
    main()
