"""Stored fingerprints and oracle digests (written by tests/golden/make_golden.py,
which calls only the input generators and the CPU oracle)."""
import os

import pytest

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _read(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return dict(line.split() for line in f if line.strip())


@pytest.mark.parametrize("name", ["tiny", "llama3-8b-decode", "restore-burst",
                                  "llama3-70b-tp8-shard", "qwen-gqa-hnd"])
def test_workload_fingerprint(name):
    from paper_2606_17787_amd import workloads as W
    assert W.WORKLOADS[name]().fingerprint() == _read("workload_fingerprints.txt")[name]


def test_oracle_digests():
    import importlib.util
    spec = importlib.util.spec_from_file_location(
        "make_golden", os.path.join(GOLDEN, "make_golden.py"))
    mg = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mg)
    assert mg.oracle_digests() == _read("oracle_digests.txt")
