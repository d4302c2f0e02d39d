"""The C ABI used from a plain HIP host program, without Python or torch:
tests/native/abi_conformance allocates its own buffers and streams, runs
plan, pack, unpack, status, the direct host copy, both staging pipelines and
validate mode through include/lumen_kv_ckpt.h, and compares every result
with the C oracle byte for byte (two layouts, three seeds each).  __graft_entry__.build() builds
it."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "native",
                   "abi_conformance")


def test_c_program_matches_oracle():
    assert os.path.exists(EXE), \
        "tests/native/abi_conformance is not built: run __graft_entry__.build()"
    print("running", EXE, flush=True)
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert "abi conformance ok" in r.stdout
