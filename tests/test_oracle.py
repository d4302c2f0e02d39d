"""The CPU oracle against its pins (no GPU needed).

Besides running every pin against the real oracle, a mutation test compiles
copies of the oracle with one plausible mistake planted each (a dropped term,
a wrong index, a transposed operand, an off-by-one bound) and checks that at
least one pin catches every one of them.
"""
import os
import shutil
import subprocess
import sys
import tempfile

import numpy as np
import pytest

import oracle
import oracle_pins as P


@pytest.mark.parametrize("pin", P.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin, oracle_lib):
    pin(oracle_lib)


# (description, text in lumen_oracle.c, replacement)
MUTANTS = [
    ("slot from division", "int64_t slot = t % sh->block_size;",
     "int64_t slot = t / sh->block_size;"),
    ("head-major index uses token-major order",
     "((((l * 2 + kv) * NB + b) * H + h) * bs + s) * D + d",
     "((((l * 2 + kv) * NB + b) * bs + s) * H + h) * D + d"),
    ("token-major index swaps head and slot",
     "((((l * 2 + kv) * NB + b) * bs + s) * H + h) * D + d;\n}",
     "((((l * 2 + kv) * NB + b) * H + h) * bs + s) * D + d;\n}"),
    ("checkpoint row swaps layer and K/V", "(((row * L + l) * 2 + kv) * H + h)",
     "(((row * 2 + kv) * L + l) * H + h)"),
    ("checkpoint row drops the head term", "(((row * L + l) * 2 + kv) * H + h)",
     "(((row * L + l) * 2 + kv) * H + 0)"),
    ("cache index drops K/V", "((l * 2 + kv) * NB + b)", "((l * 2) * NB + b)"),
    ("row off by one", "int64_t row = first_row[r] + (t - start[r]);\n            for",
     "int64_t row = first_row[r] + (t - start[r]) + 1;\n            for"),
    ("plan drops one token per request", "next += n;", "next += n - (n > 0);"),
    ("per-request rows ignore start",
     "first_row[r] = req_row_base[r] + start[r];",
     "first_row[r] = req_row_base[r];"),
    ("page bound off by one", "if (page >= bt_cols)", "if (page > bt_cols)"),
    ("block bound off by one", "b >= sh->num_blocks", "b > sh->num_blocks"),
    ("capacity bound off by one", "row >= ckpt_rows", "row > ckpt_rows"),
    ("negative start accepted", "if (start[r] < 0 || n < 0)", "if (n < 0)"),
    ("first error instead of most negative",
     "static int worse(int a, int b) { return a < b ? a : b; }",
     "static int worse(int a, int b) { return a ? a : b; }"),
    ("head dim reversed", "* H + h) * D + d;\n}\n\nstatic int worse",
     "* H + h) * D + (D - 1 - d);\n}\n\nstatic int worse"),
    ("validate takes one page too many",
     "int64_t last = (end[r] - 1) / sh->block_size;",
     "int64_t last = end[r] / sh->block_size;"),
    ("validate starts at page 0", "int64_t first = start[r] / sh->block_size;",
     "int64_t first = 0;"),
    ("validate needs three owners", "if (times[b] > 1)", "if (times[b] > 2)"),
    ("validate ignores bad ranges",
     "status = worse(status, ORACLE_ERR_RANGE);\n            continue;\n"
     "        }\n        if (end[r] == start[r])",
     "continue;\n        }\n        if (end[r] == start[r])"),
    ("validate pool bound off by one",
     "if (b < 0 || b >= sh->num_blocks) {\n                status = worse("
     "status, ORACLE_ERR_BLOCK_ID);\n                continue;\n            }"
     "\n            times[b]",
     "if (b < 0 || b > sh->num_blocks) {\n                status = worse("
     "status, ORACLE_ERR_BLOCK_ID);\n                continue;\n            }"
     "\n            times[b]"),
]


_RUN_PINS = r"""
import sys
sys.path[:0] = [{root!r}, {tests!r}]
import oracle, oracle_pins as P
lib = oracle.load({so!r})
try:
    P.pin_bruteforce_decode(lib, exhaustive=False)
    P.pin_plan_prefix_sum(lib)
    P.pin_invariants(lib)
    P.pin_torch_indexing(lib)
    P.pin_error_codes(lib)
    P.pin_validate_targets(lib, exhaustive=False)
except AssertionError as exc:
    print("PINS_FAIL", repr(exc)[:200])
    sys.exit(0)
print("PINS_PASS")
"""


@pytest.mark.parametrize("mutant", MUTANTS, ids=lambda m: m[0])
def test_pins_catch_planted_mistake(mutant):
    """The pins run in a child process: a planted mistake may write out of
    bounds, and must be caught by an assertion before it can do so."""
    _, old, new = mutant
    src = open(oracle._SRC).read()
    assert old in src, "mutation site not found; update the mutant list"
    tmp = tempfile.mkdtemp(prefix="oracle_mutant_")
    try:
        shutil.copy(oracle._HDR, tmp)
        path = os.path.join(tmp, "lumen_oracle.c")
        with open(path, "w") as f:
            f.write(src.replace(old, new))
        so = oracle.build(src=path, out=os.path.join(tmp, "mutant.so"),
                          extra_flags=("-Wno-unused-parameter",))
        here = os.path.dirname(os.path.abspath(__file__))
        code = _RUN_PINS.format(root=os.path.dirname(here), tests=here, so=so)
        res = subprocess.run([sys.executable, "-c", code], capture_output=True,
                             text=True, timeout=300)
        assert "PINS_FAIL" in res.stdout, (res.returncode, res.stdout,
                                           res.stderr[-2000:])
    finally:
        shutil.rmtree(tmp)


def test_workload_generators_reproducible():
    from paper_2606_17787_amd import workloads as W
    a, b = W.c1_tiny(), W.c1_tiny()
    assert a.fingerprint() == b.fingerprint()
    assert list(a.ctx) == [195, 202, 251, 291, 107, 128, 265, 290]
    w = W.c2_llama8b()
    assert w.num_blocks == 56323 and w.dst_num_blocks == 13836
    tok = [w.step_tokens(k) for k in range(w.num_steps)]
    assert 1993 <= min(tok) and max(tok) <= 2379


def test_c1_full_roundtrip(oracle_lib):
    from paper_2606_17787_amd import workloads as W
    w = W.c1_tiny()
    rng = np.random.default_rng(1001)
    src = W.random_bits(rng, w.shape.pool_elems(w.num_blocks))
    st, ck = oracle.pack(w.shape, w.num_blocks, src, w.block_tables,
                         w.starts[0], w.ends[0], lib=oracle_lib)
    assert st == 0 and ck.shape == (1729, 512)
    assert np.array_equal(ck, P.torch_gather(w.shape, w.num_blocks, src,
                                             w.block_tables, w.starts[0],
                                             w.ends[0]))
    dst = W.random_bits(rng, w.shape.pool_elems(w.dst_num_blocks))
    assert oracle.unpack(w.shape, w.dst_num_blocks, dst, w.dst_block_tables,
                         w.starts[0], w.ends[0], ck, lib=oracle_lib) == 0
    st, back = oracle.pack(w.shape, w.dst_num_blocks, dst, w.dst_block_tables,
                           w.starts[0], w.ends[0], lib=oracle_lib)
    assert st == 0 and np.array_equal(back, ck)
