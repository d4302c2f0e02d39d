"""GPU path vs the CPU oracle, element by element (bit-exact: the path is a
pure copy).  Sizes here let the oracle finish in seconds while spanning many
wavefront spans, partial blocks and ragged tails; full-size workloads are in
test_gpu_fullsize.py."""
import zlib

import numpy as np
import pytest
import torch

import oracle
import paper_2606_17787_amd.kvckpt as kv
from paper_2606_17787_amd import workloads as W
from paper_2606_17787_amd.workloads import CacheShape, HND, NHD

from gpu_util import (SENTINEL, assert_same, gpu_path, oracle_path, h2d,
                      d2h16, dev)

pytestmark = pytest.mark.gpu

# The two ways to run a plan's copies: the plan kernel into a workspace and
# the copies over it, or the one-launch copies that read the ranges.
VIAS = ["plan", "ranges"]


def test_smoke():
    import __graft_entry__
    __graft_entry__.smoke()


def test_tiny_workload_full_pack_and_restore():
    w = W.c1_tiny()
    rng = np.random.default_rng(101)
    src = W.random_bits(rng, w.shape.pool_elems(w.num_blocks))
    dst = W.random_bits(rng, w.shape.pool_elems(w.dst_num_blocks))
    args = (w.shape, w.num_blocks, src, w.block_tables, w.starts[0],
            w.ends[0], w.dst_num_blocks, dst, w.dst_block_tables)
    assert_same(gpu_path(*args), oracle_path(*args), "tiny")


@pytest.mark.parametrize("via", VIAS)
def test_prepared_calls_match_the_oracle(via):
    """Plan, pack and unpack (or the one-launch range copies) prepared once
    and issued twice on the same buffers, with the token ranges rewritten in
    place in between (a serving loop's use): each round equals the oracle,
    and the plain calls."""
    w = W.c1_tiny()
    sh = w.shape
    rng = np.random.default_rng(202)
    src = W.random_bits(rng, sh.pool_elems(w.num_blocks))
    dst = W.random_bits(rng, sh.pool_elems(w.dst_num_blocks))
    s0, e0 = w.starts[0], w.ends[0]
    s1 = (s0 + rng.integers(0, 40, len(s0))).astype(np.int32)
    e1 = np.maximum(s1, e0 - rng.integers(0, 40, len(e0))).astype(np.int32)
    rows = int(max((e0 - s0).sum(), (e1 - s1).sum()))
    d_s, d_e = h2d(s0), h2d(e0)
    d_src, d_dst = h2d(src), h2d(dst)
    ck = torch.zeros(rows * sh.token_row_elems, dtype=torch.int16,
                     device=dev())
    ws = kv.new_workspace(len(s0), dev())
    status = torch.zeros(1, dtype=torch.int32, device=dev())
    if via == "ranges":
        pack = kv.prepare_pack_ranges(sh, w.num_blocks, d_src,
                                      h2d(w.block_tables), d_s, d_e, ck,
                                      status)
        unpack = kv.prepare_unpack_ranges(sh, w.dst_num_blocks, d_dst,
                                          h2d(w.dst_block_tables), d_s, d_e,
                                          ck, status)

        def plan():
            pass
    else:
        plan = kv.prepare_plan(d_s, d_e, ws)
        pack = kv.prepare_pack(sh, w.num_blocks, d_src, h2d(w.block_tables),
                               ws, ck)
        unpack = kv.prepare_unpack(sh, w.dst_num_blocks, d_dst,
                                   h2d(w.dst_block_tables), ws, ck)
    want_dst = dst.copy()
    for s, e in ((s0, e0), (s1, e1)):
        d_s.copy_(torch.from_numpy(s))
        d_e.copy_(torch.from_numpy(e))
        plan()
        pack()
        unpack()
        torch.cuda.synchronize()
        assert kv.lumen_kv_ckpt_status(ws) == 0
        assert int(status.item()) == 0
        n = int((e - s).sum())
        st, want = oracle.pack(sh, w.num_blocks, src, w.block_tables, s, e)
        assert st == oracle.OK
        assert oracle.unpack(sh, w.dst_num_blocks, want_dst,
                             w.dst_block_tables, s, e, want) == oracle.OK
        got = d2h16(ck)[:n * sh.token_row_elems].reshape(want.shape)
        assert np.array_equal(got, want)
        assert np.array_equal(d2h16(d_dst), want_dst)
        # the plain call on the same ranges writes the same rows
        ck2 = torch.zeros_like(ck)
        kv.lumen_kv_ckpt_plan(d_s, d_e, ws)
        kv.lumen_kv_ckpt_pack(sh, w.num_blocks, d_src, h2d(w.block_tables),
                              ws, ck2)
        assert kv.lumen_kv_ckpt_status(ws) == 0
        assert torch.equal(ck2[:n * sh.token_row_elems],
                           ck[:n * sh.token_row_elems])


@pytest.mark.parametrize("which", ["shortest", "first", "pair"])
def test_tp8_shape_small_checkpoints(which):
    """Requests of the 70B TP=8 shard's shape (80 layers, one KV head: units
    of 512 bytes) with checkpoint buffers sized to their rows, 16 KB to
    200 MB, where the copy grid is bounded by one wavefront per 4 KiB of
    checkpoint rather than one per unit: the full pack, the same rows
    through a window (the token-major walk) and the restore into a second,
    fragmented pool, against the oracle."""
    w = W.c4_llama70b_tp8()
    sh = w.shape
    ctx = w.ends[0].astype(np.int64)
    reqs = {"shortest": [int(np.argmin(ctx))], "first": [0],
            "pair": [0, 1]}[which]
    rng = np.random.default_rng(400 + len(reqs) + int(ctx[reqs[0]]))
    lens = ctx[reqs]
    s = np.zeros(len(reqs), np.int32)
    if which == "pair":
        s[1] = lens[1] // 3  # a request whose prefix was checkpointed before
    e = lens.astype(np.int32)
    pages = -(-lens // sh.block_size)
    cols = int(pages.max())
    nb = int(pages.sum()) + 5

    def table():
        perm = rng.permutation(nb).astype(np.int32)
        bt = np.full((len(reqs), cols), -1, np.int32)
        o = 0
        for i, p in enumerate(pages):
            bt[i, :p] = perm[o:o + p]
            o += p
        return bt

    bt, bt2 = table(), table()
    src = W.random_bits(rng, sh.pool_elems(nb))
    dst = W.random_bits(rng, sh.pool_elems(nb))
    args = (sh, nb, src, bt, s, e, nb, dst, bt2)
    ref = oracle_path(*args)
    assert_same(gpu_path(*args), ref, f"70B shape, {which}")
    rows = int((e - s).sum())
    ws = kv.new_workspace(len(reqs), dev())
    kv.lumen_kv_ckpt_plan(h2d(s), h2d(e), ws)
    win = torch.empty(rows * sh.token_row_elems, dtype=torch.int16,
                      device=dev())
    kv.lumen_kv_ckpt_pack_rows(sh, nb, h2d(src), h2d(bt), ws, 0, rows, win)
    assert kv.lumen_kv_ckpt_status(ws) == 0
    assert np.array_equal(d2h16(win).reshape(-1, sh.token_row_elems), ref[1])


SHAPES = [
    CacheShape(1, 1, 8, 1, NHD), CacheShape(1, 1, 8, 1, HND),
    CacheShape(2, 2, 64, 2, NHD), CacheShape(2, 2, 64, 3, HND),
    CacheShape(5, 3, 24, 3, NHD), CacheShape(5, 3, 24, 3, HND),
    CacheShape(2, 1, 128, 16, NHD), CacheShape(3, 4, 128, 16, HND),
    CacheShape(2, 4, 64, 32, NHD), CacheShape(3, 2, 128, 32, HND),
    CacheShape(4, 8, 128, 16, NHD), CacheShape(1, 3, 40, 5, HND),
    # 8-bit and fp32 caches (still 16-byte head rows)
    CacheShape(1, 1, 16, 1, NHD, elem_bytes=1),
    CacheShape(2, 3, 32, 3, HND, elem_bytes=1),
    CacheShape(3, 8, 128, 16, NHD, elem_bytes=1),
    CacheShape(2, 2, 128, 16, HND, elem_bytes=1),
    CacheShape(1, 1, 4, 1, NHD, elem_bytes=4),
    CacheShape(2, 3, 12, 5, HND, elem_bytes=4),
    CacheShape(3, 4, 128, 16, NHD, elem_bytes=4),
    CacheShape(2, 2, 64, 32, HND, elem_bytes=4),
]


def _case(rng, shape, R, max_tok, incremental, nb_extra=7):
    bs = shape.block_size
    cols = -(-max_tok // bs) + 1
    nb = R * cols + nb_extra
    perm = rng.permutation(nb).astype(np.int32)
    bt = perm[:R * cols].reshape(R, cols)
    bt2 = rng.permutation(nb).astype(np.int32)[:R * cols].reshape(R, cols)
    if incremental:
        s = rng.integers(0, max_tok + 1, R)
        e = np.minimum(s + rng.integers(0, 3 * bs + 2, R), max_tok)
    else:
        s = np.zeros(R, np.int64)
        e = rng.integers(0, max_tok + 1, R)
    s, e = s.astype(np.int32), e.astype(np.int32)
    empty = rng.random(R) < 0.15
    e[empty] = s[empty]
    src = W.random_words(rng, shape.pool_elems(nb), shape.elem_bytes)
    dst = W.random_words(rng, shape.pool_elems(nb), shape.elem_bytes)
    return nb, bt, bt2, s, e, src, dst


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"L{s.num_layers}H{s.num_kv_heads}D{s.head_dim}bs{s.block_size}{s.order}e{s.elem_bytes}")
@pytest.mark.parametrize("incremental", [False, True])
@pytest.mark.parametrize("via", VIAS)
def test_random_shapes(shape, incremental, via):
    rng = np.random.default_rng(zlib.crc32(f"{shape}{incremental}".encode()))
    for R, max_tok in ((1, 5), (3, 40), (17, 100), (70, 30)):
        nb, bt, bt2, s, e, src, dst = _case(rng, shape, R, max_tok,
                                            incremental)
        args = (shape, nb, src, bt, s, e, nb, dst, bt2)
        assert_same(gpu_path(*args, via=via), oracle_path(*args),
                    f"R={R} packed")
        # rows placed after an offset, with spare rows that stay untouched
        n = int((e - s).sum())
        kw = dict(row_base=3, ckpt_rows=n + 6)
        assert_same(gpu_path(*args, **kw, via=via), oracle_path(*args, **kw),
                    f"R={R} row_base")
        # per-request reserved regions: token t of r at row base[r] + t
        base = np.arange(R, dtype=np.int64) * (max_tok + 2)
        kw = dict(req_row_base=base, ckpt_rows=R * (max_tok + 2))
        assert_same(gpu_path(*args, **kw, via=via), oracle_path(*args, **kw),
                    f"R={R} per-request")


@pytest.mark.parametrize("via", VIAS)
def test_empty_plan_and_all_empty_ranges(via):
    shape = CacheShape(2, 2, 64, 16, NHD)
    rng = np.random.default_rng(5)
    nb = 8
    src = W.random_bits(rng, shape.pool_elems(nb))
    dst = W.random_bits(rng, shape.pool_elems(nb))
    bt = np.arange(8, dtype=np.int32).reshape(4, 2)
    s = np.array([3, 0, 31, 7], np.int32)
    args = (shape, nb, src, bt, s, s, nb, dst, bt)
    assert_same(gpu_path(*args, ckpt_rows=2, via=via),
                oracle_path(*args, ckpt_rows=2), "all empty")


ERROR_CASES = [
    # (start, end, bt, ckpt_rows, row_base, req_row_base)
    ([0, 0], [12, 8], None, 20, 0, None),
    ([0, 0], [13, 8], None, 64, 0, None),
    ([0, 0], [12, 9], None, 64, 0, None),
    ([3, 0], [2, 8], None, 64, 0, None),
    ([-1, 0], [2, 8], None, 64, 0, None),
    ([0, 0], [8, 1], [[0, 8, 2], [3, 4, -1]], 64, 0, None),
    ([0, 0], [4, 1], [[0, 8, 2], [3, 4, -1]], 64, 0, None),
    ([0, 0], [12, 8], None, 19, 0, None),
    ([0, 0], [12, 8], None, 25, 6, None),
    ([2, 0], [4, 1], None, 100, 0, [-3, 0]),
    ([0, 0], [13, 9], None, 1, 0, None),
    ([5, 0], [4, 9], None, 64, 0, None),
]


@pytest.mark.parametrize("case", range(len(ERROR_CASES)))
@pytest.mark.parametrize("via", VIAS)
def test_device_error_codes_match_oracle(case, via):
    s, e, bt, rows, base, rb = ERROR_CASES[case]
    shape = CacheShape(2, 2, 8, 4, NHD)
    nb = 8
    bt = np.array(bt if bt is not None else [[0, 1, 2], [3, 4, -1]], np.int32)
    rng = np.random.default_rng(case)
    src = W.random_bits(rng, shape.pool_elems(nb))
    ck = np.zeros(((rows + 8), shape.token_row_elems), np.uint16)
    st_o, _ = oracle.pack(shape, nb, src, bt, s, e, base, rb, ckpt=ck,
                          ckpt_rows=rows)
    st_g, _, _ = gpu_path(shape, nb, src, bt, s, e, row_base=base,
                          req_row_base=rb, ckpt_rows=rows, via=via)
    assert st_g == st_o, (st_g, st_o)
    # a fresh plan (or status word) starts a new error epoch and a clean run
    # reports OK
    st_g, _, _ = gpu_path(shape, nb, src, np.array([[0, 1, 2], [3, 4, 5]],
                                                   np.int32), [0, 0], [1, 1],
                          via=via)
    assert st_g == kv.LUMEN_OK


# One shape per walk of the copy kernels: 32-byte token runs (the full pack
# takes the page-major walk), 1 KiB runs (token-major walk) and a head-major
# cache.
ERROR_WALK_SHAPES = {
    "nhd-page-major": CacheShape(2, 2, 8, 4, NHD),
    "nhd-token-major": CacheShape(2, 8, 64, 4, NHD),
    "hnd": CacheShape(2, 2, 8, 4, HND),
}


def _valid_token_rows(shape, nb, bt, s, e, rows, base, rb):
    """(request, token, checkpoint row) of every token that passes the
    per-row checks the header documents, in their order: page inside the
    table, entry inside the pool, row inside the buffer.  Requests whose
    range is invalid contribute no rows."""
    out, run = [], int(base)
    for r in range(len(s)):
        if s[r] < 0 or e[r] < s[r]:
            continue
        first = (int(rb[r]) + int(s[r])) if rb is not None else run
        run += int(e[r]) - int(s[r])
        for t in range(int(s[r]), int(e[r])):
            j = t // shape.block_size
            crow = first + (t - int(s[r]))
            if j >= bt.shape[1] or not 0 <= bt[r, j] < nb:
                continue
            if 0 <= crow < rows:
                out.append((r, t, crow))
    return out


@pytest.mark.parametrize("walk", list(ERROR_WALK_SHAPES))
@pytest.mark.parametrize("case", range(len(ERROR_CASES)))
@pytest.mark.parametrize("via", VIAS)
def test_error_inputs_still_copy_every_valid_row(case, walk, via):
    """On data-dependent errors only the offending token rows are skipped:
    every other row of the pack equals the oracle's pack of that token
    alone, rows no valid token names keep their sentinel, and the unpack
    writes exactly the valid tokens' slots, for each walk of the kernels."""
    s, e, bt, rows, base, rb = ERROR_CASES[case]
    shape = ERROR_WALK_SHAPES[walk]
    nb = 8
    bt = np.array(bt if bt is not None else [[0, 1, 2], [3, 4, -1]], np.int32)
    s, e = np.asarray(s, np.int32), np.asarray(e, np.int32)
    rng = np.random.default_rng(1000 + case)
    src = W.random_bits(rng, shape.pool_elems(nb))
    dst = W.random_bits(rng, shape.pool_elems(nb))
    ck_in = W.random_bits(rng, rows * shape.token_row_elems)
    valid = _valid_token_rows(shape, nb, bt, s, e, rows, base, rb)

    want_ck = np.full((rows, shape.token_row_elems), SENTINEL, np.uint16)
    want_dst = dst.copy()
    named = {}  # checkpoint row -> the rows of the tokens naming it
    for r, t, crow in valid:
        st, one = oracle.pack(shape, nb, src, bt[r:r + 1], [t], [t + 1])
        assert st == oracle.OK
        want_ck[crow] = one[0]
        named.setdefault(crow, []).append(one[0])
        assert oracle.unpack(shape, nb, want_dst, bt[r:r + 1], [t], [t + 1],
                             ck_in.reshape(rows, -1)[crow:crow + 1]) == 0
    st_o, _ = oracle.pack(shape, nb, src, bt, s, e, base, rb,
                          ckpt=np.zeros((rows + 8, shape.token_row_elems),
                                        np.uint16), ckpt_rows=rows)

    ws = kv.new_workspace(len(s), dev())
    d_rb = None if rb is None else h2d(np.asarray(rb, np.int64))
    d_s, d_e, d_bt = h2d(s), h2d(e), h2d(bt)
    ck = h2d(np.full(rows * shape.token_row_elems, SENTINEL, np.uint16))

    def copy(pack, cache, ckpt):
        if via == "ranges":
            status = torch.zeros(1, dtype=torch.int32, device=dev())
            fn = (kv.lumen_kv_ckpt_pack_ranges if pack
                  else kv.lumen_kv_ckpt_unpack_ranges)
            fn(shape, nb, cache, d_bt, d_s, d_e, ckpt, status, base, d_rb)
            return int(status.item())
        kv.lumen_kv_ckpt_plan(d_s, d_e, ws, base, d_rb)
        fn = kv.lumen_kv_ckpt_pack if pack else kv.lumen_kv_ckpt_unpack
        fn(shape, nb, cache, d_bt, ws, ckpt)
        return kv.lumen_kv_ckpt_status(ws)

    assert copy(True, h2d(src), ck) == st_o
    got_ck = d2h16(ck).reshape(rows, -1)
    # Overlapping per-request regions (a caller error): the writers of a row
    # two tokens name race, so each element holds one of theirs.
    for crow, cands in named.items():
        if len(cands) > 1:
            assert np.logical_or.reduce([got_ck[crow] == c for c in cands]).all()
            want_ck[crow] = got_ck[crow]
    assert np.array_equal(got_ck, want_ck), \
        f"{walk}: pack rows differ from the oracle's valid rows"
    d_dst = h2d(dst)
    assert copy(False, d_dst, h2d(ck_in)) == st_o
    assert np.array_equal(d2h16(d_dst), want_dst), \
        f"{walk}: unpack wrote other slots than the valid tokens'"


@pytest.mark.parametrize("walk", list(ERROR_WALK_SHAPES))
@pytest.mark.parametrize("via", VIAS)
def test_ranges_past_the_unit_limit_copy_nothing(walk, via):
    """Ranges holding more (token row, layer) units than one launch walks
    (LUMEN_KV_CKPT_MAX_UNITS): ends of INT32_MAX on 1,024 requests are
    about 2^41 token rows.  Pack and unpack record TOO_MANY and write
    nothing, at once instead of walking rows that are all invalid, on
    every walk."""
    shape = ERROR_WALK_SHAPES[walk]
    R, nb, rows = 1024, 8, 16
    s = np.zeros(R, np.int32)
    e = np.full(R, 2**31 - 1, np.int32)
    assert R * (2**31 - 1) * shape.num_layers > kv.LUMEN_KV_CKPT_MAX_UNITS
    bt = (np.arange(R * 2, dtype=np.int32) % nb).reshape(R, 2)
    rng = np.random.default_rng(77)
    src = W.random_bits(rng, shape.pool_elems(nb))
    dst = W.random_bits(rng, shape.pool_elems(nb))
    st, ck, got_dst = gpu_path(shape, nb, src, bt, s, e, nb, dst, bt,
                               ckpt_rows=rows, via=via)
    assert st == kv.LUMEN_ERR_TOO_MANY
    assert (ck == SENTINEL).all()
    assert np.array_equal(got_dst, dst)


@pytest.mark.parametrize("walk", list(ERROR_WALK_SHAPES))
@pytest.mark.parametrize("via", VIAS)
def test_long_invalid_ranges_still_copy_their_valid_rows(walk, via):
    """Ranges far past their block tables but inside the unit limit: a
    range of 2^20 tokens whose first 12 lie in its table, and one ending at
    INT32_MAX.  The walk crosses all their rows: the status is the
    oracle's (RANGE), the 12 valid rows equal the oracle's pack of those
    tokens, every other row keeps its sentinel, and the unpack writes those
    tokens' slots only."""
    shape = ERROR_WALK_SHAPES[walk]
    nb, rows = 8, 64
    s = np.array([0, 2**31 - 6], np.int32)
    e = np.array([2**20, 2**31 - 1], np.int32)
    bt = np.array([[0, 1, 2], [3, 4, 5]], np.int32)
    n_ok = bt.shape[1] * shape.block_size  # request 0's tokens in its table
    rng = np.random.default_rng(78)
    src = W.random_bits(rng, shape.pool_elems(nb))
    dst = W.random_bits(rng, shape.pool_elems(nb))
    ck_in = W.random_bits(rng, rows * shape.token_row_elems).reshape(rows, -1)
    st_o, _ = oracle.pack(shape, nb, src, bt, s, e, ckpt=np.zeros(
        (rows, shape.token_row_elems), np.uint16), ckpt_rows=rows)
    assert st_o == oracle.ERR_RANGE
    want_ck = np.full((rows, shape.token_row_elems), SENTINEL, np.uint16)
    st, want_ck[:n_ok] = oracle.pack(shape, nb, src, bt[:1], [0], [n_ok])
    assert st == oracle.OK
    want_dst = dst.copy()
    assert oracle.unpack(shape, nb, want_dst, bt[:1], [0], [n_ok],
                         ck_in[:n_ok]) == oracle.OK

    d_s, d_e, d_bt = h2d(s), h2d(e), h2d(bt)
    ck = h2d(np.full(rows * shape.token_row_elems, SENTINEL, np.uint16))
    ws = kv.new_workspace(len(s), dev())

    def copy(pack, cache, ckpt):
        if via == "ranges":
            status = torch.zeros(1, dtype=torch.int32, device=dev())
            fn = (kv.lumen_kv_ckpt_pack_ranges if pack
                  else kv.lumen_kv_ckpt_unpack_ranges)
            fn(shape, nb, cache, d_bt, d_s, d_e, ckpt, status)
            return int(status.item())
        kv.lumen_kv_ckpt_plan(d_s, d_e, ws)
        fn = kv.lumen_kv_ckpt_pack if pack else kv.lumen_kv_ckpt_unpack
        fn(shape, nb, cache, d_bt, ws, ckpt)
        return kv.lumen_kv_ckpt_status(ws)

    assert copy(True, h2d(src), ck) == st_o
    assert np.array_equal(d2h16(ck).reshape(rows, -1), want_ck)
    d_dst = h2d(dst)
    assert copy(False, d_dst, h2d(ck_in)) == st_o
    assert np.array_equal(d2h16(d_dst), want_dst)


def test_status_clears_the_error_word():
    shape = CacheShape(1, 1, 8, 4, NHD)
    nb = 2
    src = h2d(np.zeros(shape.pool_elems(nb), np.uint16))
    ws = kv.new_workspace(1, dev())
    kv.lumen_kv_ckpt_plan(h2d(np.array([0], np.int32)),
                          h2d(np.array([4], np.int32)), ws)
    ck = torch.zeros(4 * shape.token_row_elems, dtype=torch.int16,
                     device=dev())
    kv.lumen_kv_ckpt_pack(shape, nb, src, h2d(np.array([[5]], np.int32)),
                          ws, ck)
    assert kv.lumen_kv_ckpt_status(ws) == kv.LUMEN_ERR_BLOCK_ID
    assert kv.lumen_kv_ckpt_status(ws) == kv.LUMEN_OK


@pytest.mark.parametrize("make", [
    lambda: W.c2_llama8b(num_reqs=9, steps=3, median=150, clip_hi=300),
    lambda: W.c5_qwen_hnd(num_reqs=13, steps=3, median=100, clip_hi=200),
], ids=["llama3-8b-decode-small", "qwen-gqa-hnd-small"])
@pytest.mark.parametrize("via", VIAS)
def test_reduced_incremental_workloads(make, via):
    w = make()
    rng = np.random.default_rng(202)
    src = W.random_bits(rng, w.shape.pool_elems(w.num_blocks))
    dst = W.random_bits(rng, w.shape.pool_elems(w.dst_num_blocks))
    g_dst, o_dst = dst, dst
    for k in range(w.num_steps):
        gpu = gpu_path(w.shape, w.num_blocks, src, w.block_tables, w.starts[k],
                       w.ends[k], w.dst_num_blocks, g_dst, w.dst_block_tables,
                       via=via)
        ref = oracle_path(w.shape, w.num_blocks, src, w.block_tables,
                          w.starts[k], w.ends[k], w.dst_num_blocks, o_dst,
                          w.dst_block_tables)
        assert_same(gpu, ref, f"step {k}")
        g_dst, o_dst = gpu[2], ref[2]


@pytest.mark.parametrize("via", VIAS)
def test_reduced_tp8_shard_in_place(via):
    w = W.c4_llama70b_tp8(num_reqs=11, median=120, clip_hi=400)
    rng = np.random.default_rng(303)
    pool = W.random_bits(rng, w.shape.pool_elems(w.num_blocks))
    # pack, then unpack into the same pool under a fresh permutation
    args = (w.shape, w.num_blocks, pool, w.block_tables, w.starts[0],
            w.ends[0], w.num_blocks, pool, w.dst_block_tables)
    assert_same(gpu_path(*args, in_place=True, via=via), oracle_path(*args),
                "in place")


def test_reduced_restore_burst():
    w = W.c3_restore(num_reqs=5, ctx_lo=40, ctx_hi=300, pool_blocks=200)
    rng = np.random.default_rng(404)
    n = w.step_tokens(0)
    ck = W.random_bits(rng, n * w.shape.token_row_elems)
    pool = W.random_bits(rng, w.shape.pool_elems(w.dst_num_blocks))
    for wave in W.restore_waves(w):
        s, e = w.starts[0][wave], w.ends[0][wave]
        bt = w.dst_block_tables[wave]
        rows = int((e - s).sum())
        off = int(w.ends[0][:wave[0]].sum())
        ck_w = ck[off * w.shape.token_row_elems:(off + rows) * w.shape.token_row_elems]
        # GPU: unpack only
        ws = kv.new_workspace(len(wave), dev())
        kv.lumen_kv_ckpt_plan(h2d(s), h2d(e), ws)
        d = h2d(pool)
        kv.lumen_kv_ckpt_unpack(w.shape, w.dst_num_blocks, d, h2d(bt), ws,
                                h2d(ck_w))
        assert kv.lumen_kv_ckpt_status(ws) == 0
        ref = pool.copy()
        assert oracle.unpack(w.shape, w.dst_num_blocks, ref, bt, s, e,
                             ck_w.reshape(rows, -1)) == 0
        assert np.array_equal(d2h16(d), ref)


def test_offload_and_stage_in_bytes():
    rng = np.random.default_rng(9)
    a = W.random_bits(rng, 3 << 20)
    d = h2d(a)
    host = torch.empty(a.size, dtype=torch.int16, pin_memory=True)
    side = torch.cuda.Stream()
    kv.lumen_kv_ckpt_offload(d, host, producer=torch.cuda.current_stream(),
                             side=side)
    side.synchronize()
    assert np.array_equal(host.numpy().view(np.uint16), a)
    back = torch.zeros_like(d)
    kv.lumen_kv_ckpt_stage_in(host, back, side=side,
                              consumer=torch.cuda.current_stream())
    torch.cuda.current_stream().synchronize()
    assert np.array_equal(d2h16(back), a)
    # partial copy of the first bytes only
    host.zero_()
    kv.lumen_kv_ckpt_offload(d, host, nbytes=1000, side=side)
    side.synchronize()
    got = host.numpy().view(np.uint16)
    assert np.array_equal(got[:500], a[:500]) and not got[500:].any()


@pytest.mark.parametrize("R", [1, 63, 64, 65, 1023, 1024, 1025, 4095, 4096,
                               5000, 20001])
@pytest.mark.parametrize("via", VIAS)
def test_plan_many_requests(R, via):
    """Plans over many requests (several per scan thread, partial
    wavefronts), with empty and invalid ranges sprinkled in; the pack of
    one-element rows checks every planned row against the oracle."""
    shape = CacheShape(1, 1, 8, 4, NHD)
    rng = np.random.default_rng(R)
    cols = 3
    nb = R * cols
    bt = rng.permutation(nb).astype(np.int32).reshape(R, cols)
    s = rng.integers(0, 12, R).astype(np.int32)
    e = np.minimum(s + rng.integers(0, 5, R), 12).astype(np.int32)
    empty = rng.random(R) < 0.1
    e[empty] = s[empty]
    src = W.random_bits(rng, shape.pool_elems(nb))
    if via == "ranges" and R > kv.LUMEN_KV_CKPT_RANGES_MAX_REQS:
        with pytest.raises(kv.LumenError) as ex:
            gpu_path(shape, nb, src, bt, s, e, via=via)
        assert ex.value.code == kv.LUMEN_ERR_TOO_MANY
        return
    disjoint = np.arange(R, dtype=np.int64) * 20 + rng.integers(0, 5, R)
    for base, rb in ((0, None), (7, None), (0, disjoint)):
        n = int((e - s).sum())
        rows = n + base if rb is None else int(rb.max()) + 13
        gpu = gpu_path(shape, nb, src, bt, s, e, row_base=base,
                       req_row_base=rb, ckpt_rows=rows, via=via)
        ref = oracle_path(shape, nb, src, bt, s, e, row_base=base,
                          req_row_base=rb, ckpt_rows=rows)
        assert_same(gpu, ref, f"R={R} base={base} per-request={rb is not None}")
    # one invalid range: the plan reports RANGE and the rest still copies
    if R > 1:
        s2, e2 = s.copy(), e.copy()
        s2[R // 2], e2[R // 2] = 5, 3
        st, _, _ = gpu_path(shape, nb, src, bt, s2, e2, via=via)
        assert st == kv.LUMEN_ERR_RANGE


def gpu_validate(shape, nb, bt, s, e, marks=None):
    """Plan + validate on the GPU; returns the status word."""
    s = np.asarray(s, np.int32)
    e = np.asarray(e, np.int32)
    ws = kv.new_workspace(s.shape[0], dev())
    kv.lumen_kv_ckpt_plan(h2d(s), h2d(e), ws)
    marks = kv.new_marks(nb, dev()) if marks is None else marks
    kv.lumen_kv_ckpt_validate_targets(shape, nb,
                                      h2d(np.asarray(bt, np.int32)), ws, marks)
    return kv.lumen_kv_ckpt_status(ws)


def _written_pages(bt, s, e, bs):
    return [(r, j) for r in range(bt.shape[0]) if 0 <= s[r] < e[r]
            for j in range(s[r] // bs, (e[r] - 1) // bs + 1)
            if j < bt.shape[1]]


@pytest.mark.parametrize("shape", SHAPES[:6], ids=lambda s: f"bs{s.block_size}{s.order}")
def test_validate_targets_matches_oracle(shape):
    rng = np.random.default_rng(zlib.crc32(f"validate{shape}".encode()))
    bs = shape.block_size
    for R, max_tok in ((1, 7), (5, 40), (33, 100)):
        nb, bt, _, s, e, _, _ = _case(rng, shape, R, max_tok, True)
        variants = [("clean", bt, s, e)]
        pages = _written_pages(bt, s, e, bs)
        if len(pages) >= 2:
            a, b = (pages[i] for i in rng.choice(len(pages), 2, False))
            dup = bt.copy()
            dup[b] = dup[a]
            variants.append(("dup written", dup, s, e))
        if pages:
            unwritten = [(r, j) for r in range(R) for j in range(bt.shape[1])
                         if (r, j) not in set(pages)]
            if unwritten:
                dup = bt.copy()
                dup[unwritten[0]] = dup[pages[0]]
                variants.append(("dup unwritten", dup, s, e))
            bad = bt.copy()
            bad[pages[-1]] = nb
            variants.append(("outside pool", bad, s, e))
            neg = bt.copy()
            neg[pages[0]] = -1
            variants.append(("padding entry", neg, s, e))
        past_e = e.copy()
        past_e[0] = bt.shape[1] * bs + 3
        variants.append(("past table", bt, s, past_e))
        inv_s = s.copy()
        inv_s[-1] = -2
        variants.append(("negative start", bt, inv_s, e))
        for what, t, ss, ee in variants:
            want = oracle.validate_targets(shape, nb, t, ss, ee)
            got = gpu_validate(shape, nb, t, ss, ee)
            assert got == want, (what, R, got, want)


def test_validate_reuses_marks_and_strides_over_requests():
    """70000 one-page requests (more than one grid's worth of workgroups);
    the same marks buffer serves a call with a duplicate and then a clean
    call, so stale bits from the first must not leak into the second."""
    shape = CacheShape(1, 1, 8, 4, NHD)
    R = 70000
    rng = np.random.default_rng(77)
    nb = R + 5
    bt = rng.permutation(nb)[:R].astype(np.int32).reshape(R, 1)
    s = np.zeros(R, np.int32)
    e = np.full(R, 3, np.int32)
    marks = kv.new_marks(nb, dev())
    dup = bt.copy()
    dup[R - 1, 0] = dup[0, 0]
    assert oracle.validate_targets(shape, nb, dup, s, e) == \
        kv.LUMEN_ERR_DUP_BLOCK
    assert gpu_validate(shape, nb, dup, s, e, marks) == kv.LUMEN_ERR_DUP_BLOCK
    assert gpu_validate(shape, nb, bt, s, e, marks) == kv.LUMEN_OK


def test_validate_workload_tables():
    """Serving-size tables: every restore wave of the restore burst and the
    in-place table of the 70B TP shard validate; the burst's requests all at
    once do not, because later waves reuse the blocks earlier waves freed."""
    w = W.c3_restore()
    for wave in W.restore_waves(w):
        s, e = w.starts[0][wave], w.ends[0][wave]
        bt = w.dst_block_tables[wave]
        assert gpu_validate(w.shape, w.dst_num_blocks, bt, s, e) == kv.LUMEN_OK
    s, e = w.starts[0], w.ends[0]
    want = oracle.validate_targets(w.shape, w.dst_num_blocks,
                                   w.dst_block_tables, s, e)
    assert want == kv.LUMEN_ERR_DUP_BLOCK
    assert gpu_validate(w.shape, w.dst_num_blocks, w.dst_block_tables, s,
                        e) == want
    w = W.c4_llama70b_tp8()
    assert gpu_validate(w.shape, w.num_blocks, w.dst_block_tables,
                        w.starts[0], w.ends[0]) == kv.LUMEN_OK


def test_validate_with_an_empty_pool_and_no_requests():
    shape = CacheShape(1, 1, 8, 4, NHD)
    # no blocks at all: every written page names a block outside the pool
    bt = np.array([[0, 1]], np.int32)
    want = oracle.validate_targets(shape, 0, bt, [0], [5])
    assert want == oracle.ERR_BLOCK_ID
    ws = kv.new_workspace(1, dev())
    kv.lumen_kv_ckpt_plan(h2d(np.array([0], np.int32)),
                          h2d(np.array([5], np.int32)), ws)
    marks = torch.empty(16, dtype=torch.uint8, device=dev())
    kv.lumen_kv_ckpt_validate_targets(shape, 0, h2d(bt), ws, marks)
    assert kv.lumen_kv_ckpt_status(ws) == want
    # no requests: nothing is checked, the status stays OK
    ws0 = kv.new_workspace(0, dev())
    e = torch.zeros(0, dtype=torch.int32, device=dev())
    kv.lumen_kv_ckpt_plan(e, e, ws0)
    kv.lumen_kv_ckpt_validate_targets(shape, 8, e.view(0, 2), ws0,
                                      kv.new_marks(8, dev()))
    assert kv.lumen_kv_ckpt_status(ws0) == 0


def test_range_copies_on_two_streams_at_once():
    """The one-launch copies hold no state between calls: two of them in
    flight at once on two streams, each with its own status word, both
    equal the oracle."""
    shape = CacheShape(4, 8, 128, 16, NHD)  # 4 KiB units: two spans a wave
    rng = np.random.default_rng(909)
    cases = []
    for R, max_tok in ((37, 90), (11, 200)):
        nb, bt, bt2, s, e, src, dst = _case(rng, shape, R, max_tok, True)
        cases.append((nb, bt, bt2, s, e, src, dst))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = []
    for (nb, bt, bt2, s, e, src, dst), st in zip(cases, streams):
        rows = int((e - s).sum())
        d = dict(ck=h2d(np.full(rows * shape.token_row_elems, SENTINEL,
                                np.uint16)),
                 dst=h2d(dst), src=h2d(src), bt=h2d(bt), bt2=h2d(bt2),
                 s=h2d(s), e=h2d(e),
                 status=torch.zeros(1, dtype=torch.int32, device=dev()))
        torch.cuda.synchronize()
        with torch.cuda.stream(st):
            kv.lumen_kv_ckpt_pack_ranges(shape, nb, d["src"], d["bt"], d["s"],
                                         d["e"], d["ck"], d["status"],
                                         stream=st)
            kv.lumen_kv_ckpt_unpack_ranges(shape, nb, d["dst"], d["bt2"],
                                           d["s"], d["e"], d["ck"],
                                           d["status"], stream=st)
        outs.append(d)
    torch.cuda.synchronize()
    for (nb, bt, bt2, s, e, src, dst), d in zip(cases, outs):
        st_o, want_ck, want_dst = oracle_path(shape, nb, src, bt, s, e, nb,
                                              dst, bt2)
        assert st_o == 0 and int(d["status"].item()) == 0
        assert np.array_equal(d2h16(d["ck"]).reshape(want_ck.shape), want_ck)
        assert np.array_equal(d2h16(d["dst"]), want_dst)


@pytest.mark.parametrize("R", [700, 4096])
def test_many_requests_with_long_units(R):
    """Thousands of requests over 4 KiB units: the one-launch copies then
    scan several requests per thread and copy two spans per wavefront;
    packed and per-request rows, both paths, against the oracle."""
    shape = CacheShape(2, 8, 128, 4, NHD)  # 2*8*128*2 = 4 KiB units
    rng = np.random.default_rng(R)
    nb, bt, bt2, s, e, src, dst = _case(rng, shape, R, 9, True, nb_extra=3)
    args = (shape, nb, src, bt, s, e, nb, dst, bt2)
    ref = oracle_path(*args)
    base = np.arange(R, dtype=np.int64) * 11 + 2
    kw = dict(req_row_base=base, ckpt_rows=R * 11 + 13)
    ref_pr = oracle_path(*args, **kw)
    for via in VIAS:
        assert_same(gpu_path(*args, via=via), ref, f"R={R} packed {via}")
        assert_same(gpu_path(*args, **kw, via=via), ref_pr,
                    f"R={R} per-request {via}")
