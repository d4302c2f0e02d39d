"""Seeded random configurations against the oracle: each draws a cache shape
(layers, heads, head_dim, block size, element width, NHD or HND), a request
count, block tables, token ranges (empty ones included), the plan mode
(packed from a row base, or per-request rows) and a grid size, then checks
pack, unpack, windowed packs, the direct host copy and the one-launch copies
that read the ranges element by element.
One configuration in eight plants an error (a page past the table, or a
block id outside the pool); then only the status is compared, since the GPU
still copies the rows that are fine while the oracle writes nothing."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_17787_amd.kvckpt as kv
from paper_2606_17787_amd import workloads as W
from paper_2606_17787_amd.workloads import CacheShape, HND, NHD

from gpu_util import SENTINEL, d2h_words, dev, h2d

pytestmark = pytest.mark.gpu

WORD = {1: np.uint8, 2: np.uint16, 4: np.uint32}


def draw(seed):
    rng = np.random.default_rng(5000 + seed)
    elem = int(rng.choice([1, 2, 4]))
    D = (16 // elem) * int(rng.integers(1, 9))  # D*elem a multiple of 16
    shape = CacheShape(int(rng.integers(1, 6)), int(rng.integers(1, 7)), D,
                       int(rng.integers(1, 41)),
                       HND if rng.random() < 0.5 else NHD, elem)
    R = int(rng.integers(1, 41))
    cols = int(rng.integers(1, 9))
    nb = R * cols + int(rng.integers(0, 9))
    perm = rng.permutation(nb).astype(np.int32)
    bt = perm[:R * cols].reshape(R, cols).copy()
    bt2 = rng.permutation(nb).astype(np.int32)[:R * cols].reshape(R, cols)
    cap = cols * shape.block_size
    s = rng.integers(0, cap + 1, R).astype(np.int32)
    e = np.minimum(s + rng.integers(0, cap + 1, R), cap).astype(np.int32)
    empty = rng.random(R) < 0.2
    e[empty] = s[empty]
    error = None
    if rng.random() < 0.125 and (e > s).any():
        r = int(np.flatnonzero(e > s)[0])
        if rng.random() < 0.5:
            bt[r, s[r] // shape.block_size] = nb + 3  # BLOCK_ID
            error = "block"
        else:
            e[r] = cap + int(rng.integers(1, 5))      # RANGE: past the table
            error = "range"
    per_request = rng.random() < 0.3
    row_base = int(rng.integers(0, 5))
    waves = int(rng.choice([0, 1, 7, 64]))
    src = W.random_words(rng, shape.pool_elems(nb), elem)
    dst = W.random_words(rng, shape.pool_elems(nb), elem)
    return (rng, shape, R, nb, bt, bt2, s, e, error, per_request, row_base,
            waves, src, dst)


@pytest.mark.parametrize("seed", range(400))
def test_random_configuration_matches_oracle(seed):
    (rng, shape, R, nb, bt, bt2, s, e, error, per_request, row_base, waves,
     src, dst) = draw(seed)
    eb, re_ = shape.elem_bytes, shape.token_row_elems
    n = np.maximum(e.astype(np.int64) - s, 0)
    if per_request:
        base = np.concatenate([[0], np.cumsum(n + 1)[:-1]]) - s + 2
        ck_rows = int((n + 1).sum()) + 2
        kw = dict(req_row_base=base)
    else:
        base = None
        ck_rows = int(n.sum()) + row_base
        kw = dict(row_base=row_base)
    want_ck = np.full((max(ck_rows, 0), re_), SENTINEL, WORD[eb])
    st_o, want_ck = oracle.pack(shape, nb, src, bt, s, e, ckpt=want_ck, **kw)
    want_dst = dst.copy()
    if st_o == oracle.OK:
        assert oracle.unpack(shape, nb, want_dst, bt2, s, e, want_ck,
                             **kw) == oracle.OK
    if error:
        assert st_o != oracle.OK

    d_src, d_bt, d_bt2 = h2d(src), h2d(bt), h2d(bt2)
    d_s, d_e = h2d(s), h2d(e)
    d_base = None if base is None else h2d(base.astype(np.int64))
    ws = kv.new_workspace(R, dev())
    ck = h2d(np.full(max(ck_rows, 1) * re_, SENTINEL, WORD[eb]))
    ck_view = ck[:ck_rows * re_]
    kv.lumen_kv_ckpt_plan(d_s, d_e, ws, 0 if per_request else row_base,
                          d_base)
    kv.lumen_kv_ckpt_pack(shape, nb, d_src, d_bt, ws, ck_view)
    st_g = kv.lumen_kv_ckpt_status(ws)
    assert st_g == st_o, (seed, st_g, st_o)

    # the one-launch pack and unpack that read the ranges themselves
    status = torch.zeros(1, dtype=torch.int32, device=dev())
    ck_r = h2d(np.full(max(ck_rows, 1) * re_, SENTINEL, WORD[eb]))
    kv.lumen_kv_ckpt_pack_ranges(shape, nb, d_src, d_bt, d_s, d_e,
                                 ck_r[:ck_rows * re_], status,
                                 0 if per_request else row_base, d_base)
    assert int(status.item()) == st_o, (seed, "ranges", int(status.item()))
    if st_o != oracle.OK:
        return
    assert np.array_equal(d2h_words(ck_view, eb).reshape(-1, re_), want_ck)
    assert np.array_equal(
        d2h_words(ck_r[:ck_rows * re_], eb).reshape(-1, re_), want_ck)
    d_dst_r = h2d(dst)
    kv.lumen_kv_ckpt_unpack_ranges(shape, nb, d_dst_r, d_bt2, d_s, d_e,
                                   ck_view, status,
                                   0 if per_request else row_base, d_base)
    assert int(status.item()) == 0
    assert np.array_equal(d2h_words(d_dst_r, eb), want_dst)

    # restore into another pool under the second table
    d_dst = h2d(dst)
    kv.lumen_kv_ckpt_plan(d_s, d_e, ws, 0 if per_request else row_base,
                          d_base)
    kv.lumen_kv_ckpt_unpack(shape, nb, d_dst, d_bt2, ws, ck_view)
    assert kv.lumen_kv_ckpt_status(ws) == 0
    assert np.array_equal(d2h_words(d_dst, eb), want_dst)

    # the direct copy into pinned host memory, on a drawn grid size
    host = torch.empty((ck_rows * re_ * eb,), dtype=torch.uint8,
                       pin_memory=True)
    host.numpy().view(WORD[eb])[:] = SENTINEL  # the oracle's untouched rows
    kv.lumen_kv_ckpt_plan(d_s, d_e, ws, 0 if per_request else row_base,
                          d_base)
    kv.lumen_kv_ckpt_pack_to_host_direct(shape, nb, d_src, d_bt, ws, host,
                                         workgroups=waves)
    assert kv.lumen_kv_ckpt_status(ws) == 0
    got = host.numpy().view(WORD[eb]).reshape(-1, re_)
    assert np.array_equal(got, want_ck)

    # windowed packs of random chunk sizes (packed mode: a chunk of packed
    # rows [lo, hi) is the window of checkpoint rows row_base + [lo, hi))
    total = int(n.sum())
    if not per_request and total:
        k = int(rng.integers(1, total + 1))
        kv.lumen_kv_ckpt_plan(d_s, d_e, ws, row_base)
        parts = []
        for lo in range(0, total, k):
            hi = min(lo + k, total)
            win = torch.zeros((hi - lo) * re_, dtype=ck.dtype, device=dev())
            kv.lumen_kv_ckpt_pack_rows(shape, nb, d_src, d_bt, ws, lo, hi,
                                       win, ckpt_first_row=row_base + lo)
            parts.append(win)
        assert kv.lumen_kv_ckpt_status(ws) == 0
        got = np.concatenate([d2h_words(p, eb) for p in parts])
        assert np.array_equal(got.reshape(-1, re_), want_ck[row_base:])


def draw_larger(seed):
    """Serving-sized random shapes (up to 48 layers, 16 KV heads, head_dim
    256, blocks of 64, 300 requests of up to 3,000 tokens), redrawn until
    the pool fits 1.2 GB and the checkpoint 200 MB."""
    rng = np.random.default_rng(9000 + seed)
    while True:
        shape = CacheShape(int(rng.integers(1, 49)), int(rng.integers(1, 17)),
                           int(rng.choice([64, 128, 256])),
                           int(rng.choice([8, 16, 32, 64])),
                           HND if rng.random() < 0.5 else NHD)
        R = int(rng.integers(1, 301))
        ctx = rng.integers(1, 3001, R)
        pages = -(-ctx // shape.block_size)
        nb = int(pages.sum()) + int(rng.integers(0, 50))
        s = np.where(rng.random(R) < 0.5, 0, rng.integers(0, ctx)).astype(np.int32)
        e = np.minimum(s + rng.integers(0, 3001, R), ctx).astype(np.int32)
        rows = int((e - s).sum())
        if (shape.pool_elems(nb) * 2 <= 1.2e9
                and rows * shape.token_row_bytes <= 2e8):
            return rng, shape, R, nb, pages, s, e


@pytest.mark.parametrize("seed", range(12))
def test_larger_random_shape_matches_oracle(seed):
    """Pack and restore of a serving-sized random shape, in the packed or
    the per-request row mode, against the oracle.  At these sizes the copy
    grid's spans cover several units and cross request boundaries, and the
    unit sizes fall on both sides of the grid's 4 KiB threshold."""
    from gpu_util import assert_same, gpu_path, oracle_path
    rng, shape, R, nb, pages, s, e = draw_larger(seed)
    cols = int(pages.max()) + int(rng.integers(0, 3))

    def table():
        perm = rng.permutation(nb).astype(np.int32)
        bt = np.full((R, cols), -1, np.int32)
        o = 0
        for i, p in enumerate(pages):
            bt[i, :p] = perm[o:o + p]
            o += p
        return bt

    bt, bt2 = table(), table()
    src = W.random_bits(rng, shape.pool_elems(nb))
    dst = W.random_bits(rng, shape.pool_elems(nb))
    if rng.random() < 0.3:
        n = (e - s).astype(np.int64)
        kw = dict(req_row_base=np.concatenate([[0], np.cumsum(n + 2)[:-1]])
                  - s + 1, ckpt_rows=int((n + 2).sum()) + 1)
    else:
        kw = dict(row_base=int(rng.integers(0, 5)))
    args = (shape, nb, src, bt, s, e, nb, dst, bt2)
    ref = oracle_path(*args, **kw)
    for via in ("plan", "ranges"):
        assert_same(gpu_path(*args, **kw, via=via), ref,
                    f"seed {seed} via {via}: {shape}, {R} requests")
