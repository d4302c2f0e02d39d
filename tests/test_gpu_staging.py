"""Row ranges, checkpoint windows and the host staging pipelines against the
CPU oracle, element by element.

A chunk of packed rows [lo, hi) of a plan is the plan's ranges clipped to
those rows; packed from row_base 0 it fills rows [0, hi - lo), which is the
window [lo, hi) of the checkpoint.  So every chunked call has an exact
oracle counterpart, error codes included."""
import zlib

import numpy as np
import pytest
import torch

import oracle
import paper_2606_17787_amd.kvckpt as kv
from paper_2606_17787_amd import workloads as W
from paper_2606_17787_amd.workloads import CacheShape, HND, NHD

from gpu_util import SENTINEL, d2h_words, dev, h2d

pytestmark = pytest.mark.gpu

SHAPES = [CacheShape(2, 2, 64, 16, NHD), CacheShape(3, 2, 128, 32, HND),
          CacheShape(1, 3, 40, 5, HND), CacheShape(2, 1, 16, 3, NHD, 1),
          CacheShape(2, 2, 8, 4, NHD, 4)]
WORD = {1: np.uint8, 2: np.uint16, 4: np.uint32}


def clip_ranges(s, e, lo, hi):
    """Per-request sub-ranges whose packed rows fall in [lo, hi)."""
    n = np.maximum(e.astype(np.int64) - s, 0)
    first = np.concatenate([[0], np.cumsum(n)[:-1]])
    a = np.clip(lo - first, 0, n)
    b = np.clip(hi - first, 0, n)
    return (s + a).astype(np.int32), (s + b).astype(np.int32)


def case(shape, seed, R=13, max_tok=90):
    rng = np.random.default_rng(seed)
    bs = shape.block_size
    cols = -(-max_tok // bs) + 1
    nb = R * cols + 5
    bt = rng.permutation(nb).astype(np.int32)[:R * cols].reshape(R, cols)
    bt2 = rng.permutation(nb).astype(np.int32)[:R * cols].reshape(R, cols)
    s = rng.integers(0, max_tok, R).astype(np.int32)
    e = np.minimum(s + rng.integers(0, 40, R), max_tok).astype(np.int32)
    empty = rng.random(R) < 0.2
    e[empty] = s[empty]
    src = W.random_words(rng, shape.pool_elems(nb), shape.elem_bytes)
    dst = W.random_words(rng, shape.pool_elems(nb), shape.elem_bytes)
    return nb, bt, bt2, s, e, src, dst


def planned(s, e):
    """Plan on the current stream (the range tensors are freed after the
    call, which is safe only for work on the stream they were made on)."""
    ws = kv.new_workspace(len(s), dev())
    kv.lumen_kv_ckpt_plan(h2d(s), h2d(e), ws)
    return ws


def window(shape, rows):
    w = np.full(max(rows, 0) * shape.token_row_elems, SENTINEL,
                WORD[shape.elem_bytes])
    return h2d(w)


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"bs{s.block_size}{s.order}e{s.elem_bytes}")
def test_pack_rows_chunks(shape):
    nb, bt, _, s, e, src, _ = case(shape, zlib.crc32(repr(shape).encode()))
    total = int((e - s).sum())
    d_src, d_bt = h2d(src), h2d(bt)
    ws = planned(s, e)
    for C in (1, 7, 64, total + 5):
        for lo in range(0, total + 1, C):
            hi = lo + C
            for spare in (0, 2):
                win = window(shape, C + spare)
                kv.lumen_kv_ckpt_pack_rows(shape, nb, d_src, d_bt, ws, lo, hi,
                                           win, ckpt_first_row=lo)
                st = kv.lumen_kv_ckpt_status(ws)
                cs, ce = clip_ranges(s, e, lo, hi)
                want = np.full((C + spare, shape.token_row_elems), SENTINEL,
                               WORD[shape.elem_bytes])
                st_o, want = oracle.pack(shape, nb, src, bt, cs, ce,
                                         ckpt=want)
                assert st == st_o == 0, (C, lo, st, st_o)
                got = d2h_words(win, shape.elem_bytes).reshape(want.shape)
                assert np.array_equal(got, want), (C, lo, spare)


def test_window_too_small_reports_capacity():
    shape = SHAPES[0]
    nb, bt, _, s, e, src, _ = case(shape, 5)
    total = int((e - s).sum())
    assert total > 12
    ws = planned(s, e)
    lo, hi = 3, 12
    win = window(shape, hi - lo - 1)
    kv.lumen_kv_ckpt_pack_rows(shape, nb, h2d(src), h2d(bt), ws, lo, hi, win,
                               ckpt_first_row=lo)
    cs, ce = clip_ranges(s, e, lo, hi)
    st_o, _ = oracle.pack(shape, nb, src, bt, cs, ce,
                          ckpt_rows=hi - lo - 1,
                          ckpt=np.zeros((hi - lo + 4, shape.token_row_elems),
                                        np.uint16))
    assert st_o == oracle.ERR_CAPACITY
    assert kv.lumen_kv_ckpt_status(ws) == kv.LUMEN_ERR_CAPACITY
    # a window that starts past the chunk's rows misses every row
    win = window(shape, 20)
    ws = planned(s, e)
    kv.lumen_kv_ckpt_pack_rows(shape, nb, h2d(src), h2d(bt), ws, lo, hi, win,
                               ckpt_first_row=lo + 1)
    assert kv.lumen_kv_ckpt_status(ws) == kv.LUMEN_ERR_CAPACITY


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"bs{s.block_size}{s.order}e{s.elem_bytes}")
def test_unpack_rows_chunks(shape):
    nb, _, bt2, s, e, _, dst = case(shape, zlib.crc32(repr(shape).encode()) + 1)
    total = int((e - s).sum())
    rng = np.random.default_rng(3)
    ck = W.random_words(rng, total * shape.token_row_elems, shape.elem_bytes)
    want = dst.copy()
    assert oracle.unpack(shape, nb, want, bt2, s, e,
                         ck.reshape(total, -1)) == 0
    for C in (1, 9, total + 1):
        d_dst = h2d(dst)
        ws = planned(s, e)
        re = shape.token_row_elems
        for lo in range(0, total, C):
            hi = min(lo + C, total)
            win = h2d(ck[lo * re:hi * re])
            kv.lumen_kv_ckpt_unpack_rows(shape, nb, d_dst, h2d(bt2), ws, lo,
                                         lo + C, win, ckpt_first_row=lo)
        assert kv.lumen_kv_ckpt_status(ws) == 0
        assert np.array_equal(d2h_words(d_dst, shape.elem_bytes), want), C


def pinned(a: np.ndarray) -> torch.Tensor:
    t = torch.empty(a.nbytes, dtype=torch.uint8, pin_memory=True)
    t.numpy()[:] = a.view(np.uint8).reshape(-1)
    return t


@pytest.mark.parametrize("shape", SHAPES[:3], ids=lambda s: f"bs{s.block_size}{s.order}")
def test_pack_to_host_and_back(shape):
    nb, bt, bt2, s, e, src, dst = case(shape, zlib.crc32(repr(shape).encode()) + 2,
                                       R=29, max_tok=150)
    total = int((e - s).sum())
    rb = shape.token_row_bytes
    st_o, want = oracle.pack(shape, nb, src, bt, s, e)
    assert st_o == 0
    want_dst = dst.copy()
    assert oracle.unpack(shape, nb, want_dst, bt2, s, e, want) == 0
    # every device tensor the side streams read stays referenced until they
    # have drained (the caching allocator knows only the current stream)
    d_src, d_bt, d_bt2 = h2d(src), h2d(bt), h2d(bt2)
    d_s, d_e = h2d(s), h2d(e)
    torch.cuda.synchronize()
    pack_s, copy_s = torch.cuda.Stream(), torch.cuda.Stream()
    for slots, slot_rows in ((1, 5), (2, 1), (2, 17), (3, 40), (2, total + 3)):
        staging = torch.empty(slots * slot_rows * rb, dtype=torch.uint8,
                              device=dev())
        host = torch.zeros(total * rb + 64, dtype=torch.uint8,
                           pin_memory=True)
        ws = kv.new_workspace(len(s), dev())
        torch.cuda.synchronize()
        kv.lumen_kv_ckpt_plan(d_s, d_e, ws, stream=pack_s)
        kv.lumen_kv_ckpt_pack_to_host(shape, nb, d_src, d_bt, ws, total,
                                      staging, slots, host,
                                      pack_stream=pack_s, copy_stream=copy_s)
        copy_s.synchronize()
        assert kv.lumen_kv_ckpt_status(ws, stream=pack_s) == 0
        got = host.numpy()[:total * rb].view(want.dtype).reshape(want.shape)
        assert np.array_equal(got, want), (slots, slot_rows)
        assert not host.numpy()[total * rb:].any()
        # and back from the host copy into another pool
        d_dst = h2d(dst)
        ws2 = kv.new_workspace(len(s), dev())
        torch.cuda.synchronize()
        unpack_s = torch.cuda.Stream()
        kv.lumen_kv_ckpt_plan(d_s, d_e, ws2, stream=unpack_s)
        kv.lumen_kv_ckpt_unpack_from_host(shape, nb, d_dst, d_bt2, ws2,
                                          total, host, staging, slots,
                                          copy_stream=copy_s,
                                          unpack_stream=unpack_s)
        unpack_s.synchronize()
        assert kv.lumen_kv_ckpt_status(ws2, stream=unpack_s) == 0
        assert np.array_equal(d2h_words(d_dst, shape.elem_bytes),
                              want_dst), (slots, slot_rows)


def test_restore_from_host_restore_burst_requests():
    """Two whole requests of the restore-burst workload (4K-32K tokens of a
    Llama-3-8B-shaped cache) restored from pinned host memory into their
    fragmented blocks, against the oracle on a compact pool of those
    blocks."""
    w = W.c3_restore()
    sh = w.shape
    order = np.argsort(w.ctx)[:2]  # the two shortest, about 1 GB together
    s, e = w.starts[0][order], w.ends[0][order]
    bt = w.dst_block_tables[order]
    total = int((e - s).sum())
    rb = sh.token_row_bytes
    rng = np.random.default_rng(31)
    ck = W.random_bits(rng, total * sh.token_row_elems)
    host = pinned(ck)
    # compact pool: only the blocks the two requests own, relabelled
    used = np.unique(bt[bt >= 0])
    relabel = np.full(w.dst_num_blocks, -1, np.int32)
    relabel[used] = np.arange(used.size, dtype=np.int32)
    bt_c = np.where(bt >= 0, relabel[np.maximum(bt, 0)], -1).astype(np.int32)
    nb = int(used.size)
    pool = W.random_bits(rng, sh.pool_elems(nb))
    want = pool.copy()
    assert oracle.unpack(sh, nb, want, bt_c, s, e, ck.reshape(total, -1)) == 0
    d_pool = h2d(pool)
    staging = torch.empty(2 * 2048 * rb, dtype=torch.uint8, device=dev())
    ws = kv.new_workspace(2, dev())
    d_s, d_e, d_bt = h2d(s), h2d(e), h2d(bt_c)
    torch.cuda.synchronize()
    cs, us = torch.cuda.Stream(), torch.cuda.Stream()
    kv.lumen_kv_ckpt_plan(d_s, d_e, ws, stream=us)
    kv.lumen_kv_ckpt_unpack_from_host(sh, nb, d_pool, d_bt, ws, total,
                                      host, staging, 2, copy_stream=cs,
                                      unpack_stream=us)
    us.synchronize()
    assert kv.lumen_kv_ckpt_status(ws, stream=us) == 0
    assert np.array_equal(d2h_words(d_pool, 2), want)


def test_page_tags_drive_the_restore_of_a_cut_stream():
    """Three requests are checkpointed to host memory in one pipeline.  The
    stream is then cut after `cut` rows, which is forced from the host: only
    pages wholly inside the rows received so far are published.  Recovery
    regenerates each request's tags from its token history and restores the
    longest contiguous prefix from host memory.  The tokens after it are
    left for recomputation, and the pool must equal the oracle's restore of
    exactly those prefixes."""
    from oracle import tags as O
    from paper_2606_17787_amd import tags as T
    shape = CacheShape(2, 2, 64, 16, NHD)
    bs = shape.block_size
    rng = np.random.default_rng(77)
    ctx = np.array([70, 33, 91], np.int32)
    R = ctx.size
    cols = -(-int(ctx.max()) // bs)
    nb = R * cols + 3
    bt = rng.permutation(nb).astype(np.int32)[:R * cols].reshape(R, cols)
    bt2 = rng.permutation(nb).astype(np.int32)[:R * cols].reshape(R, cols)
    s = np.zeros(R, np.int32)
    src = W.random_bits(rng, shape.pool_elems(nb))
    dst = W.random_bits(rng, shape.pool_elems(nb))
    hist = [rng.integers(0, 1 << 17, n).astype(np.int32) for n in ctx]
    total = int(ctx.sum())
    first = np.concatenate([[0], np.cumsum(ctx)[:-1]]).astype(np.int64)
    rb = shape.token_row_bytes
    d_src, d_bt, d_bt2 = h2d(src), h2d(bt), h2d(bt2)
    d_s, d_e = h2d(s), h2d(ctx)
    host = torch.zeros(total * rb, dtype=torch.uint8, pin_memory=True)
    staging = torch.empty(2 * 8 * rb, dtype=torch.uint8, device=dev())
    ws = kv.new_workspace(R, dev())
    torch.cuda.synchronize()
    ps, cs = torch.cuda.Stream(), torch.cuda.Stream()
    kv.lumen_kv_ckpt_plan(d_s, d_e, ws, stream=ps)
    kv.lumen_kv_ckpt_pack_to_host(shape, nb, d_src, d_bt, ws, total, staging,
                                  2, host, pack_stream=ps, copy_stream=cs)
    cs.synchronize()
    assert kv.lumen_kv_ckpt_status(ws, stream=ps) == 0
    ck = host.numpy().view(np.uint16).reshape(total, -1)
    for cut in (0, 5, 16, 70, 71, 100, 150, total):
        nat, ora = T.TagStore(bs), O.TagStore(bs)
        for r in range(R):
            got = int(np.clip(cut - first[r], 0, ctx[r]))
            pages = got // bs
            nat.publish_pages(r, hist[r], 0, pages)
            for i, tg in enumerate(O.page_tags(hist[r].tolist(), bs, 0,
                                               pages)):
                ora.publish(r, i, tg)
        want = dst.copy()
        d_dst = h2d(dst)
        for r in range(R):
            e_star = nat.longest_prefix(r, hist[r])
            assert e_star == ora.longest_prefix(r, hist[r].tolist())
            assert e_star == (int(np.clip(cut - first[r], 0, ctx[r])) // bs) * bs
            if e_star == 0:
                continue
            assert oracle.unpack(shape, nb, want, bt2[r:r + 1], [0],
                                 [e_star], ck[first[r]:first[r] + e_star]) == 0
            d_e1 = h2d(np.array([e_star], np.int32))
            d_s1 = h2d(np.array([0], np.int32))
            d_btr = d_bt2[r:r + 1]
            ws1 = kv.new_workspace(1, dev())
            torch.cuda.synchronize()
            us = torch.cuda.Stream()
            kv.lumen_kv_ckpt_plan(d_s1, d_e1, ws1, stream=us)
            kv.lumen_kv_ckpt_unpack_from_host(
                shape, nb, d_dst, d_btr, ws1, e_star,
                host[int(first[r]) * rb:], staging, 2, copy_stream=cs,
                unpack_stream=us)
            us.synchronize()
            assert kv.lumen_kv_ckpt_status(ws1, stream=us) == 0
        assert np.array_equal(d2h_words(d_dst, 2), want), cut


def test_pipeline_and_row_range_errors_match_oracle():
    """A block-table entry outside the pool, seen through a chunked pack,
    the host pipelines and a row-range unpack, reports the oracle's code;
    the other rows are still copied where the code allows."""
    shape = SHAPES[0]
    nb, bt, bt2, s, e, src, dst = case(shape, 99, R=7, max_tok=60)
    total = int((e - s).sum())
    assert total > 10
    # poison a page that some token reads
    r = int(np.argmax(e - s))
    bad = bt.copy()
    bad[r, s[r] // shape.block_size] = nb + 3
    st_o, _ = oracle.pack(shape, nb, src, bad, s, e)
    assert st_o == oracle.ERR_BLOCK_ID
    rb = shape.token_row_bytes
    d_src, d_bad = h2d(src), h2d(bad)
    d_s, d_e = h2d(s), h2d(e)
    torch.cuda.synchronize()
    # chunked pack through windows
    ws = planned(s, e)
    for lo in range(0, total, 9):
        win = window(shape, 9)
        kv.lumen_kv_ckpt_pack_rows(shape, nb, d_src, d_bad, ws, lo, lo + 9,
                                   win, ckpt_first_row=lo)
    assert kv.lumen_kv_ckpt_status(ws) == kv.LUMEN_ERR_BLOCK_ID
    # the pipeline to host memory
    staging = torch.empty(2 * 8 * rb, dtype=torch.uint8, device=dev())
    host = torch.zeros(total * rb, dtype=torch.uint8, pin_memory=True)
    ps, cs = torch.cuda.Stream(), torch.cuda.Stream()
    ws2 = kv.new_workspace(len(s), dev())
    torch.cuda.synchronize()
    kv.lumen_kv_ckpt_plan(d_s, d_e, ws2, stream=ps)
    kv.lumen_kv_ckpt_pack_to_host(shape, nb, d_src, d_bad, ws2, total,
                                  staging, 2, host, pack_stream=ps,
                                  copy_stream=cs)
    cs.synchronize()
    assert kv.lumen_kv_ckpt_status(ws2, stream=ps) == kv.LUMEN_ERR_BLOCK_ID
    # the restore pipeline into a table with the same bad entry
    st_u = oracle.unpack(shape, nb, dst.copy(), bad, s, e,
                         np.zeros((total, shape.token_row_elems), np.uint16))
    assert st_u == oracle.ERR_BLOCK_ID
    d_dst = h2d(dst)
    us = torch.cuda.Stream()
    ws3 = kv.new_workspace(len(s), dev())
    torch.cuda.synchronize()
    kv.lumen_kv_ckpt_plan(d_s, d_e, ws3, stream=us)
    kv.lumen_kv_ckpt_unpack_from_host(shape, nb, d_dst, d_bad, ws3, total,
                                      host, staging, 2, copy_stream=cs,
                                      unpack_stream=us)
    us.synchronize()
    assert kv.lumen_kv_ckpt_status(ws3, stream=us) == kv.LUMEN_ERR_BLOCK_ID


def test_pipeline_rejects_misused_buffers():
    shape = SHAPES[0]
    nb, bt, _, s, e, src, _ = case(shape, 3, R=3, max_tok=30)
    total = int((e - s).sum())
    rb = shape.token_row_bytes
    ws = planned(s, e)
    small_host = torch.zeros(total * rb - 16, dtype=torch.uint8,
                             pin_memory=True)
    staging = torch.empty(2 * 4 * rb, dtype=torch.uint8, device=dev())
    ps, cs = torch.cuda.Stream(), torch.cuda.Stream()
    with pytest.raises(ValueError):   # host copy smaller than the rows
        kv.lumen_kv_ckpt_pack_to_host(shape, nb, h2d(src), h2d(bt), ws,
                                      total, staging, 2, small_host,
                                      pack_stream=ps, copy_stream=cs)
    with pytest.raises(ValueError):   # staging not whole rows per slot
        kv.lumen_kv_ckpt_pack_to_host(
            shape, nb, h2d(src), h2d(bt), ws, total,
            torch.empty(2 * 4 * rb + 16, dtype=torch.uint8, device=dev()),
            2, torch.zeros(total * rb, dtype=torch.uint8, pin_memory=True),
            pack_stream=ps, copy_stream=cs)
    with pytest.raises(ValueError):   # host tensor on the device
        kv.lumen_kv_ckpt_pack_to_host(
            shape, nb, h2d(src), h2d(bt), ws, total, staging, 2,
            torch.zeros(total * rb, dtype=torch.uint8, device=dev()),
            pack_stream=ps, copy_stream=cs)
    with pytest.raises(ValueError):   # a stream left out
        kv.lumen_kv_ckpt_pack_to_host(
            shape, nb, h2d(src), h2d(bt), ws, total, staging, 2,
            torch.zeros(total * rb, dtype=torch.uint8, pin_memory=True),
            pack_stream=ps, copy_stream=None)


def test_back_to_back_pipelines_share_one_ring():
    """Pipeline calls issued one after another on one staging ring, with no
    host synchronisation between them and nothing else ordering them:
    eight checkpoints of different plans to eight host buffers, then three
    restores from host buffers prepared beforehand, on two other streams.
    Each call's first write into the ring waits for the previous call on
    that ring, so every host copy and every restored pool equals the
    oracle's."""
    shape = CacheShape(4, 8, 128, 16, NHD)  # 16 KiB rows
    rb = shape.token_row_bytes
    rng = np.random.default_rng(404)
    R, max_tok, bs = 16, 256, shape.block_size
    cols = max_tok // bs
    nb = R * cols + 9
    bt = rng.permutation(nb).astype(np.int32)[:R * cols].reshape(R, cols)
    bt2 = rng.permutation(nb).astype(np.int32)[:R * cols].reshape(R, cols)
    src = W.random_words(rng, shape.pool_elems(nb), 2)
    dst = W.random_words(rng, shape.pool_elems(nb), 2)
    steps = []
    for _ in range(8):
        s = rng.integers(0, max_tok // 2, R).astype(np.int32)
        e = np.minimum(s + rng.integers(40, 200, R), max_tok).astype(np.int32)
        steps.append((s, e, int((e - s).sum())))
    wants = []
    for s, e, _ in steps:
        st, want = oracle.pack(shape, nb, src, bt, s, e)
        assert st == 0
        wants.append(want)
    restores = (0, 3, 6)
    # everything allocated and filled before the first call
    d_src, d_bt, d_bt2 = h2d(src), h2d(bt), h2d(bt2)
    ranges = [(h2d(s), h2d(e)) for s, e, _ in steps]
    slots, slot_rows = 2, 96  # 3 MiB ring, about 20 chunks per call
    staging = torch.empty(slots * slot_rows * rb, dtype=torch.uint8,
                          device=dev())
    hosts = [torch.zeros(t * rb, dtype=torch.uint8, pin_memory=True)
             for _, _, t in steps]
    wss = [kv.new_workspace(R, dev()) for _ in steps]
    sources = [pinned(wants[k]) for k in restores]
    pools = [h2d(dst) for _ in restores]
    wss_r = [kv.new_workspace(R, dev()) for _ in restores]
    ps, cs = torch.cuda.Stream(), torch.cuda.Stream()
    cs2, us2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    for (d_s, d_e), (_, _, total), host, ws in zip(ranges, steps, hosts, wss):
        kv.lumen_kv_ckpt_plan(d_s, d_e, ws, stream=ps)
        kv.lumen_kv_ckpt_pack_to_host(shape, nb, d_src, d_bt, ws, total,
                                      staging, slots, host, pack_stream=ps,
                                      copy_stream=cs)
    for k, host, d_pool, ws in zip(restores, sources, pools, wss_r):
        kv.lumen_kv_ckpt_plan(ranges[k][0], ranges[k][1], ws, stream=us2)
        kv.lumen_kv_ckpt_unpack_from_host(shape, nb, d_pool, d_bt2, ws,
                                          steps[k][2], host, staging, slots,
                                          copy_stream=cs2, unpack_stream=us2)
    torch.cuda.synchronize()
    for i, (host, want, ws) in enumerate(zip(hosts, wants, wss)):
        assert kv.lumen_kv_ckpt_status(ws, stream=ps) == 0
        got = host.numpy().view(np.uint16).reshape(want.shape)
        assert np.array_equal(got, want), i
    for k, d_pool, ws in zip(restores, pools, wss_r):
        assert kv.lumen_kv_ckpt_status(ws, stream=us2) == 0
        want_dst = dst.copy()
        assert oracle.unpack(shape, nb, want_dst, bt2, steps[k][0],
                             steps[k][1], wants[k]) == 0
        assert np.array_equal(d2h_words(d_pool, 2), want_dst), k


def test_pipelines_from_several_host_threads():
    """Four host threads, each with its own streams, staging ring,
    workspaces and pinned buffers, checkpoint to pinned host memory and
    restore from it (through the staging ring, then directly) three times
    over, at the same time.  The library's per-device state (device info,
    the pipelines' event pool and ring table) is shared by all of them;
    every host copy and restored pool must equal the oracle's."""
    import threading

    shape = CacheShape(3, 2, 64, 16, NHD)
    rb = shape.token_row_bytes
    jobs = []
    for i in range(4):
        nb, bt, bt2, s, e, src, dst = case(shape, 700 + i, R=17, max_tok=120)
        st, want = oracle.pack(shape, nb, src, bt, s, e)
        assert st == 0
        want_dst = dst.copy()
        assert oracle.unpack(shape, nb, want_dst, bt2, s, e, want) == 0
        jobs.append(dict(nb=nb, total=int((e - s).sum()), dst=dst, want=want,
                         want_dst=want_dst, d_src=h2d(src), d_bt=h2d(bt),
                         d_bt2=h2d(bt2), d_s=h2d(s), d_e=h2d(e)))
    torch.cuda.synchronize()
    errors = []

    def worker(i):
        try:
            j = jobs[i]
            nb, total, want = j["nb"], j["total"], j["want"]
            pack_s, copy_s, unpack_s = (torch.cuda.Stream(), torch.cuda.Stream(),
                                        torch.cuda.Stream())
            slots, slot_rows = 2, 7
            staging = torch.empty(slots * slot_rows * rb, dtype=torch.uint8,
                                  device=dev())
            host = torch.zeros(total * rb, dtype=torch.uint8, pin_memory=True)
            ws = kv.new_workspace(j["d_s"].numel(), dev())
            for it in range(3):
                host.zero_()
                torch.cuda.synchronize()
                kv.lumen_kv_ckpt_plan(j["d_s"], j["d_e"], ws, stream=pack_s)
                kv.lumen_kv_ckpt_pack_to_host(
                    shape, nb, j["d_src"], j["d_bt"], ws, total, staging,
                    slots, host, pack_stream=pack_s, copy_stream=copy_s)
                copy_s.synchronize()
                assert kv.lumen_kv_ckpt_status(ws, stream=pack_s) == 0
                got = host.numpy().view(want.dtype).reshape(want.shape)
                assert np.array_equal(got, want), (i, it, "ring pack")
                for direct in (False, True):
                    d_dst = h2d(j["dst"])
                    torch.cuda.synchronize()
                    kv.lumen_kv_ckpt_plan(j["d_s"], j["d_e"], ws,
                                          stream=unpack_s)
                    if direct:
                        kv.lumen_kv_ckpt_unpack_from_host_direct(
                            shape, nb, d_dst, j["d_bt2"], ws, host,
                            stream=unpack_s)
                    else:
                        kv.lumen_kv_ckpt_unpack_from_host(
                            shape, nb, d_dst, j["d_bt2"], ws, total, host,
                            staging, slots, copy_stream=copy_s,
                            unpack_stream=unpack_s)
                    unpack_s.synchronize()
                    assert kv.lumen_kv_ckpt_status(ws, stream=unpack_s) == 0
                    assert np.array_equal(d2h_words(d_dst, shape.elem_bytes),
                                          j["want_dst"]), (i, it, direct)
        except BaseException as ex:  # reported by the main thread
            errors.append((i, repr(ex)))

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=90)
    assert not any(t.is_alive() for t in threads), "a worker did not finish"
    assert not errors, errors
