"""Direct host copies: the gather writing checkpoint rows into pinned host
memory itself, and the scatter reading them from there, against the CPU
oracle element by element (full plans, row windows through interior
pointers of one pinned buffer, several grid sizes, error codes, and a
captured graph)."""
import ctypes
import zlib

import numpy as np
import pytest
import torch

import oracle
import paper_2606_17787_amd.kvckpt as kv
from paper_2606_17787_amd import workloads as W
from paper_2606_17787_amd.workloads import CacheShape, HND, NHD

from gpu_util import d2h_words, dev, h2d

pytestmark = pytest.mark.gpu

SHAPES = [CacheShape(2, 2, 64, 16, NHD), CacheShape(3, 2, 128, 32, HND),
          CacheShape(1, 3, 40, 5, HND), CacheShape(2, 1, 16, 3, NHD, 1),
          CacheShape(2, 2, 8, 4, NHD, 4), CacheShape(4, 1, 128, 16, NHD)]
WORD = {1: np.uint8, 2: np.uint16, 4: np.uint32}


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


def pinned_bytes(n, fill=0x5A):
    t = torch.empty(max(n, 0), dtype=torch.uint8, pin_memory=True)
    t.fill_(fill)
    return t


def pinned(a: np.ndarray) -> torch.Tensor:
    t = torch.empty(a.nbytes, dtype=torch.uint8, pin_memory=True)
    t.numpy()[:] = a.view(np.uint8).reshape(-1)
    return t


def planned(d_s, d_e, R, stream=None):
    ws = kv.new_workspace(R, dev())
    kv.lumen_kv_ckpt_plan(d_s, d_e, ws, stream=stream)
    return ws


@pytest.mark.parametrize("shape", SHAPES,
                         ids=lambda s: f"L{s.num_layers}H{s.num_kv_heads}"
                                       f"bs{s.block_size}{s.order}e{s.elem_bytes}")
@pytest.mark.parametrize("workgroups", [0, 1, 3, 4096])
def test_direct_roundtrip_matches_oracle(shape, workgroups):
    nb, bt, bt2, s, e, src, dst = case(shape, zlib.crc32(repr(shape).encode()),
                                       R=23, max_tok=140)
    total = int((e - s).sum())
    rb = shape.token_row_bytes
    st, want = oracle.pack(shape, nb, src, bt, s, e)
    assert st == 0
    want_dst = dst.copy()
    assert oracle.unpack(shape, nb, want_dst, bt2, s, e, want) == 0
    d_src, d_dst = h2d(src), h2d(dst)
    d_bt, d_bt2, d_s, d_e = h2d(bt), h2d(bt2), h2d(s), h2d(e)
    host = pinned_bytes(total * rb)
    ws = planned(d_s, d_e, len(s))
    kv.lumen_kv_ckpt_pack_to_host_direct(shape, nb, d_src, d_bt, ws, host,
                                         workgroups=workgroups)
    torch.cuda.synchronize()
    assert kv.lumen_kv_ckpt_status(ws) == 0
    got = host.numpy().view(WORD[shape.elem_bytes]).reshape(want.shape)
    assert np.array_equal(got, want)
    # restore from a second pinned buffer holding the oracle's rows
    src_rows = pinned(want)
    ws2 = planned(d_s, d_e, len(s))
    kv.lumen_kv_ckpt_unpack_from_host_direct(shape, nb, d_dst, d_bt2, ws2,
                                             src_rows, workgroups=workgroups)
    torch.cuda.synchronize()
    assert kv.lumen_kv_ckpt_status(ws2) == 0
    assert np.array_equal(d2h_words(d_dst, shape.elem_bytes), want_dst)


@pytest.mark.parametrize("shape", SHAPES[:3],
                         ids=lambda s: f"bs{s.block_size}{s.order}")
def test_direct_windows_through_interior_pointers(shape):
    """Chunks of k packed rows go to host[lo*rb:(lo+k)*rb] as windows
    starting at checkpoint row lo: the device address of each interior
    pointer is the pinned buffer's plus the offset."""
    nb, bt, bt2, s, e, src, dst = case(shape, 77, R=17, max_tok=120)
    total = int((e - s).sum())
    rb = shape.token_row_bytes
    st, want = oracle.pack(shape, nb, src, bt, s, e)
    assert st == 0
    want_dst = dst.copy()
    assert oracle.unpack(shape, nb, want_dst, bt2, s, e, want) == 0
    d_src, d_dst = h2d(src), h2d(dst)
    d_bt, d_bt2, d_s, d_e = h2d(bt), h2d(bt2), h2d(s), h2d(e)
    for k in (1, 7, 64):
        host = pinned_bytes(total * rb + 2 * rb)  # one spare row each end
        ws = planned(d_s, d_e, len(s))
        for lo in range(0, total, k):
            hi = min(lo + k, total)
            view = host[(lo + 1) * rb:(hi + 1) * rb]
            kv.lumen_kv_ckpt_pack_to_host_direct(
                shape, nb, d_src, d_bt, ws, view, row_begin=lo, row_end=hi,
                ckpt_first_row=lo, workgroups=2)
        torch.cuda.synchronize()
        assert kv.lumen_kv_ckpt_status(ws) == 0
        raw = host.numpy()
        assert (raw[:rb] == 0x5A).all() and (raw[-rb:] == 0x5A).all()
        got = raw[rb:-rb].view(WORD[shape.elem_bytes]).reshape(want.shape)
        assert np.array_equal(got, want), k
        # and back, window by window, from the same buffer
        d_out = h2d(dst)
        ws2 = planned(d_s, d_e, len(s))
        for lo in range(0, total, k):
            hi = min(lo + k, total)
            kv.lumen_kv_ckpt_unpack_from_host_direct(
                shape, nb, d_out, d_bt2, ws2,
                host[(lo + 1) * rb:(hi + 1) * rb], row_begin=lo, row_end=hi,
                ckpt_first_row=lo, workgroups=2)
        torch.cuda.synchronize()
        assert kv.lumen_kv_ckpt_status(ws2) == 0
        assert np.array_equal(d2h_words(d_out, shape.elem_bytes),
                              want_dst), k


def test_direct_error_codes_match_oracle():
    """A poisoned block-table entry gives the oracle's BLOCK_ID, a window
    too small gives CAPACITY; rows that are fine are still copied."""
    shape = SHAPES[0]
    nb, bt, _, s, e, src, _ = case(shape, 5, R=9, max_tok=80)
    total = int((e - s).sum())
    rb = shape.token_row_bytes
    r = int(np.argmax(e - s))
    bad = bt.copy()
    bad[r, s[r] // shape.block_size] = nb + 2
    st_o, _ = oracle.pack(shape, nb, src, bad, s, e)
    assert st_o == oracle.ERR_BLOCK_ID
    d_src, d_bad, d_s, d_e = h2d(src), h2d(bad), h2d(s), h2d(e)
    ws = planned(d_s, d_e, len(s))
    host = pinned_bytes(total * rb)  # referenced until the kernel is done
    kv.lumen_kv_ckpt_pack_to_host_direct(shape, nb, d_src, d_bad, ws, host)
    assert kv.lumen_kv_ckpt_status(ws) == kv.LUMEN_ERR_BLOCK_ID
    # window of total-3 rows: the last three rows are CAPACITY errors
    st_c, want = oracle.pack(shape, nb, src, bt, s, e)
    assert st_c == 0
    ws = planned(d_s, d_e, len(s))
    small = pinned_bytes((total - 3) * rb)
    kv.lumen_kv_ckpt_pack_to_host_direct(shape, nb, d_src, h2d(bt), ws, small)
    assert kv.lumen_kv_ckpt_status(ws) == kv.LUMEN_ERR_CAPACITY
    got = small.numpy().view(np.uint16).reshape(total - 3, -1)
    assert np.array_equal(got, want[:total - 3])


def test_direct_refuses_memory_the_device_cannot_reach():
    shape = SHAPES[0]
    nb, bt, _, s, e, src, _ = case(shape, 6, R=4, max_tok=40)
    total = int((e - s).sum())
    rb = shape.token_row_bytes
    d_src, d_bt = h2d(src), h2d(bt)
    ws = planned(h2d(s), h2d(e), len(s))
    torch.cuda.synchronize()
    with pytest.raises(ValueError):  # the binding checks first
        kv.lumen_kv_ckpt_pack_to_host_direct(
            shape, nb, d_src, d_bt, ws, torch.zeros(total * rb,
                                                    dtype=torch.uint8))
    # Straight through the C ABI: pageable memory is refused before
    # anything is enqueued.  The cache pointer is deliberately misaligned,
    # so that a refusal that failed would still stop at the alignment check
    # (MISALIGNED) and never launch a kernel at pageable memory.
    pageable = np.zeros(total * rb + 16, np.uint8)
    addr = (pageable.ctypes.data + 15) & ~15
    lay = kv.layout(shape, nb)
    lib = kv.load_library()
    for f in (lib.lumen_kv_ckpt_pack_to_host_direct,
              lib.lumen_kv_ckpt_unpack_from_host_direct):
        code = f(ctypes.byref(lay), ctypes.c_void_p(d_src.data_ptr() + 2),
                 ctypes.c_void_p(d_bt.data_ptr()), bt.shape[1], len(s),
                 ctypes.c_void_p(ws.data_ptr()), 0, (1 << 63) - 1,
                 ctypes.c_void_p(addr), 0, total, 0, None)
        assert code == kv.LUMEN_ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert kv.lumen_kv_ckpt_status(ws) == 0
    assert not pageable.any()


def test_direct_restore_burst_request():
    """The shortest restore-burst request (about 4K tokens of a
    Llama-3-8B-shaped cache, 0.5 GB) restored straight from pinned host
    memory into its fragmented blocks, against the oracle on a compact pool
    of those blocks."""
    w = W.c3_restore()
    sh = w.shape
    order = np.argsort(w.ctx)[:1]
    s, e = w.starts[0][order], w.ends[0][order]
    bt = w.dst_block_tables[order]
    total = int((e - s).sum())
    rng = np.random.default_rng(32)
    ck = W.random_bits(rng, total * sh.token_row_elems)
    host = pinned(ck)
    used = np.unique(bt[bt >= 0])
    relabel = np.full(w.dst_num_blocks, -1, np.int32)
    relabel[used] = np.arange(used.size, dtype=np.int32)
    bt_c = np.where(bt >= 0, relabel[np.maximum(bt, 0)], -1).astype(np.int32)
    nb = int(used.size)
    pool = W.random_bits(rng, sh.pool_elems(nb))
    want = pool.copy()
    assert oracle.unpack(sh, nb, want, bt_c, s, e, ck.reshape(total, -1)) == 0
    d_pool = h2d(pool)
    ws = planned(h2d(s), h2d(e), 1)
    kv.lumen_kv_ckpt_unpack_from_host_direct(sh, nb, d_pool, h2d(bt_c), ws,
                                             host)
    torch.cuda.synchronize()
    assert kv.lumen_kv_ckpt_status(ws) == 0
    assert np.array_equal(d2h_words(d_pool, 2), want)


def test_direct_copies_captured_in_a_graph():
    """Plan, direct pack to host and direct unpack from host captured once
    and replayed; before each replay the source cache and the destination
    pool are rewritten eagerly, and each replay is checked against the
    oracle on those inputs."""
    shape = SHAPES[1]
    nb, bt, bt2, s, e, src, dst = case(shape, 8, R=11, max_tok=100)
    total = int((e - s).sum())
    rb = shape.token_row_bytes
    d_src, d_dst = h2d(src), h2d(dst)
    d_bt, d_bt2, d_s, d_e = h2d(bt), h2d(bt2), h2d(s), h2d(e)
    host = pinned_bytes(total * rb)
    ws_a, ws_b = kv.new_workspace(len(s), dev()), kv.new_workspace(len(s), dev())

    def step():
        kv.lumen_kv_ckpt_plan(d_s, d_e, ws_a)
        kv.lumen_kv_ckpt_pack_to_host_direct(shape, nb, d_src, d_bt, ws_a,
                                             host)
        kv.lumen_kv_ckpt_plan(d_s, d_e, ws_b)
        kv.lumen_kv_ckpt_unpack_from_host_direct(shape, nb, d_dst, d_bt2,
                                                 ws_b, host)

    step()
    torch.cuda.synchronize()
    assert kv.lumen_kv_ckpt_status(ws_a) == 0
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    rng = np.random.default_rng(9)
    for rep in range(3):
        new_src = W.random_words(rng, shape.pool_elems(nb), 2)
        d_src.copy_(h2d(new_src))
        d_dst.copy_(h2d(dst))
        host.fill_(0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert kv.lumen_kv_ckpt_status(ws_a) == 0
        assert kv.lumen_kv_ckpt_status(ws_b) == 0
        st, want = oracle.pack(shape, nb, new_src, bt, s, e)
        assert st == 0
        want_dst = dst.copy()
        assert oracle.unpack(shape, nb, want_dst, bt2, s, e, want) == 0
        got = host.numpy().view(np.uint16).reshape(want.shape)
        assert np.array_equal(got, want), rep
        assert np.array_equal(d2h_words(d_dst, 2), want_dst), rep
