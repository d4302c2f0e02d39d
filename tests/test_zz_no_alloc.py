"""The allocation-free plan + pack (lumen_kv_ckpt_pack_noalloc) against the
existing entry points (lumen_kv_ckpt_plan + lumen_kv_ckpt_pack with a
caller-owned workspace), bit for bit, through the C ABI."""
import numpy as np
import pytest
import torch

import paper_2606_17787_amd.kvckpt as kv
from paper_2606_17787_amd import workloads as W
from paper_2606_17787_amd.workloads import CacheShape, HND, NHD

from gpu_util import SENTINEL, d2h16, dev, h2d

pytestmark = pytest.mark.gpu

SHAPES = [
    CacheShape(2, 2, 64, 16, NHD),   # 256-byte token runs: page-major walk
    CacheShape(4, 8, 128, 16, NHD),  # 2 KiB runs: token-major walk
    CacheShape(3, 4, 128, 32, HND),  # head-major cache
]


def _case(rng, shape, R, max_tok, nb_extra=5):
    bs = shape.block_size
    cols = -(-max_tok // bs) + 1
    nb = R * cols + nb_extra
    bt = rng.permutation(nb).astype(np.int32)[:R * cols].reshape(R, cols)
    s = rng.integers(0, max_tok + 1, R)
    e = np.minimum(s + rng.integers(0, 3 * bs + 2, R), max_tok)
    src = W.random_bits(rng, shape.pool_elems(nb))
    return nb, bt, s.astype(np.int32), e.astype(np.int32), src


def _reference(shape, nb, src, bt, s, e, rows, row_base=0, rb=None):
    """The existing entry points on the same inputs: (status, rows)."""
    ws = kv.new_workspace(len(s), dev())
    ck = h2d(np.full(rows * shape.token_row_elems, SENTINEL, np.uint16))
    kv.lumen_kv_ckpt_plan(h2d(s), h2d(e), ws, row_base,
                          None if rb is None else h2d(rb))
    kv.lumen_kv_ckpt_pack(shape, nb, h2d(src), h2d(bt), ws, ck)
    return kv.lumen_kv_ckpt_status(ws), d2h16(ck)


@pytest.mark.parametrize("shape", SHAPES, ids=["nhd-short", "nhd", "hnd"])
def test_two_calls_in_a_row_match_plan_and_pack(shape):
    """Two allocation-free calls queued back to back on one stream (the
    second with fewer requests and rows, so it reuses a prefix of the
    scratch the first left behind), then one sync: each equals the
    workspace path, and both report OK."""
    rng = np.random.default_rng(31 + shape.num_kv_heads)
    calls = []
    for R, max_tok, row_base in ((40, 120, 0), (7, 50, 3)):
        nb, bt, s, e, src = _case(rng, shape, R, max_tok)
        rows = int((e - s).sum()) + row_base
        d = dict(nb=nb, bt=bt, s=s, e=e, src=src, rows=rows, row_base=row_base,
                 d_src=h2d(src), d_bt=h2d(bt), d_s=h2d(s), d_e=h2d(e),
                 ck=h2d(np.full(rows * shape.token_row_elems, SENTINEL,
                                np.uint16)),
                 st=torch.full((1,), 12345, dtype=torch.int32, device=dev()))
        calls.append(d)
    for d in calls:
        kv.lumen_kv_ckpt_pack_noalloc(shape, d["nb"], d["d_src"], d["d_bt"],
                                      d["d_s"], d["d_e"], d["ck"], d["st"],
                                      row_base=d["row_base"])
    torch.cuda.synchronize()
    for i, d in enumerate(calls):
        st_ref, ck_ref = _reference(shape, d["nb"], d["src"], d["bt"], d["s"],
                                    d["e"], d["rows"], d["row_base"])
        assert st_ref == kv.LUMEN_OK
        assert int(d["st"].item()) == kv.LUMEN_OK, f"call {i}"
        assert np.array_equal(d2h16(d["ck"]), ck_ref), f"call {i} differs"


def test_per_request_rows_and_error_status_match():
    """Per-request row mode, then an input with a block id outside the pool
    and a row past the buffer: the rows and the status equal the workspace
    path's; a later clean call reports OK again."""
    shape = CacheShape(2, 2, 64, 16, NHD)
    rng = np.random.default_rng(77)
    nb, bt, s, e, src = _case(rng, shape, 12, 90)
    base = (np.arange(12, dtype=np.int64) * 100)
    rows = 1200
    st = torch.zeros(1, dtype=torch.int32, device=dev())
    ck = h2d(np.full(rows * shape.token_row_elems, SENTINEL, np.uint16))
    kv.lumen_kv_ckpt_pack_noalloc(shape, nb, h2d(src), h2d(bt), h2d(s),
                                  h2d(e), ck, st, req_row_base=h2d(base))
    st_ref, ck_ref = _reference(shape, nb, src, bt, s, e, rows, 0, base)
    assert int(st.item()) == st_ref == kv.LUMEN_OK
    assert np.array_equal(d2h16(ck), ck_ref)

    bad = bt.copy()
    bad[3, :] = nb + 2  # every page of request 3 outside the pool
    rows = int((e - s).sum()) - 1  # the last row does not fit
    ck = h2d(np.full(rows * shape.token_row_elems, SENTINEL, np.uint16))
    kv.lumen_kv_ckpt_pack_noalloc(shape, nb, h2d(src), h2d(bad), h2d(s),
                                  h2d(e), ck, st)
    st_ref, ck_ref = _reference(shape, nb, src, bad, s, e, rows)
    assert st_ref != kv.LUMEN_OK
    assert int(st.item()) == st_ref
    assert np.array_equal(d2h16(ck), ck_ref)

    ck = h2d(np.full(3 * shape.token_row_elems, SENTINEL, np.uint16))
    one = np.array([0], np.int32), np.array([3], np.int32)
    kv.lumen_kv_ckpt_pack_noalloc(shape, nb, h2d(src), h2d(bt[:1]),
                                  h2d(one[0]), h2d(one[1]), ck, st)
    assert int(st.item()) == kv.LUMEN_OK


def test_limits_and_empty_calls():
    """More requests than the scratch holds is refused before anything is
    enqueued (the status word keeps its value); zero requests report OK."""
    shape = CacheShape(1, 1, 8, 4, NHD)
    R = kv.LUMEN_KV_CKPT_NOALLOC_MAX_REQS + 1
    z = torch.zeros(R, dtype=torch.int32, device=dev())
    bt = torch.zeros((R, 1), dtype=torch.int32, device=dev())
    pool = torch.zeros(shape.pool_elems(1), dtype=torch.int16, device=dev())
    ck = torch.zeros(shape.token_row_elems, dtype=torch.int16, device=dev())
    st = torch.full((1,), 777, dtype=torch.int32, device=dev())
    with pytest.raises(kv.LumenError) as exc:
        kv.lumen_kv_ckpt_pack_noalloc(shape, 1, pool, bt, z, z, ck, st)
    assert exc.value.code == kv.LUMEN_ERR_TOO_MANY
    torch.cuda.synchronize()
    assert int(st.item()) == 777
    e0 = torch.zeros(0, dtype=torch.int32, device=dev())
    kv.lumen_kv_ckpt_pack_noalloc(shape, 1, pool, bt[:0], e0, e0, ck, st)
    assert int(st.item()) == kv.LUMEN_OK
