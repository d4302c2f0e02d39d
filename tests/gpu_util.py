"""Helpers shared by the GPU tests: run the HIP path and the CPU oracle on the
same seeded inputs and hand back host copies for element-by-element
comparison."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2606_17787_amd.kvckpt as kv

SENTINEL = 0x5A


def dev():
    return torch.device("cuda:0")


_SIGNED = {np.dtype(np.uint16): np.int16, np.dtype(np.uint32): np.int32}
_WORD = {1: np.uint8, 2: np.uint16, 4: np.uint32}


def h2d(a: np.ndarray) -> torch.Tensor:
    """Host array to a device tensor (unsigned words travel as signed)."""
    a = np.ascontiguousarray(a)
    if a.dtype in _SIGNED:
        a = a.view(_SIGNED[a.dtype])
    return torch.from_numpy(a).to(dev())


def d2h16(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


def d2h_words(t: torch.Tensor, elem_bytes: int) -> np.ndarray:
    return t.cpu().numpy().view(_WORD[elem_bytes])


def gpu_path(shape, nb_src, src_pool, bt, s, e, nb_dst=None, dst_pool=None,
             bt_dst=None, row_base=0, req_row_base=None, ckpt_rows=None,
             in_place=False, via="plan"):
    """Plan + pack (+ unpack) on the GPU.  Returns (status, ckpt, dst_pool)
    as host arrays (dst_pool None when no unpack was asked for).  in_place:
    the unpack writes into the pool the pack read from.  via="plan": the
    plan kernel into a workspace, then the copies over it; via="ranges":
    the one-launch copies that read the ranges themselves."""
    s = np.asarray(s, np.int32)
    e = np.asarray(e, np.int32)
    R = s.shape[0]
    if ckpt_rows is None:
        ckpt_rows = int(np.maximum(e.astype(np.int64) - s, 0).sum()) + row_base
    row_elems = shape.token_row_elems
    eb = shape.elem_bytes
    ck_h = np.full(max(ckpt_rows, 0) * row_elems, SENTINEL, _WORD[eb])
    ck = h2d(ck_h)
    rb = None if req_row_base is None else h2d(np.asarray(req_row_base, np.int64))
    d_s, d_e = h2d(s), h2d(e)
    src = h2d(src_pool)
    d_bt = h2d(np.asarray(bt, np.int32))
    dst = None
    if dst_pool is not None:
        dst = src if in_place else h2d(dst_pool)
        d_bt2 = h2d(np.asarray(bt_dst, np.int32))
    if via == "ranges":
        status = torch.zeros(1, dtype=torch.int32, device=dev())
        kv.lumen_kv_ckpt_pack_ranges(shape, nb_src, src, d_bt, d_s, d_e, ck,
                                     status, row_base, rb)
        if dst is not None:
            kv.lumen_kv_ckpt_unpack_ranges(shape, nb_dst, dst, d_bt2, d_s,
                                           d_e, ck, status, row_base, rb)
        st = int(status.item())
    else:
        assert via == "plan", via
        ws = kv.new_workspace(R, dev())
        kv.lumen_kv_ckpt_plan(d_s, d_e, ws, row_base, rb)
        kv.lumen_kv_ckpt_pack(shape, nb_src, src, d_bt, ws, ck)
        if dst is not None:
            kv.lumen_kv_ckpt_unpack(shape, nb_dst, dst, d_bt2, ws, ck)
        st = kv.lumen_kv_ckpt_status(ws)
    return (st, d2h_words(ck, eb).reshape(-1, row_elems),
            None if dst is None else d2h_words(dst, eb))


def oracle_path(shape, nb_src, src_pool, bt, s, e, nb_dst=None,
                dst_pool=None, bt_dst=None, row_base=0, req_row_base=None,
                ckpt_rows=None):
    s = np.asarray(s, np.int32)
    e = np.asarray(e, np.int32)
    if ckpt_rows is None:
        ckpt_rows = int(np.maximum(e.astype(np.int64) - s, 0).sum()) + row_base
    ck = np.full((ckpt_rows, shape.token_row_elems), SENTINEL,
                 _WORD[shape.elem_bytes])
    st, ck = oracle.pack(shape, nb_src, src_pool, bt, s, e, row_base,
                         req_row_base, ckpt=ck)
    dst = None
    if dst_pool is not None and st == oracle.OK:
        dst = dst_pool.copy()
        st = oracle.unpack(shape, nb_dst, dst, bt_dst, s, e, ck, row_base,
                           req_row_base)
    return st, ck, dst


def assert_same(gpu, ref, what=""):
    st_g, ck_g, dst_g = gpu
    st_o, ck_o, dst_o = ref
    assert st_g == st_o == 0, (what, st_g, st_o)
    if not np.array_equal(ck_g, ck_o):
        bad = np.argwhere(ck_g != ck_o)
        raise AssertionError(f"{what}: checkpoint differs at {len(bad)} "
                             f"elements, first (row, elem) {bad[:4].tolist()}")
    if dst_o is not None:
        if not np.array_equal(dst_g, dst_o):
            bad = np.flatnonzero(dst_g != dst_o)
            raise AssertionError(f"{what}: restored pool differs at "
                                 f"{len(bad)} elements, first {bad[:4]}")
