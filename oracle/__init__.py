"""CPU oracle for the paged-KV checkpoint path (ctypes over plain C).

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import this package.  It shares no code with
the GPU library: the C source here is compiled with gcc into its own shared
object, and nothing here imports the GPU package.

What it computes, and the passages it follows, is stated in lumen_oracle.h:
checkpoint pack gathers the token range [start, end) of every request out of
the paged cache through its block table into token-major checkpoint rows
(LUMEN Sec. 2.1 for pages, Sec. 4.2 for incremental ranges); unpack scatters
checkpoint rows back into the blocks a new block table names (Sec. 4.3,
KV-reuse recovery).  Elements (1, 2 or 4 bytes) are moved as raw bits.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lumen_oracle.c")
_HDR = os.path.join(_HERE, "lumen_oracle.h")
LIB_PATH = os.path.join(_HERE, "liblumen_oracle.so")

OK = 0
ERR_INVALID_ARG = -1
ERR_UNSUPPORTED = -2
ERR_RANGE = -5
ERR_BLOCK_ID = -6
ERR_CAPACITY = -7
ERR_DUP_BLOCK = -8


class _Shape(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32),
                ("block_size", ctypes.c_int32),
                ("num_blocks", ctypes.c_int64),
                ("head_major", ctypes.c_int32),
                ("elem_bytes", ctypes.c_int32)]

_WORD = {1: np.uint8, 2: np.uint16, 4: np.uint32}


def word_dtype(shape):
    """Unsigned integer dtype of one cache element (raw bits)."""
    return _WORD[getattr(shape, "elem_bytes", 2)]


def build(src: str = _SRC, out: str = LIB_PATH, extra_flags=()) -> str:
    """Compile the oracle with gcc (plain C11, -O2) into a shared object."""
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror",
           "-shared", "-fPIC", "-I", _HERE, *extra_flags, src, "-o", out]
    subprocess.run(cmd, check=True)
    return out


def _bind(lib: ctypes.CDLL) -> ctypes.CDLL:
    p = ctypes.c_void_p
    i32, i64 = ctypes.c_int32, ctypes.c_int64
    lib.oracle_plan.restype = ctypes.c_int
    lib.oracle_plan.argtypes = [p, p, i32, i64, p, p, p]
    for name in ("oracle_pack", "oracle_unpack"):
        f = getattr(lib, name)
        f.restype = ctypes.c_int
        f.argtypes = [ctypes.POINTER(_Shape), p, p, i32, p, p, i32, i64, p,
                      p, i64]
    lib.oracle_validate_targets.restype = ctypes.c_int
    lib.oracle_validate_targets.argtypes = [ctypes.POINTER(_Shape), p, i32,
                                            p, p, i32]
    return lib


_LIB: Optional[ctypes.CDLL] = None


def load(path: Optional[str] = None) -> ctypes.CDLL:
    """Load the oracle, building it first if the shared object is missing or
    older than its source."""
    global _LIB
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _LIB is None:
        stale = (not os.path.exists(LIB_PATH)
                 or os.path.getmtime(LIB_PATH) < max(os.path.getmtime(_SRC),
                                                     os.path.getmtime(_HDR)))
        if stale:
            build()
        _LIB = _bind(ctypes.CDLL(LIB_PATH))
    return _LIB


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _shape(shape, num_blocks: int) -> _Shape:
    return _Shape(shape.num_layers, shape.num_kv_heads, shape.head_dim,
                  shape.block_size, int(num_blocks),
                  1 if shape.order == "HND" else 0,
                  getattr(shape, "elem_bytes", 2))


def plan(start, end, row_base: int = 0, req_row_base=None,
         lib: Optional[ctypes.CDLL] = None) -> Tuple[int, np.ndarray, int]:
    """Returns (status, first_row[R], total_rows)."""
    lib = lib or load()
    s, e = _i32(start), _i32(end)
    base = (None if req_row_base is None else
            np.ascontiguousarray(np.asarray(req_row_base, np.int64)))
    first = np.zeros(max(s.shape[0], 1), np.int64)
    total = ctypes.c_int64(0)
    st = lib.oracle_plan(_ptr(s), _ptr(e), s.shape[0], int(row_base),
                         _ptr(base), _ptr(first), ctypes.byref(total))
    return st, first[:s.shape[0]], int(total.value)


def pack(shape, num_blocks: int, cache: np.ndarray, block_tables, start, end,
         row_base: int = 0, req_row_base=None, ckpt: Optional[np.ndarray] = None,
         ckpt_rows: Optional[int] = None,
         lib: Optional[ctypes.CDLL] = None) -> Tuple[int, np.ndarray]:
    """Gather the ranges into checkpoint rows.  `cache` is the flat pool as
    raw element words; returns (status, ckpt) with ckpt of shape
    [rows, row_elems] in the same word type."""
    lib = lib or load()
    word = word_dtype(shape)
    cache = np.ascontiguousarray(cache).view(word).reshape(-1)
    assert cache.size == shape.pool_elems(num_blocks)
    bt = _i32(block_tables)
    assert bt.ndim == 2
    s, e = _i32(start), _i32(end)
    base = (None if req_row_base is None else
            np.ascontiguousarray(np.asarray(req_row_base, np.int64)))
    row_elems = shape.token_row_elems
    if ckpt is None:
        if ckpt_rows is None:
            ckpt_rows = int(np.maximum(e.astype(np.int64) - s, 0).sum()) + \
                max(int(row_base), 0)
        ckpt = np.zeros((ckpt_rows, row_elems), word)
    else:
        assert ckpt.dtype == word and ckpt.flags.c_contiguous
        ckpt_rows = ckpt.size // row_elems if ckpt_rows is None else ckpt_rows
        assert ckpt_rows * row_elems <= ckpt.size
    sh = _shape(shape, num_blocks)
    st = lib.oracle_pack(ctypes.byref(sh), _ptr(cache), _ptr(bt),
                         bt.shape[1], _ptr(s),
                         _ptr(e), s.shape[0], int(row_base), _ptr(base),
                         _ptr(ckpt), int(ckpt_rows))
    return st, ckpt


def unpack(shape, num_blocks: int, cache: np.ndarray, block_tables, start,
           end, ckpt: np.ndarray, row_base: int = 0, req_row_base=None,
           ckpt_rows: Optional[int] = None,
           lib: Optional[ctypes.CDLL] = None) -> int:
    """Scatter checkpoint rows into `cache` (a contiguous array of element
    words that is modified in place).  Returns the status."""
    lib = lib or load()
    word = word_dtype(shape)
    assert cache.dtype == word and cache.flags.c_contiguous
    assert cache.size == shape.pool_elems(num_blocks)
    bt = _i32(block_tables)
    assert bt.ndim == 2
    s, e = _i32(start), _i32(end)
    base = (None if req_row_base is None else
            np.ascontiguousarray(np.asarray(req_row_base, np.int64)))
    ck = np.ascontiguousarray(ckpt).view(word)
    row_elems = shape.token_row_elems
    if ckpt_rows is None:
        ckpt_rows = ck.size // row_elems
    assert ckpt_rows * row_elems <= ck.size
    sh = _shape(shape, num_blocks)
    return lib.oracle_unpack(ctypes.byref(sh), _ptr(cache), _ptr(bt),
                             bt.shape[1], _ptr(s),
                             _ptr(e), s.shape[0], int(row_base), _ptr(base),
                             _ptr(ck), int(ckpt_rows))


def validate_targets(shape, num_blocks: int, block_tables, start, end,
                     lib: Optional[ctypes.CDLL] = None) -> int:
    """Status of the blocks an unpack of [start, end) under `block_tables`
    would write: RANGE / BLOCK_ID for pages past the table or outside the
    pool, DUP_BLOCK when one block is named by two written pages."""
    lib = lib or load()
    bt = _i32(block_tables)
    assert bt.ndim == 2
    s, e = _i32(start), _i32(end)
    assert s.shape == e.shape and bt.shape[0] == s.shape[0]
    sh = _shape(shape, num_blocks)
    return lib.oracle_validate_targets(ctypes.byref(sh), _ptr(bt), bt.shape[1],
                                       _ptr(s), _ptr(e), s.shape[0])
