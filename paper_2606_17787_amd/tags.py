"""Python binding of the page-tag store (ctypes; argument marshalling only).

Functions and methods map one to one onto include/lumen_page_tags.h, which
states what they compute: tags of complete pages (a BLAKE2b-64 hash of the
page's token IDs paired with its end position) and a store that answers
the longest contiguous checkpointed prefix of a request from its token
history.  The code runs in the shared library; this module raises if the
library has not been built.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional

import numpy as np

from . import kvckpt as _kv

HEADER = os.path.join(os.path.dirname(_kv.HEADER), "lumen_page_tags.h")
TAG_DTYPE = np.dtype([("hash", "<u8"), ("end", "<i8")])


class lumen_page_tag(ctypes.Structure):
    _fields_ = [("hash", ctypes.c_uint64), ("end", ctypes.c_int64)]


def exported_names():
    """Entry points declared in include/lumen_page_tags.h."""
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(lumen_(?:page_tags|tag_store_\w+))\s*\(",
                                 text)))


_BOUND = None


def _lib():
    global _BOUND
    lib = _kv.load_library()
    if _BOUND is lib:
        return lib
    p, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    sigs = {
        "lumen_page_tags": (ctypes.c_int, [p, i64, i32, i64, i64, p]),
        "lumen_tag_store_create": (p, [i32]),
        "lumen_tag_store_destroy": (None, [p]),
        "lumen_tag_store_publish": (ctypes.c_int, [p, i64, i64,
                                                   lumen_page_tag]),
        "lumen_tag_store_publish_pages": (ctypes.c_int,
                                          [p, i64, p, i64, i64, i64]),
        "lumen_tag_store_release": (ctypes.c_int, [p, i64]),
        "lumen_tag_store_longest_prefix": (i64, [p, i64, p, i64]),
        "lumen_tag_store_pages": (i64, [p, i64]),
    }
    for name, (res, args) in sigs.items():
        f = getattr(lib, name)
        f.restype, f.argtypes = res, args
    _BOUND = lib
    return lib


def _tokens(tokens) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(tokens, dtype=np.int32))


def _check(code: int, where: str):
    if code < 0:
        raise _kv.LumenError(int(code), where)


def lumen_page_tags(tokens, block_size: int, page_begin: int = 0,
                    page_end: Optional[int] = None) -> np.ndarray:
    """Tags of complete pages [page_begin, page_end) of a token history, as
    a structured array with fields hash (uint64) and end (int64)."""
    t = _tokens(tokens)
    if page_end is None:
        page_end = t.size // block_size if block_size > 0 else 0
    out = np.zeros(max(page_end - page_begin, 0), TAG_DTYPE)
    _check(_lib().lumen_page_tags(t.ctypes.data, t.size, block_size,
                                  page_begin, page_end, out.ctypes.data),
           "lumen_page_tags")
    return out


class TagStore:
    """lumen_tag_store: per request, the tags of completely received pages."""

    def __init__(self, block_size: int):
        self.block_size = block_size
        self._h = _lib().lumen_tag_store_create(block_size)
        if not self._h:
            raise _kv.LumenError(_kv.LUMEN_ERR_INVALID_ARG,
                                 "lumen_tag_store_create")
        self._destroy = _lib().lumen_tag_store_destroy

    def close(self):
        if getattr(self, "_h", None):
            self._destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()

    def publish(self, request: int, page: int, tag_hash: int, end: int):
        _check(_lib().lumen_tag_store_publish(
            self._h, request, page, lumen_page_tag(tag_hash, end)),
            "lumen_tag_store_publish")

    def publish_pages(self, request: int, tokens, page_begin: int,
                      page_end: int):
        t = _tokens(tokens)
        _check(_lib().lumen_tag_store_publish_pages(
            self._h, request, t.ctypes.data, t.size, page_begin, page_end),
            "lumen_tag_store_publish_pages")

    def release(self, request: int):
        _check(_lib().lumen_tag_store_release(self._h, request),
               "lumen_tag_store_release")

    def longest_prefix(self, request: int, tokens) -> int:
        t = _tokens(tokens)
        n = _lib().lumen_tag_store_longest_prefix(self._h, request,
                                                  t.ctypes.data, t.size)
        _check(n, "lumen_tag_store_longest_prefix")
        return int(n)

    def pages(self, request: int) -> int:
        n = _lib().lumen_tag_store_pages(self._h, request)
        _check(n, "lumen_tag_store_pages")
        return int(n)
