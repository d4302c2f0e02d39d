"""Python binding of the checkpoint-progress tracker (ctypes; argument
marshalling only).  include/lumen_progress.h states what it computes: per
request the tokens already handed to the checkpoint pipeline, and for each
batch the ranges [sent, length) still to send."""
from __future__ import annotations

import ctypes
import os
import re
from typing import Sequence, Tuple

import numpy as np

from . import kvckpt as _kv

HEADER = os.path.join(os.path.dirname(_kv.HEADER), "lumen_progress.h")


def exported_names():
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(lumen_progress_\w+)\s*\(", text)))


_BOUND = None


def _lib():
    global _BOUND
    lib = _kv.load_library()
    if _BOUND is lib:
        return lib
    p, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    sigs = {
        "lumen_progress_create": (p, []),
        "lumen_progress_destroy": (None, [p]),
        "lumen_progress_ranges": (ctypes.c_int, [p, p, p, i32, p, p]),
        "lumen_progress_sent": (i64, [p, i64]),
        "lumen_progress_release": (ctypes.c_int, [p, i64]),
    }
    for name, (res, args) in sigs.items():
        f = getattr(lib, name)
        f.restype, f.argtypes = res, args
    _BOUND = lib
    return lib


class Progress:
    """lumen_progress: what each request has already sent."""

    def __init__(self):
        self._h = _lib().lumen_progress_create()
        if not self._h:
            raise MemoryError("lumen_progress_create")
        self._destroy = _lib().lumen_progress_destroy

    def close(self):
        if getattr(self, "_h", None):
            self._destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()

    def ranges(self, ids: Sequence[int],
               lengths: Sequence[int]) -> Tuple[np.ndarray, np.ndarray]:
        i = np.ascontiguousarray(np.asarray(ids, np.int64))
        n = np.ascontiguousarray(np.asarray(lengths, np.int32))
        if i.shape != n.shape:
            raise ValueError("ids and lengths differ in length")
        s = np.zeros(i.size, np.int32)
        e = np.zeros(i.size, np.int32)
        c = _lib().lumen_progress_ranges(self._h, i.ctypes.data, n.ctypes.data,
                                         i.size, s.ctypes.data, e.ctypes.data)
        if c != 0:
            raise _kv.LumenError(c, "lumen_progress_ranges")
        return s, e

    def sent(self, request: int) -> int:
        v = _lib().lumen_progress_sent(self._h, request)
        if v < 0:
            raise _kv.LumenError(int(v), "lumen_progress_sent")
        return int(v)

    def release(self, request: int):
        c = _lib().lumen_progress_release(self._h, request)
        if c != 0:
            raise _kv.LumenError(c, "lumen_progress_release")
