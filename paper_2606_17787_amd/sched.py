"""Python binding of the placement and recovery scheduler (ctypes; argument
marshalling only).  The decisions are computed by the shared library, as
include/lumen_sched.h specifies: Eq. 1 checkpoint placement with reserved
footprints, recovery dispatch to checkpoint holders, and the average-based
request-count rebalancing."""
from __future__ import annotations

import ctypes
import os
import re
from typing import List, Sequence, Tuple

import numpy as np

from . import kvckpt as _kv

HEADER = os.path.join(os.path.dirname(_kv.HEADER), "lumen_sched.h")


def exported_names():
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(lumen_sched_\w+)\s*\(", text)))


_BOUND = None


def _lib():
    global _BOUND
    lib = _kv.load_library()
    if _BOUND is lib:
        return lib
    p, i32, i64, d = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                      ctypes.c_double)
    sigs = {
        "lumen_sched_create": (p, [i32, p, d, d]),
        "lumen_sched_destroy": (None, [p]),
        "lumen_sched_set_worker": (ctypes.c_int, [p, i32, d, i64, i64]),
        "lumen_sched_place": (ctypes.c_int, [p, i64, i32, i64, p]),
        "lumen_sched_set_persisted": (ctypes.c_int, [p, i64, i64]),
        "lumen_sched_release": (ctypes.c_int, [p, i64]),
        "lumen_sched_holder": (ctypes.c_int, [p, i64, p]),
        "lumen_sched_reserved": (i64, [p, i32]),
        "lumen_sched_recover": (ctypes.c_int, [p, p, i32, p, p, p, i64, p]),
    }
    for name, (res, args) in sigs.items():
        f = getattr(lib, name)
        f.restype, f.argtypes = res, args
    _BOUND = lib
    return lib


def _check(code: int, where: str):
    if code < 0:
        raise _kv.LumenError(int(code), where)


class Scheduler:
    """lumen_sched: placement and recovery decisions for a cluster."""

    def __init__(self, budgets: Sequence[int], h2d_bytes_per_s: float,
                 lam: float = 1.0):
        b = np.ascontiguousarray(np.asarray(budgets, np.int64))
        self.num_workers = int(b.size)
        self._h = _lib().lumen_sched_create(b.size, b.ctypes.data,
                                            float(h2d_bytes_per_s), float(lam))
        if not self._h:
            raise _kv.LumenError(_kv.LUMEN_ERR_INVALID_ARG,
                                 "lumen_sched_create")
        self._requests = set()
        self._destroy = _lib().lumen_sched_destroy

    def close(self):
        if getattr(self, "_h", None):
            self._destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()

    def set_worker(self, w: int, queueing_delay: float, queued: int = 0,
                   running: int = 0):
        c = _lib().lumen_sched_set_worker(self._h, w, float(queueing_delay),
                                          queued, running)
        if c != 0:
            raise _kv.LumenError(c, "lumen_sched_set_worker")

    def place(self, request: int, serving: int, reserved: int) -> int:
        h = ctypes.c_int32(-1)
        c = _lib().lumen_sched_place(self._h, request, serving, reserved,
                                     ctypes.byref(h))
        if c != 0:
            raise _kv.LumenError(c, "lumen_sched_place")
        self._requests.add(request)
        return int(h.value)

    def set_persisted(self, request: int, nbytes: int):
        c = _lib().lumen_sched_set_persisted(self._h, request, nbytes)
        if c != 0:
            raise _kv.LumenError(c, "lumen_sched_set_persisted")

    def release(self, request: int):
        c = _lib().lumen_sched_release(self._h, request)
        if c != 0:
            raise _kv.LumenError(c, "lumen_sched_release")
        self._requests.discard(request)

    def holder(self, request: int) -> int:
        h = ctypes.c_int32(-1)
        c = _lib().lumen_sched_holder(self._h, request, ctypes.byref(h))
        if c != 0:
            raise _kv.LumenError(c, "lumen_sched_holder")
        return int(h.value)

    def reserved(self, w: int) -> int:
        n = _lib().lumen_sched_reserved(self._h, w)
        _check(n, "lumen_sched_reserved")
        return int(n)

    def recover(self, failed: Sequence[int]) -> List[Tuple[int, int, bool]]:
        f = np.ascontiguousarray(np.asarray(failed, np.int32))
        n = max(len(self._requests), 1)
        req = np.zeros(n, np.int64)
        wk = np.zeros(n, np.int32)
        reuse = np.zeros(n, np.int8)
        cnt = ctypes.c_int64(0)
        c = _lib().lumen_sched_recover(self._h, f.ctypes.data, f.size,
                                       req.ctypes.data, wk.ctypes.data,
                                       reuse.ctypes.data, n,
                                       ctypes.byref(cnt))
        if c != 0:
            raise _kv.LumenError(c, "lumen_sched_recover")
        k = int(cnt.value)
        return [(int(req[i]), int(wk[i]), bool(reuse[i])) for i in range(k)]
