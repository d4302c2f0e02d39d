"""Python binding of liblumen_kv_ckpt.so (ctypes; argument marshalling only).

Each function has the name of the C entry point it calls and takes torch
tensors for the device buffers; torch provides device memory, pinned host
memory and streams, nothing else.  Every step of the path runs in the HIP
library: if the library has not been built this module raises on first use
rather than falling back to anything else.

Before calling into the library, the binding checks that every tensor is on
the right device, contiguous, of the right dtype and large enough for the
sizes passed, because the C ABI sees only raw pointers.  Host-detected
argument errors of the library raise LumenError; device-detected errors are
returned by lumen_kv_ckpt_status.
"""
from __future__ import annotations

import ctypes
import functools
import os
import re
from typing import Optional

import torch

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "liblumen_kv_ckpt.so")
HEADER = os.path.join(os.path.dirname(PKG), "include", "lumen_kv_ckpt.h")

LUMEN_OK = 0
LUMEN_ERR_INVALID_ARG = -1
LUMEN_ERR_UNSUPPORTED = -2
LUMEN_ERR_MISALIGNED = -3
LUMEN_ERR_HIP = -4
LUMEN_ERR_RANGE = -5
LUMEN_ERR_BLOCK_ID = -6
LUMEN_ERR_CAPACITY = -7
LUMEN_ERR_DUP_BLOCK = -8
LUMEN_ERR_TOO_MANY = -9
LUMEN_KV_CKPT_NOALLOC_MAX_REQS = 16384  # include/lumen_kv_ckpt.h
LUMEN_KV_CKPT_RANGES_MAX_REQS = 4096  # include/lumen_kv_ckpt.h
LUMEN_KV_CKPT_MAX_UNITS = 1 << 40  # include/lumen_kv_ckpt.h
LUMEN_CACHE_NHD = 0
LUMEN_CACHE_HND = 1


class LumenError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {lumen_kv_ckpt_strerror(code)} ({code})")


class lumen_kv_layout(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32),
                ("block_size", ctypes.c_int32),
                ("num_blocks", ctypes.c_int64),
                ("elem_bytes", ctypes.c_int32),
                ("cache_order", ctypes.c_int32)]


def exported_names():
    """Entry points declared in include/lumen_kv_ckpt.h."""
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(lumen_kv_(?:ckpt|draft)_\w+)\s*\(",
                                 text)))


_LIB: Optional[ctypes.CDLL] = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    global _LIB
    if _LIB is not None and path == LIB_PATH:
        return _LIB
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build the HIP library first "
            "(python -m paper_2606_17787_amd.build)")
    lib = ctypes.CDLL(path)
    p, i32, i64, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                       ctypes.c_size_t)
    lay = ctypes.POINTER(lumen_kv_layout)
    sigs = {
        "lumen_kv_ckpt_plan_workspace_bytes": (sz, [i32]),
        "lumen_kv_ckpt_plan": (ctypes.c_int, [p, p, i32, i64, p, p, p]),
        "lumen_kv_ckpt_pack": (ctypes.c_int, [lay, p, p, i32, i32, p, p, i64, p]),
        "lumen_kv_ckpt_unpack": (ctypes.c_int, [lay, p, p, i32, i32, p, p, i64, p]),
        "lumen_kv_ckpt_pack_noalloc": (ctypes.c_int,
                                       [lay, p, p, i32, p, p, i32, i64, p, p,
                                        i64, p, p]),
        "lumen_kv_ckpt_pack_ranges": (ctypes.c_int,
                                      [lay, p, p, i32, p, p, i32, i64, p, p,
                                       i64, p, p]),
        "lumen_kv_ckpt_unpack_ranges": (ctypes.c_int,
                                        [lay, p, p, i32, p, p, i32, i64, p, p,
                                         i64, p, p]),
        "lumen_kv_ckpt_status": (ctypes.c_int, [p, p]),
        "lumen_kv_ckpt_marks_bytes": (sz, [i64]),
        "lumen_kv_draft_align": (ctypes.c_int,
                                 [p, i32, p, p, i32, p, p, p, i32, i32, i32,
                                  p, p, i64, p, p, p]),
        "lumen_kv_ckpt_pack_rows": (ctypes.c_int,
                                    [lay, p, p, i32, i32, p, i64, i64, p, i64,
                                     i64, p]),
        "lumen_kv_ckpt_unpack_rows": (ctypes.c_int,
                                      [lay, p, p, i32, i32, p, i64, i64, p,
                                       i64, i64, p]),
        "lumen_kv_ckpt_pack_to_host": (ctypes.c_int,
                                       [lay, p, p, i32, i32, p, i64, p, i64,
                                        i32, p, p, p]),
        "lumen_kv_ckpt_unpack_from_host": (ctypes.c_int,
                                           [lay, p, p, i32, i32, p, i64, p, p,
                                            i64, i32, p, p]),
        "lumen_kv_ckpt_pack_to_host_direct": (ctypes.c_int,
                                              [lay, p, p, i32, i32, p, i64,
                                               i64, p, i64, i64, i32, p]),
        "lumen_kv_ckpt_unpack_from_host_direct": (ctypes.c_int,
                                                  [lay, p, p, i32, i32, p,
                                                   i64, i64, p, i64, i64,
                                                   i32, p]),
        "lumen_kv_ckpt_validate_targets": (ctypes.c_int,
                                           [lay, p, i32, i32, p, p, sz, p]),
        "lumen_kv_ckpt_strerror": (ctypes.c_char_p, [ctypes.c_int]),
        "lumen_kv_ckpt_time_next_copy": (ctypes.c_int, [p, p]),
        "lumen_kv_ckpt_offload": (ctypes.c_int, [p, p, sz, p, p]),
        "lumen_kv_ckpt_stage_in": (ctypes.c_int, [p, p, sz, p, p]),
    }
    for name, (res, args) in sigs.items():
        f = getattr(lib, name)
        f.restype, f.argtypes = res, args
    if path == LIB_PATH:
        _LIB = lib
    return lib


# ------------------------------------------------------------ marshalling

def layout(shape, num_blocks: int) -> lumen_kv_layout:
    """lumen_kv_layout from a cache shape (num_layers, num_kv_heads,
    head_dim, block_size, order 'NHD'/'HND', elem_bytes)."""
    order = {"NHD": LUMEN_CACHE_NHD, "HND": LUMEN_CACHE_HND}[shape.order]
    return lumen_kv_layout(shape.num_layers, shape.num_kv_heads,
                           shape.head_dim, shape.block_size, int(num_blocks),
                           getattr(shape, "elem_bytes", 2), order)


# Small checkpoints are launch-bound, so the per-call marshalling below is
# kept cheap.
def _stream_handle(stream: Optional[torch.cuda.Stream]):
    if stream is not None:
        return ctypes.c_void_p(stream.cuda_stream)
    # the raw handle of the current stream, without building a Stream object
    return ctypes.c_void_p(torch._C._cuda_getCurrentRawStream(
        torch.cuda.current_device()))


def _required_stream(stream) -> ctypes.c_void_p:
    if not isinstance(stream, torch.cuda.Stream):
        raise ValueError("the staging pipelines need explicit streams "
                         "(torch.cuda.Stream); see their docstrings")
    return ctypes.c_void_p(stream.cuda_stream)


def _dev(t: torch.Tensor, what: str, dtype=None) -> ctypes.c_void_p:
    d = t.get_device()
    if d < 0:
        raise ValueError(f"{what} must be a device tensor")
    if d != torch.cuda.current_device():
        # the library launches on the current device
        raise ValueError(f"{what} is on cuda:{d}, the current device is "
                         f"cuda:{torch.cuda.current_device()}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{what} must be {dtype}, got {t.dtype}")
    return ctypes.c_void_p(t.data_ptr())


def _check(code: int, where: str):
    if code != LUMEN_OK:
        raise LumenError(code, where)


def _row_elems(shape) -> int:
    return shape.num_layers * 2 * shape.num_kv_heads * shape.head_dim


def _elem_bytes(shape) -> int:
    return getattr(shape, "elem_bytes", 2)


def _check_cache(shape, num_blocks: int, cache: torch.Tensor, what: str):
    if cache.element_size() != _elem_bytes(shape):
        raise ValueError(f"{what} must have {_elem_bytes(shape)}-byte "
                         "elements")
    need = (shape.num_layers * 2 * int(num_blocks) * shape.block_size
            * shape.num_kv_heads * shape.head_dim)
    if cache.numel() != need:
        raise ValueError(f"{what} has {cache.numel()} elements, the layout "
                         f"needs {need}")


def _check_tables(block_tables: torch.Tensor, num_reqs: int):
    if block_tables.dim() != 2 or block_tables.shape[0] != num_reqs:
        raise ValueError("block_tables must be [num_reqs, bt_cols]")


# ------------------------------------------------------------- entry points

@functools.lru_cache(maxsize=1024)
def lumen_kv_ckpt_plan_workspace_bytes(num_reqs: int) -> int:
    return int(load_library().lumen_kv_ckpt_plan_workspace_bytes(num_reqs))


def lumen_kv_ckpt_strerror(code: int) -> str:
    return load_library().lumen_kv_ckpt_strerror(code).decode()


def lumen_kv_ckpt_time_next_copy(start_event, stop_event) -> None:
    """Time the next copy kernel this thread launches on two HIP events
    (raw hipEvent_t handles as ints or ctypes pointers, created with timing
    enabled; None for either): `start` takes the time that kernel starts,
    `stop` the time it ends.  Calls that launch no copy kernel leave them
    armed; the launch that uses them clears them."""
    def raw(ev):
        if ev is None:
            return None
        return ev.value if isinstance(ev, ctypes.c_void_p) else int(ev)
    _check(load_library().lumen_kv_ckpt_time_next_copy(raw(start_event),
                                                       raw(stop_event)),
           "lumen_kv_ckpt_time_next_copy")


def new_workspace(num_reqs: int, device=None) -> torch.Tensor:
    """Device workspace of the size a plan over num_reqs requests needs."""
    n = lumen_kv_ckpt_plan_workspace_bytes(num_reqs)
    return torch.zeros(n, dtype=torch.uint8, device=device or "cuda")


def _plan_args(start, end, workspace, row_base, req_row_base):
    R = start.numel()
    if end.numel() != R:
        raise ValueError("start and end differ in length")
    ps = _dev(start, "start", torch.int32)
    pe = _dev(end, "end", torch.int32)
    pw = _dev(workspace, "workspace")
    if workspace.numel() * workspace.element_size() < \
            lumen_kv_ckpt_plan_workspace_bytes(R):
        raise ValueError("workspace too small for this many requests")
    pb = None
    if req_row_base is not None:
        if req_row_base.numel() != R:
            raise ValueError("req_row_base must have one entry per request")
        pb = _dev(req_row_base, "req_row_base", torch.int64)
    return (ps, pe, R, int(row_base), pb, pw)


def lumen_kv_ckpt_plan(start: torch.Tensor, end: torch.Tensor,
                       workspace: torch.Tensor, row_base: int = 0,
                       req_row_base: Optional[torch.Tensor] = None,
                       stream: Optional[torch.cuda.Stream] = None) -> None:
    args = _plan_args(start, end, workspace, row_base, req_row_base)
    _check(load_library().lumen_kv_ckpt_plan(*args, _stream_handle(stream)),
           "lumen_kv_ckpt_plan")


def _copy_args(shape, num_blocks: int, cache: torch.Tensor,
               block_tables: torch.Tensor, workspace: torch.Tensor,
               ckpt: torch.Tensor):
    """(layout struct, argument tuple without the stream) of a pack or
    unpack; the struct must outlive every use of the tuple."""
    R = block_tables.shape[0] if block_tables.dim() == 2 else -1
    _check_tables(block_tables, R)
    _check_cache(shape, num_blocks, cache, "cache")
    if workspace.numel() * workspace.element_size() < \
            lumen_kv_ckpt_plan_workspace_bytes(R):
        raise ValueError("workspace too small for this many requests")
    if (ckpt.element_size() != _elem_bytes(shape)
            or ckpt.numel() % _row_elems(shape)):
        raise ValueError("checkpoint must hold whole rows of "
                         f"{_elem_bytes(shape)}-byte elements")
    rows = ckpt.numel() // _row_elems(shape)
    lay = layout(shape, num_blocks)
    return lay, (ctypes.byref(lay), _dev(cache, "cache"),
                 _dev(block_tables, "block_tables", torch.int32),
                 block_tables.shape[1], R, _dev(workspace, "workspace"),
                 _dev(ckpt, "ckpt"), rows)


def _copy(name: str, shape, num_blocks: int, cache: torch.Tensor,
          block_tables: torch.Tensor, workspace: torch.Tensor,
          ckpt: torch.Tensor, stream):
    lay, args = _copy_args(shape, num_blocks, cache, block_tables, workspace,
                           ckpt)
    _check(getattr(load_library(), name)(*args, _stream_handle(stream)), name)


class PreparedCall:
    """One entry point with its arguments checked and marshalled once.

    A serving loop issues the same plan, pack and unpack on the same
    buffers every step (the token ranges are device tensors it rewrites in
    place), and for small checkpoints the per-call checks cost as much as
    the launch.  Calling the object enqueues the entry point on `stream` or
    the current stream, with no checks but the device's.  It keeps the
    tensors alive; they must keep their storage (no resize or reallocation)
    for as long as the object is used."""
    __slots__ = ("_fn", "_args", "_name", "_device", "_keep")

    def __init__(self, name: str, args: tuple, keep: tuple):
        self._fn = getattr(load_library(), name)
        self._args = args
        self._name = name
        self._device = torch.cuda.current_device()
        self._keep = keep

    def __call__(self, stream: Optional[torch.cuda.Stream] = None) -> None:
        if torch.cuda.current_device() != self._device:
            raise ValueError(f"{self._name} was prepared on "
                             f"cuda:{self._device}; the current device is "
                             f"cuda:{torch.cuda.current_device()}")
        h = (stream.cuda_stream if stream is not None else
             torch._C._cuda_getCurrentRawStream(self._device))
        _check(self._fn(*self._args, ctypes.c_void_p(h)), self._name)


def prepare_plan(start: torch.Tensor, end: torch.Tensor,
                 workspace: torch.Tensor, row_base: int = 0,
                 req_row_base: Optional[torch.Tensor] = None) -> PreparedCall:
    """lumen_kv_ckpt_plan with its arguments checked once; see PreparedCall."""
    return PreparedCall("lumen_kv_ckpt_plan",
                        _plan_args(start, end, workspace, row_base,
                                   req_row_base),
                        (start, end, workspace, req_row_base))


def prepare_pack(shape, num_blocks: int, cache: torch.Tensor,
                 block_tables: torch.Tensor, workspace: torch.Tensor,
                 ckpt: torch.Tensor) -> PreparedCall:
    """lumen_kv_ckpt_pack with its arguments checked once; see PreparedCall."""
    lay, args = _copy_args(shape, num_blocks, cache, block_tables, workspace,
                           ckpt)
    return PreparedCall("lumen_kv_ckpt_pack", args,
                        (lay, cache, block_tables, workspace, ckpt))


def prepare_unpack(shape, num_blocks: int, cache: torch.Tensor,
                   block_tables: torch.Tensor, workspace: torch.Tensor,
                   ckpt: torch.Tensor) -> PreparedCall:
    """lumen_kv_ckpt_unpack with its arguments checked once; see
    PreparedCall."""
    lay, args = _copy_args(shape, num_blocks, cache, block_tables, workspace,
                           ckpt)
    return PreparedCall("lumen_kv_ckpt_unpack", args,
                        (lay, cache, block_tables, workspace, ckpt))


def lumen_kv_ckpt_pack(shape, num_blocks: int, cache: torch.Tensor,
                       block_tables: torch.Tensor, workspace: torch.Tensor,
                       ckpt: torch.Tensor,
                       stream: Optional[torch.cuda.Stream] = None) -> None:
    """Gather the planned token ranges of `cache` into `ckpt` rows
    ([rows, L*2*H*D] elements of elem_bytes bytes; rows =
    ckpt.numel() // row_elems)."""
    _copy("lumen_kv_ckpt_pack", shape, num_blocks, cache, block_tables,
          workspace, ckpt, stream)


def _ranges_args(shape, num_blocks: int, cache: torch.Tensor,
                 block_tables: torch.Tensor, start: torch.Tensor,
                 end: torch.Tensor, ckpt: torch.Tensor, status: torch.Tensor,
                 row_base: int, req_row_base: Optional[torch.Tensor]):
    """(layout struct, argument tuple without the stream) of the calls that
    take the ranges instead of a workspace; the struct must outlive every
    use of the tuple."""
    R = start.numel()
    if end.numel() != R:
        raise ValueError("start and end differ in length")
    _check_tables(block_tables, R)
    _check_cache(shape, num_blocks, cache, "cache")
    if (ckpt.element_size() != _elem_bytes(shape)
            or ckpt.numel() % _row_elems(shape)):
        raise ValueError("checkpoint must hold whole rows of "
                         f"{_elem_bytes(shape)}-byte elements")
    if status.numel() != 1:
        raise ValueError("status must be one int32 element")
    pb = None
    if req_row_base is not None:
        if req_row_base.numel() != R:
            raise ValueError("req_row_base must have one entry per request")
        pb = _dev(req_row_base, "req_row_base", torch.int64)
    lay = layout(shape, num_blocks)
    return lay, (ctypes.byref(lay), _dev(cache, "cache"),
                 _dev(block_tables, "block_tables", torch.int32),
                 block_tables.shape[1], _dev(start, "start", torch.int32),
                 _dev(end, "end", torch.int32), R, int(row_base), pb,
                 _dev(ckpt, "ckpt"), ckpt.numel() // _row_elems(shape),
                 _dev(status, "status", torch.int32))


def _ranges_call(name: str, shape, num_blocks: int, cache: torch.Tensor,
                 block_tables: torch.Tensor, start: torch.Tensor,
                 end: torch.Tensor, ckpt: torch.Tensor, status: torch.Tensor,
                 row_base: int, req_row_base: Optional[torch.Tensor],
                 stream: Optional[torch.cuda.Stream]) -> None:
    """Marshals the calls that take the ranges instead of a workspace."""
    lay, args = _ranges_args(shape, num_blocks, cache, block_tables, start,
                             end, ckpt, status, row_base, req_row_base)
    _check(getattr(load_library(), name)(*args, _stream_handle(stream)), name)


def prepare_pack_ranges(shape, num_blocks: int, cache: torch.Tensor,
                        block_tables: torch.Tensor, start: torch.Tensor,
                        end: torch.Tensor, ckpt: torch.Tensor,
                        status: torch.Tensor, row_base: int = 0,
                        req_row_base: Optional[torch.Tensor] = None
                        ) -> PreparedCall:
    """lumen_kv_ckpt_pack_ranges with its arguments checked once; see
    PreparedCall."""
    lay, args = _ranges_args(shape, num_blocks, cache, block_tables, start,
                             end, ckpt, status, row_base, req_row_base)
    return PreparedCall("lumen_kv_ckpt_pack_ranges", args,
                        (lay, cache, block_tables, start, end, ckpt, status,
                         req_row_base))


def prepare_unpack_ranges(shape, num_blocks: int, cache: torch.Tensor,
                          block_tables: torch.Tensor, start: torch.Tensor,
                          end: torch.Tensor, ckpt: torch.Tensor,
                          status: torch.Tensor, row_base: int = 0,
                          req_row_base: Optional[torch.Tensor] = None
                          ) -> PreparedCall:
    """lumen_kv_ckpt_unpack_ranges with its arguments checked once; see
    PreparedCall."""
    lay, args = _ranges_args(shape, num_blocks, cache, block_tables, start,
                             end, ckpt, status, row_base, req_row_base)
    return PreparedCall("lumen_kv_ckpt_unpack_ranges", args,
                        (lay, cache, block_tables, start, end, ckpt, status,
                         req_row_base))


def lumen_kv_ckpt_pack_noalloc(shape, num_blocks: int, cache: torch.Tensor,
                               block_tables: torch.Tensor,
                               start: torch.Tensor, end: torch.Tensor,
                               ckpt: torch.Tensor, status: torch.Tensor,
                               row_base: int = 0,
                               req_row_base: Optional[torch.Tensor] = None,
                               stream: Optional[torch.cuda.Stream] = None
                               ) -> None:
    """Plan + pack with the library's own device scratch instead of a
    workspace (for callers that cannot allocate).  `status` is a device
    int32 tensor of one element that receives the call's status once the
    stream has passed it."""
    _ranges_call("lumen_kv_ckpt_pack_noalloc", shape, num_blocks, cache,
                 block_tables, start, end, ckpt, status, row_base,
                 req_row_base, stream)


def lumen_kv_ckpt_pack_ranges(shape, num_blocks: int, cache: torch.Tensor,
                              block_tables: torch.Tensor, start: torch.Tensor,
                              end: torch.Tensor, ckpt: torch.Tensor,
                              status: torch.Tensor, row_base: int = 0,
                              req_row_base: Optional[torch.Tensor] = None,
                              stream: Optional[torch.cuda.Stream] = None
                              ) -> None:
    """Plan and pack in one launch, straight from the ranges.  `status` is
    a device int32 tensor of one element that the call only lowers to the
    most negative status it records: set it to 0 (LUMEN_OK) first."""
    _ranges_call("lumen_kv_ckpt_pack_ranges", shape, num_blocks, cache,
                 block_tables, start, end, ckpt, status, row_base,
                 req_row_base, stream)


def lumen_kv_ckpt_unpack_ranges(shape, num_blocks: int, cache: torch.Tensor,
                                block_tables: torch.Tensor,
                                start: torch.Tensor, end: torch.Tensor,
                                ckpt: torch.Tensor, status: torch.Tensor,
                                row_base: int = 0,
                                req_row_base: Optional[torch.Tensor] = None,
                                stream: Optional[torch.cuda.Stream] = None
                                ) -> None:
    """Plan and unpack in one launch: the inverse of
    lumen_kv_ckpt_pack_ranges, with the same status rule."""
    _ranges_call("lumen_kv_ckpt_unpack_ranges", shape, num_blocks, cache,
                 block_tables, start, end, ckpt, status, row_base,
                 req_row_base, stream)


def lumen_kv_ckpt_unpack(shape, num_blocks: int, cache: torch.Tensor,
                         block_tables: torch.Tensor, workspace: torch.Tensor,
                         ckpt: torch.Tensor,
                         stream: Optional[torch.cuda.Stream] = None) -> None:
    """Scatter the planned checkpoint rows of `ckpt` into `cache`."""
    _copy("lumen_kv_ckpt_unpack", shape, num_blocks, cache, block_tables,
          workspace, ckpt, stream)


def _rows_call(name: str, shape, num_blocks: int, cache: torch.Tensor,
               block_tables: torch.Tensor, workspace: torch.Tensor,
               row_begin: int, row_end: int, ckpt: torch.Tensor,
               ckpt_first_row: int, stream):
    R = block_tables.shape[0] if block_tables.dim() == 2 else -1
    _check_tables(block_tables, R)
    _check_cache(shape, num_blocks, cache, "cache")
    if workspace.numel() * workspace.element_size() < \
            lumen_kv_ckpt_plan_workspace_bytes(R):
        raise ValueError("workspace too small for this many requests")
    if (ckpt.element_size() != _elem_bytes(shape)
            or ckpt.numel() % _row_elems(shape)):
        raise ValueError("checkpoint window must hold whole rows of "
                         f"{_elem_bytes(shape)}-byte elements")
    rows = ckpt.numel() // _row_elems(shape)
    lay = layout(shape, num_blocks)
    _check(getattr(load_library(), name)(
        ctypes.byref(lay), _dev(cache, "cache"),
        _dev(block_tables, "block_tables", torch.int32),
        block_tables.shape[1], R, _dev(workspace, "workspace"),
        int(row_begin), int(row_end), _dev(ckpt, "ckpt"),
        int(ckpt_first_row), rows, _stream_handle(stream)), name)


INT64_MAX = (1 << 63) - 1


def lumen_kv_ckpt_pack_rows(shape, num_blocks: int, cache: torch.Tensor,
                            block_tables: torch.Tensor,
                            workspace: torch.Tensor, row_begin: int,
                            row_end: int, ckpt: torch.Tensor,
                            ckpt_first_row: int = 0,
                            stream: Optional[torch.cuda.Stream] = None):
    """Pack the plan's packed rows [row_begin, row_end) into `ckpt`, a window
    holding checkpoint rows [ckpt_first_row, ckpt_first_row + rows)."""
    _rows_call("lumen_kv_ckpt_pack_rows", shape, num_blocks, cache,
               block_tables, workspace, row_begin, row_end, ckpt,
               ckpt_first_row, stream)


def lumen_kv_ckpt_unpack_rows(shape, num_blocks: int, cache: torch.Tensor,
                              block_tables: torch.Tensor,
                              workspace: torch.Tensor, row_begin: int,
                              row_end: int, ckpt: torch.Tensor,
                              ckpt_first_row: int = 0,
                              stream: Optional[torch.cuda.Stream] = None):
    """Unpack the plan's packed rows [row_begin, row_end) from the window."""
    _rows_call("lumen_kv_ckpt_unpack_rows", shape, num_blocks, cache,
               block_tables, workspace, row_begin, row_end, ckpt,
               ckpt_first_row, stream)


def _direct_call(name: str, shape, num_blocks: int, cache: torch.Tensor,
                 block_tables: torch.Tensor, workspace: torch.Tensor,
                 host: torch.Tensor, row_begin: int, row_end: int,
                 ckpt_first_row: int, workgroups: int, stream):
    R = block_tables.shape[0] if block_tables.dim() == 2 else -1
    _check_tables(block_tables, R)
    _check_cache(shape, num_blocks, cache, "cache")
    if workspace.numel() * workspace.element_size() < \
            lumen_kv_ckpt_plan_workspace_bytes(R):
        raise ValueError("workspace too small for this many requests")
    if host.is_cuda or not host.is_contiguous():
        raise ValueError("host checkpoint must be a contiguous host tensor")
    if host.numel() and not host.is_pinned():
        raise ValueError("host checkpoint must be pinned (pin_memory=True)")
    rb = _row_elems(shape) * _elem_bytes(shape)
    if _nbytes(host) % rb:
        raise ValueError("host checkpoint must hold whole rows")
    rows = _nbytes(host) // rb
    lay = layout(shape, num_blocks)
    _check(getattr(load_library(), name)(
        ctypes.byref(lay), _dev(cache, "cache"),
        _dev(block_tables, "block_tables", torch.int32),
        block_tables.shape[1], R, _dev(workspace, "workspace"),
        int(row_begin), int(row_end),
        ctypes.c_void_p(host.data_ptr() if host.numel() else None),
        int(ckpt_first_row), rows, int(workgroups), _stream_handle(stream)),
        name)


def lumen_kv_ckpt_pack_to_host_direct(shape, num_blocks: int,
                                      cache: torch.Tensor,
                                      block_tables: torch.Tensor,
                                      workspace: torch.Tensor,
                                      host: torch.Tensor, row_begin: int = 0,
                                      row_end: int = None,
                                      ckpt_first_row: int = 0,
                                      workgroups: int = 0,
                                      stream: Optional[torch.cuda.Stream] = None):
    """Pack the plan's packed rows [row_begin, row_end) straight into the
    pinned host tensor `host`, a window holding checkpoint rows
    [ckpt_first_row, ckpt_first_row + rows), on a grid of `workgroups`
    workgroups (0: the library's default)."""
    _direct_call("lumen_kv_ckpt_pack_to_host_direct", shape, num_blocks,
                 cache, block_tables, workspace, host, row_begin,
                 INT64_MAX if row_end is None else row_end, ckpt_first_row,
                 workgroups, stream)


def lumen_kv_ckpt_unpack_from_host_direct(shape, num_blocks: int,
                                          cache: torch.Tensor,
                                          block_tables: torch.Tensor,
                                          workspace: torch.Tensor,
                                          host: torch.Tensor,
                                          row_begin: int = 0,
                                          row_end: int = None,
                                          ckpt_first_row: int = 0,
                                          workgroups: int = 0,
                                          stream: Optional[torch.cuda.Stream] = None):
    """Unpack the plan's packed rows [row_begin, row_end) straight from the
    pinned host tensor `host` (the window, as for the pack)."""
    _direct_call("lumen_kv_ckpt_unpack_from_host_direct", shape, num_blocks,
                 cache, block_tables, workspace, host, row_begin,
                 INT64_MAX if row_end is None else row_end, ckpt_first_row,
                 workgroups, stream)


def _pipeline_args(shape, num_blocks, cache, block_tables, workspace,
                   total_rows, staging, slots, host):
    R = block_tables.shape[0] if block_tables.dim() == 2 else -1
    _check_tables(block_tables, R)
    _check_cache(shape, num_blocks, cache, "cache")
    if workspace.numel() * workspace.element_size() < \
            lumen_kv_ckpt_plan_workspace_bytes(R):
        raise ValueError("workspace too small for this many requests")
    rb = _row_elems(shape) * _elem_bytes(shape)
    if host.is_cuda or not host.is_contiguous():
        raise ValueError("host checkpoint must be a contiguous host tensor")
    if _nbytes(host) < int(total_rows) * rb:
        raise ValueError("host checkpoint smaller than total_rows rows")
    if slots < 1 or _nbytes(staging) % (slots * rb):
        raise ValueError("staging must hold `slots` slots of whole rows")
    slot_rows = _nbytes(staging) // (slots * rb)
    if slot_rows < 1:
        raise ValueError("staging holds no row per slot")
    return R, slot_rows


def lumen_kv_ckpt_pack_to_host(shape, num_blocks: int, cache: torch.Tensor,
                               block_tables: torch.Tensor,
                               workspace: torch.Tensor, total_rows: int,
                               staging: torch.Tensor, slots: int,
                               host: torch.Tensor, *,
                               pack_stream: torch.cuda.Stream,
                               copy_stream: torch.cuda.Stream):
    """Pack the planned rows through a device staging ring of `slots` equal
    slots (`staging` is split evenly) into host tensor `host` (pinned).
    Both streams are required: for the checkpoint to overlap serving they
    must differ from the serving stream (passing the serving stream, e.g.
    torch.cuda.current_stream(), runs the pipeline serially on it)."""
    R, slot_rows = _pipeline_args(shape, num_blocks, cache, block_tables,
                                  workspace, total_rows, staging, slots, host)
    lay = layout(shape, num_blocks)
    _check(load_library().lumen_kv_ckpt_pack_to_host(
        ctypes.byref(lay), _dev(cache, "cache"),
        _dev(block_tables, "block_tables", torch.int32),
        block_tables.shape[1], R, _dev(workspace, "workspace"),
        int(total_rows), _dev(staging, "staging"), slot_rows, int(slots),
        ctypes.c_void_p(host.data_ptr()), _required_stream(pack_stream),
        _required_stream(copy_stream)), "lumen_kv_ckpt_pack_to_host")


def lumen_kv_ckpt_unpack_from_host(shape, num_blocks: int,
                                   cache: torch.Tensor,
                                   block_tables: torch.Tensor,
                                   workspace: torch.Tensor, total_rows: int,
                                   host: torch.Tensor, staging: torch.Tensor,
                                   slots: int, *,
                                   copy_stream: torch.cuda.Stream,
                                   unpack_stream: torch.cuda.Stream):
    """Restore the planned rows from host tensor `host` through the staging
    ring into `cache`.  Both streams are required, as for
    lumen_kv_ckpt_pack_to_host."""
    R, slot_rows = _pipeline_args(shape, num_blocks, cache, block_tables,
                                  workspace, total_rows, staging, slots, host)
    lay = layout(shape, num_blocks)
    _check(load_library().lumen_kv_ckpt_unpack_from_host(
        ctypes.byref(lay), _dev(cache, "cache"),
        _dev(block_tables, "block_tables", torch.int32),
        block_tables.shape[1], R, _dev(workspace, "workspace"),
        int(total_rows), ctypes.c_void_p(host.data_ptr()),
        _dev(staging, "staging"), slot_rows, int(slots),
        _required_stream(copy_stream), _required_stream(unpack_stream)),
        "lumen_kv_ckpt_unpack_from_host")


def lumen_kv_draft_align(draft: torch.Tensor, draft_len: torch.Tensor,
                         committed: torch.Tensor,
                         committed_len: torch.Tensor, kv_len: torch.Tensor,
                         block_tables: torch.Tensor, block_size: int,
                         replay: torch.Tensor, freed: torch.Tensor,
                         freed_count: torch.Tensor, workspace: torch.Tensor,
                         stream: Optional[torch.cuda.Stream] = None) -> None:
    """Draft-state alignment: truncates kv_len and block_tables in place at
    the first draft/committed mismatch of every request; replay receives
    the committed tokens to replay, freed the freed block ids and
    freed_count (one int64) their number."""
    R = block_tables.shape[0] if block_tables.dim() == 2 else -1
    for t, name in ((draft, "draft"), (committed, "committed")):
        if t.dim() != 2 or t.shape[0] != R:
            raise ValueError(f"{name} must be [num_reqs, cols]")
    for t, name in ((draft_len, "draft_len"), (committed_len, "committed_len"),
                    (kv_len, "kv_len"), (replay, "replay")):
        if t.numel() != R:
            raise ValueError(f"{name} must have one entry per request")
    if freed_count.numel() < 1:
        raise ValueError("freed_count needs one element")
    if workspace.numel() * workspace.element_size() < \
            lumen_kv_ckpt_plan_workspace_bytes(R):
        raise ValueError("workspace too small for this many requests")
    i32 = torch.int32
    _check(load_library().lumen_kv_draft_align(
        _dev(draft, "draft", i32), draft.shape[1],
        _dev(draft_len, "draft_len", i32),
        _dev(committed, "committed", i32), committed.shape[1],
        _dev(committed_len, "committed_len", i32),
        _dev(kv_len, "kv_len", i32), _dev(block_tables, "block_tables", i32),
        block_tables.shape[1], int(block_size), R,
        _dev(replay, "replay", i32), _dev(freed, "freed", i32),
        freed.numel(), _dev(freed_count, "freed_count", torch.int64),
        _dev(workspace, "workspace"), _stream_handle(stream)),
        "lumen_kv_draft_align")


def lumen_kv_ckpt_marks_bytes(num_blocks: int) -> int:
    return int(load_library().lumen_kv_ckpt_marks_bytes(int(num_blocks)))


def new_marks(num_blocks: int, device=None) -> torch.Tensor:
    """Device scratch for lumen_kv_ckpt_validate_targets over a pool of
    num_blocks blocks."""
    n = lumen_kv_ckpt_marks_bytes(num_blocks)
    return torch.empty(max(n, 16), dtype=torch.uint8, device=device or "cuda")


def lumen_kv_ckpt_validate_targets(shape, num_blocks: int,
                                   block_tables: torch.Tensor,
                                   workspace: torch.Tensor,
                                   marks: torch.Tensor,
                                   stream: Optional[torch.cuda.Stream] = None
                                   ) -> None:
    """Validate mode of a restore: records RANGE / BLOCK_ID / DUP_BLOCK in
    the workspace's error word for the pages an unpack under this plan and
    table would write (read it with lumen_kv_ckpt_status)."""
    R = block_tables.shape[0] if block_tables.dim() == 2 else -1
    _check_tables(block_tables, R)
    if workspace.numel() * workspace.element_size() < \
            lumen_kv_ckpt_plan_workspace_bytes(R):
        raise ValueError("workspace too small for this many requests")
    nbytes = _nbytes(marks)
    if nbytes < lumen_kv_ckpt_marks_bytes(num_blocks):
        raise ValueError("marks buffer too small for this pool")
    lay = layout(shape, num_blocks)
    _check(load_library().lumen_kv_ckpt_validate_targets(
        ctypes.byref(lay), _dev(block_tables, "block_tables", torch.int32),
        block_tables.shape[1], R, _dev(workspace, "workspace"),
        _dev(marks, "marks"), nbytes, _stream_handle(stream)),
        "lumen_kv_ckpt_validate_targets")


def lumen_kv_ckpt_status(workspace: torch.Tensor,
                         stream: Optional[torch.cuda.Stream] = None) -> int:
    return int(load_library().lumen_kv_ckpt_status(
        _dev(workspace, "workspace"), _stream_handle(stream)))


def _nbytes(t: torch.Tensor) -> int:
    return t.numel() * t.element_size()


def lumen_kv_ckpt_offload(src: torch.Tensor, dst: torch.Tensor,
                          nbytes: Optional[int] = None,
                          producer: Optional[torch.cuda.Stream] = None,
                          side: Optional[torch.cuda.Stream] = None) -> None:
    """Copy the first `nbytes` of device tensor `src` into host tensor `dst`
    (pinned for overlap) on stream `side`, after `producer`'s queued work."""
    n = min(_nbytes(src), _nbytes(dst)) if nbytes is None else int(nbytes)
    if n > _nbytes(src) or n > _nbytes(dst):
        raise ValueError("nbytes exceeds a buffer")
    if dst.is_cuda or not dst.is_contiguous():
        raise ValueError("dst must be a contiguous host tensor")
    _check(load_library().lumen_kv_ckpt_offload(
        _dev(src, "src"), ctypes.c_void_p(dst.data_ptr()), n,
        _stream_handle(producer), _stream_handle(side)),
        "lumen_kv_ckpt_offload")


def lumen_kv_ckpt_stage_in(src: torch.Tensor, dst: torch.Tensor,
                           nbytes: Optional[int] = None,
                           side: Optional[torch.cuda.Stream] = None,
                           consumer: Optional[torch.cuda.Stream] = None) -> None:
    """Copy the first `nbytes` of host tensor `src` into device tensor `dst`
    on stream `side`; later work on `consumer` waits for it."""
    n = min(_nbytes(src), _nbytes(dst)) if nbytes is None else int(nbytes)
    if n > _nbytes(src) or n > _nbytes(dst):
        raise ValueError("nbytes exceeds a buffer")
    if src.is_cuda or not src.is_contiguous():
        raise ValueError("src must be a contiguous host tensor")
    _check(load_library().lumen_kv_ckpt_stage_in(
        ctypes.c_void_p(src.data_ptr()), _dev(dst, "dst"), n,
        _stream_handle(side), _stream_handle(consumer)),
        "lumen_kv_ckpt_stage_in")
