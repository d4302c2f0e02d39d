"""The C ABI without a GPU: the library loads, exports every entry point its
header declares, and rejects bad host-side arguments before any HIP call
(the fake pointers below are never dereferenced)."""
import ctypes

import pytest

import paper_2606_17787_amd.kvckpt as kv

FAKE = ctypes.c_void_p(0x7F0000000000)       # 16-byte aligned, never touched
FAKE_ODD = ctypes.c_void_p(0x7F0000000008)   # misaligned for 16 bytes


@pytest.fixture(scope="module")
def lib():
    return kv.load_library()


def test_exports_every_declared_entry_point(lib):
    names = kv.exported_names()
    assert set(names) >= {"lumen_kv_ckpt_plan", "lumen_kv_ckpt_pack",
                          "lumen_kv_ckpt_unpack", "lumen_kv_ckpt_status",
                          "lumen_kv_ckpt_strerror",
                          "lumen_kv_ckpt_plan_workspace_bytes",
                          "lumen_kv_ckpt_offload", "lumen_kv_ckpt_stage_in",
                          "lumen_kv_ckpt_marks_bytes",
                          "lumen_kv_ckpt_validate_targets",
                          "lumen_kv_ckpt_pack_rows",
                          "lumen_kv_ckpt_unpack_rows",
                          "lumen_kv_ckpt_pack_to_host",
                          "lumen_kv_ckpt_unpack_from_host",
                          "lumen_kv_ckpt_pack_to_host_direct",
                          "lumen_kv_ckpt_unpack_from_host_direct",
                          "lumen_kv_draft_align"}
    for n in names:
        assert hasattr(lib, n), n


def _header_defines():
    """Integer #defines of the header, evaluated: decimal literals,
    parentheses, unary minus, an int64_t cast and a left shift."""
    import ast
    import os
    import re
    path = os.path.join(os.path.dirname(os.path.dirname(
        os.path.abspath(__file__))), "include", "lumen_kv_ckpt.h")
    out = {}
    for m in re.finditer(r"^#define (LUMEN_\w+) +(\(.*?\)|-?\d+)(?: |$)",
                         open(path).read(), re.M):
        expr = m.group(2).replace("(int64_t)", "")
        node = ast.parse(expr, mode="eval").body

        def ev(n):
            if isinstance(n, ast.Constant) and isinstance(n.value, int):
                return n.value
            if isinstance(n, ast.UnaryOp) and isinstance(n.op, ast.USub):
                return -ev(n.operand)
            if isinstance(n, ast.BinOp) and isinstance(n.op, ast.LShift):
                return ev(n.left) << ev(n.right)
            raise ValueError(f"{m.group(1)}: {expr}")
        out[m.group(1)] = ev(node)
    return out


def test_binding_constants_match_the_header():
    """Every status code, layout tag and limit the binding names has the
    header's value."""
    defines = _header_defines()
    names = [n for n in dir(kv) if n.startswith("LUMEN_")
             and isinstance(getattr(kv, n), int)]
    assert len(names) >= 15
    for n in names:
        assert n in defines, n
        assert getattr(kv, n) == defines[n], (n, getattr(kv, n), defines[n])
    # and the binding knows every status code
    codes = [n for n in defines if n.startswith("LUMEN_ERR_")]
    assert len(codes) == 9 and all(hasattr(kv, n) for n in codes)
    assert defines["LUMEN_KV_CKPT_MAX_UNITS"] == 2 ** 40


def test_exports_every_page_tag_entry_point(lib):
    from paper_2606_17787_amd import tags
    names = tags.exported_names()
    assert set(names) >= {"lumen_page_tags", "lumen_tag_store_create",
                          "lumen_tag_store_publish",
                          "lumen_tag_store_longest_prefix"}
    for n in names:
        assert hasattr(lib, n), n


def test_exports_every_scheduler_entry_point(lib):
    from paper_2606_17787_amd import sched
    names = sched.exported_names()
    assert set(names) >= {"lumen_sched_create", "lumen_sched_place",
                          "lumen_sched_recover", "lumen_sched_release"}
    for n in names:
        assert hasattr(lib, n), n


def test_exports_every_progress_entry_point(lib):
    from paper_2606_17787_amd import progress
    names = progress.exported_names()
    assert set(names) >= {"lumen_progress_create", "lumen_progress_ranges",
                          "lumen_progress_sent", "lumen_progress_release"}
    for n in names:
        assert hasattr(lib, n), n


def test_missing_library_fails_loudly(tmp_path):
    with pytest.raises(RuntimeError, match="build the HIP library"):
        kv.load_library(str(tmp_path / "absent.so"))


def test_strerror(lib):
    for code in range(-9, 1):
        assert kv.lumen_kv_ckpt_strerror(code) not in ("", "unknown status")
    assert kv.lumen_kv_ckpt_strerror(-99) == "unknown status"


def test_workspace_bytes():
    assert kv.lumen_kv_ckpt_plan_workspace_bytes(-1) == 0
    prev = 0
    for R in (0, 1, 2, 7, 256, 1024, 100000):
        n = kv.lumen_kv_ckpt_plan_workspace_bytes(R)
        assert n % 16 == 0 and n > prev
        assert n >= 64 + 8 * (R + 1) + 8 * R + 4 * R
        prev = n


def _layout(**kw):
    d = dict(num_layers=2, num_kv_heads=2, head_dim=64, block_size=16,
             num_blocks=8, elem_bytes=2, cache_order=kv.LUMEN_CACHE_NHD)
    d.update(kw)
    return kv.lumen_kv_layout(**d)


@pytest.mark.parametrize("fn", ["lumen_kv_ckpt_pack", "lumen_kv_ckpt_unpack"])
def test_copy_host_validation(lib, fn):
    f = getattr(lib, fn)

    def call(lay=None, cache=FAKE, bt=FAKE, cols=4, R=2, ws=FAKE, ck=FAKE,
             rows=100):
        lay = _layout() if lay is None else lay
        return f(ctypes.byref(lay) if lay is not False else None, cache, bt,
                 cols, R, ws, ck, rows, None)

    assert call(lay=False) == kv.LUMEN_ERR_INVALID_ARG
    assert call(lay=_layout(num_layers=0)) == kv.LUMEN_ERR_INVALID_ARG
    assert call(lay=_layout(num_kv_heads=-1)) == kv.LUMEN_ERR_INVALID_ARG
    assert call(lay=_layout(block_size=0)) == kv.LUMEN_ERR_INVALID_ARG
    assert call(lay=_layout(num_blocks=-1)) == kv.LUMEN_ERR_INVALID_ARG
    assert call(lay=_layout(elem_bytes=3)) == kv.LUMEN_ERR_UNSUPPORTED
    assert call(lay=_layout(elem_bytes=8)) == kv.LUMEN_ERR_UNSUPPORTED
    assert call(lay=_layout(elem_bytes=0)) == kv.LUMEN_ERR_UNSUPPORTED
    # a head row must be whole 16-byte vectors: 8 one-byte elements are not
    assert call(lay=_layout(elem_bytes=1, head_dim=8)) == \
        kv.LUMEN_ERR_UNSUPPORTED
    assert call(lay=_layout(cache_order=2)) == kv.LUMEN_ERR_UNSUPPORTED
    assert call(lay=_layout(head_dim=4)) == kv.LUMEN_ERR_UNSUPPORTED
    assert call(lay=_layout(head_dim=12)) == kv.LUMEN_ERR_UNSUPPORTED
    assert call(R=-1) == kv.LUMEN_ERR_INVALID_ARG
    assert call(cols=-1) == kv.LUMEN_ERR_INVALID_ARG
    assert call(rows=-1) == kv.LUMEN_ERR_INVALID_ARG
    assert call(ws=None) == kv.LUMEN_ERR_INVALID_ARG
    assert call(ws=FAKE_ODD) == kv.LUMEN_ERR_MISALIGNED
    assert call(R=0, cache=None, bt=None, ck=None) == kv.LUMEN_OK
    assert call(cache=None) == kv.LUMEN_ERR_INVALID_ARG
    assert call(bt=None) == kv.LUMEN_ERR_INVALID_ARG
    assert call(ck=None) == kv.LUMEN_ERR_INVALID_ARG
    # null is an error only for a non-empty buffer; empty ones pass on to
    # the device (checked here only up to the first HIP call, which fails
    # without a GPU)
    assert call(ck=None, rows=0) in (kv.LUMEN_OK, kv.LUMEN_ERR_HIP)
    assert call(bt=None, cols=0) in (kv.LUMEN_OK, kv.LUMEN_ERR_HIP)
    assert call(cache=FAKE_ODD) == kv.LUMEN_ERR_MISALIGNED
    assert call(ck=FAKE_ODD) == kv.LUMEN_ERR_MISALIGNED


def test_marks_bytes():
    assert kv.lumen_kv_ckpt_marks_bytes(-1) == 0
    assert kv.lumen_kv_ckpt_marks_bytes(0) == 0
    for nb in (1, 127, 128, 129, 56323, 182657):
        n = kv.lumen_kv_ckpt_marks_bytes(nb)
        assert n % 16 == 0 and n * 8 >= nb and (n - 16) * 8 < nb


def test_validate_targets_host_validation(lib):
    f = lib.lumen_kv_ckpt_validate_targets
    need = kv.lumen_kv_ckpt_marks_bytes(8)

    def call(lay=None, bt=FAKE, cols=4, R=2, ws=FAKE, marks=FAKE,
             nbytes=need):
        lay = _layout() if lay is None else lay
        return f(ctypes.byref(lay) if lay is not False else None, bt, cols, R,
                 ws, marks, nbytes, None)

    assert call(lay=False) == kv.LUMEN_ERR_INVALID_ARG
    assert call(lay=_layout(block_size=0)) == kv.LUMEN_ERR_INVALID_ARG
    assert call(lay=_layout(elem_bytes=3)) == kv.LUMEN_ERR_UNSUPPORTED
    assert call(R=-1) == kv.LUMEN_ERR_INVALID_ARG
    assert call(cols=-1) == kv.LUMEN_ERR_INVALID_ARG
    assert call(ws=None) == kv.LUMEN_ERR_INVALID_ARG
    assert call(ws=FAKE_ODD) == kv.LUMEN_ERR_MISALIGNED
    assert call(marks=FAKE_ODD) == kv.LUMEN_ERR_MISALIGNED
    assert call(nbytes=need - 1) == kv.LUMEN_ERR_INVALID_ARG
    assert call(marks=None) == kv.LUMEN_ERR_INVALID_ARG
    assert call(bt=None) == kv.LUMEN_ERR_INVALID_ARG
    assert call(R=0, bt=None, marks=None, nbytes=0) == kv.LUMEN_OK
    # an empty pool needs no marks (passes on to the first HIP call)
    assert call(lay=_layout(num_blocks=0), marks=None, nbytes=0) in (
        kv.LUMEN_OK, kv.LUMEN_ERR_HIP)


def test_plan_host_validation(lib):
    f = lib.lumen_kv_ckpt_plan
    assert f(FAKE, FAKE, -1, 0, None, FAKE, None) == kv.LUMEN_ERR_INVALID_ARG
    assert f(FAKE, FAKE, 2, 0, None, None, None) == kv.LUMEN_ERR_INVALID_ARG
    assert f(None, FAKE, 2, 0, None, FAKE, None) == kv.LUMEN_ERR_INVALID_ARG
    assert f(FAKE, None, 2, 0, None, FAKE, None) == kv.LUMEN_ERR_INVALID_ARG
    assert f(FAKE, FAKE, 2, 0, None, FAKE_ODD, None) == kv.LUMEN_ERR_MISALIGNED


@pytest.mark.parametrize("fn", ["lumen_kv_ckpt_pack_ranges",
                                "lumen_kv_ckpt_unpack_ranges"])
def test_ranges_host_validation(lib, fn):
    """The one-launch copies refuse bad host arguments before any HIP call,
    among them a missing or misaligned status word and more requests than
    one launch's range scan takes."""
    f = getattr(lib, fn)
    odd4 = ctypes.c_void_p(0x7F0000000002)  # not 4-byte aligned

    def call(lay=None, cache=FAKE, bt=FAKE, cols=4, s=FAKE, e=FAKE, R=2,
             ck=FAKE, rows=100, status=FAKE):
        lay = _layout() if lay is None else lay
        return f(ctypes.byref(lay), cache, bt, cols, s, e, R, 0, None, ck,
                 rows, status, None)

    assert call(lay=_layout(num_layers=0)) == kv.LUMEN_ERR_INVALID_ARG
    assert call(lay=_layout(elem_bytes=3)) == kv.LUMEN_ERR_UNSUPPORTED
    assert call(R=-1) == kv.LUMEN_ERR_INVALID_ARG
    assert call(cols=-1) == kv.LUMEN_ERR_INVALID_ARG
    assert call(rows=-1) == kv.LUMEN_ERR_INVALID_ARG
    assert call(status=None) == kv.LUMEN_ERR_INVALID_ARG
    assert call(R=0, status=None) == kv.LUMEN_ERR_INVALID_ARG
    assert call(status=odd4) == kv.LUMEN_ERR_MISALIGNED
    cap = kv.LUMEN_KV_CKPT_RANGES_MAX_REQS
    assert call(R=cap + 1) == kv.LUMEN_ERR_TOO_MANY
    assert call(R=1 << 30) == kv.LUMEN_ERR_TOO_MANY
    assert call(s=None) == kv.LUMEN_ERR_INVALID_ARG
    assert call(e=None) == kv.LUMEN_ERR_INVALID_ARG
    # no requests: nothing to do, nothing enqueued, whatever the buffers
    assert call(R=0, s=None, e=None, cache=None, bt=None, ck=None) == \
        kv.LUMEN_OK
    assert call(cache=None) == kv.LUMEN_ERR_INVALID_ARG
    assert call(bt=None) == kv.LUMEN_ERR_INVALID_ARG
    assert call(ck=None) == kv.LUMEN_ERR_INVALID_ARG
    assert call(cache=FAKE_ODD) == kv.LUMEN_ERR_MISALIGNED
    assert call(ck=FAKE_ODD) == kv.LUMEN_ERR_MISALIGNED
    # a status word needs 4-byte alignment only
    assert call(status=FAKE_ODD, cache=None) == kv.LUMEN_ERR_INVALID_ARG


def test_status_and_copies_host_validation(lib):
    assert lib.lumen_kv_ckpt_status(None, None) == kv.LUMEN_ERR_INVALID_ARG
    assert lib.lumen_kv_ckpt_status(FAKE_ODD, None) == kv.LUMEN_ERR_MISALIGNED
    for f in (lib.lumen_kv_ckpt_offload, lib.lumen_kv_ckpt_stage_in):
        assert f(FAKE, FAKE, 0, None, None) == kv.LUMEN_OK
        assert f(None, FAKE, 16, None, None) == kv.LUMEN_ERR_INVALID_ARG
        assert f(FAKE, None, 16, None, None) == kv.LUMEN_ERR_INVALID_ARG


def test_binding_checks_shapes_before_calling():
    """The binding rejects host tensors and mis-sized buffers itself."""
    import torch
    from paper_2606_17787_amd.workloads import CacheShape
    sh = CacheShape(2, 2, 64, 16)
    cpu = torch.zeros(4, dtype=torch.int32)
    with pytest.raises(ValueError):
        kv.lumen_kv_ckpt_plan(cpu, cpu, torch.zeros(256, dtype=torch.uint8))
    with pytest.raises(ValueError):
        kv.lumen_kv_ckpt_pack(sh, 8, torch.zeros(10, dtype=torch.int16),
                              torch.zeros(2, 4, dtype=torch.int32),
                              torch.zeros(256, dtype=torch.uint8),
                              torch.zeros(512, dtype=torch.int16))


def test_row_range_host_validation(lib):
    for name in ("lumen_kv_ckpt_pack_rows", "lumen_kv_ckpt_unpack_rows"):
        f = getattr(lib, name)

        def call(lay=None, R=2, ws=FAKE, lo=0, hi=10, first=0, rows=10,
                 ck=FAKE):
            lay = _layout() if lay is None else lay
            return f(ctypes.byref(lay), FAKE, FAKE, 4, R, ws, lo, hi, ck,
                     first, rows, None)

        assert call(lo=-1) == kv.LUMEN_ERR_INVALID_ARG
        assert call(lo=5, hi=4) == kv.LUMEN_ERR_INVALID_ARG
        assert call(first=-1) == kv.LUMEN_ERR_INVALID_ARG
        assert call(rows=-1) == kv.LUMEN_ERR_INVALID_ARG
        assert call(ws=None) == kv.LUMEN_ERR_INVALID_ARG
        assert call(lay=_layout(elem_bytes=3)) == kv.LUMEN_ERR_UNSUPPORTED
        assert call(ck=FAKE_ODD) == kv.LUMEN_ERR_MISALIGNED
        # an empty row range or no requests enqueues nothing
        assert call(lo=7, hi=7) == kv.LUMEN_OK
        assert call(R=0) == kv.LUMEN_OK


def test_pipeline_host_validation(lib):
    for name in ("lumen_kv_ckpt_pack_to_host",
                 "lumen_kv_ckpt_unpack_from_host"):
        f = getattr(lib, name)
        pack = name.endswith("to_host")

        def call(R=2, ws=FAKE, total=100, staging=FAKE, slot_rows=8,
                 slots=2, host=FAKE):
            lay = _layout()
            if pack:
                return f(ctypes.byref(lay), FAKE, FAKE, 4, R, ws, total,
                         staging, slot_rows, slots, host, None, None)
            return f(ctypes.byref(lay), FAKE, FAKE, 4, R, ws, total, host,
                     staging, slot_rows, slots, None, None)

        assert call(slots=0) == kv.LUMEN_ERR_INVALID_ARG
        assert call(slots=65) == kv.LUMEN_ERR_INVALID_ARG
        assert call(slot_rows=0) == kv.LUMEN_ERR_INVALID_ARG
        assert call(total=-1) == kv.LUMEN_ERR_INVALID_ARG
        assert call(ws=None) == kv.LUMEN_ERR_INVALID_ARG
        assert call(staging=None) == kv.LUMEN_ERR_INVALID_ARG
        assert call(host=None) == kv.LUMEN_ERR_INVALID_ARG
        assert call(staging=FAKE_ODD) == kv.LUMEN_ERR_MISALIGNED
        assert call(ws=FAKE_ODD) == kv.LUMEN_ERR_MISALIGNED
        # nothing to move: no HIP call at all
        assert call(total=0, staging=None, host=None) == kv.LUMEN_OK
        assert call(R=0) == kv.LUMEN_OK


def test_direct_host_copy_validation(lib):
    for name in ("lumen_kv_ckpt_pack_to_host_direct",
                 "lumen_kv_ckpt_unpack_from_host_direct"):
        f = getattr(lib, name)

        def call(lay=None, R=2, ws=FAKE, lo=0, hi=10, first=0, rows=10,
                 host=None, wg=0):
            lay = _layout() if lay is None else lay
            return f(ctypes.byref(lay), FAKE, FAKE, 4, R, ws, lo, hi, host,
                     first, rows, wg, None)

        assert call(wg=-1) == kv.LUMEN_ERR_INVALID_ARG
        assert call(wg=4097) == kv.LUMEN_ERR_INVALID_ARG
        assert call(lo=-1) == kv.LUMEN_ERR_INVALID_ARG
        assert call(lo=5, hi=4) == kv.LUMEN_ERR_INVALID_ARG
        assert call(first=-1) == kv.LUMEN_ERR_INVALID_ARG
        assert call(rows=-1) == kv.LUMEN_ERR_INVALID_ARG
        assert call(ws=None) == kv.LUMEN_ERR_INVALID_ARG
        assert call(lay=_layout(elem_bytes=3)) == kv.LUMEN_ERR_UNSUPPORTED
        # a window of rows but no host memory: refused before any HIP call
        assert call(host=None) == kv.LUMEN_ERR_INVALID_ARG
        # an empty row range or no requests enqueues nothing
        assert call(lo=7, hi=7) == kv.LUMEN_OK
        assert call(R=0) == kv.LUMEN_OK


def test_draft_align_host_validation(lib):
    f = lib.lumen_kv_draft_align

    def call(dc=8, cc=8, btc=4, bs=4, R=2, cap=10, ws=FAKE, cnt=FAKE,
             freed=FAKE, kl=FAKE):
        return f(FAKE, dc, FAKE, FAKE, cc, FAKE, kl, FAKE, btc, bs, R, FAKE,
                 freed, cap, cnt, ws, None)

    assert call(bs=0) == kv.LUMEN_ERR_INVALID_ARG
    assert call(R=-1) == kv.LUMEN_ERR_INVALID_ARG
    assert call(dc=-1) == kv.LUMEN_ERR_INVALID_ARG
    assert call(btc=-1) == kv.LUMEN_ERR_INVALID_ARG
    assert call(cap=-1) == kv.LUMEN_ERR_INVALID_ARG
    assert call(ws=None) == kv.LUMEN_ERR_INVALID_ARG
    assert call(cnt=None) == kv.LUMEN_ERR_INVALID_ARG
    assert call(kl=None) == kv.LUMEN_ERR_INVALID_ARG
    assert call(freed=None) == kv.LUMEN_ERR_INVALID_ARG
    assert call(ws=FAKE_ODD) == kv.LUMEN_ERR_MISALIGNED


@pytest.mark.parametrize("header", ["lumen_kv_ckpt.h", "lumen_page_tags.h",
                                    "lumen_sched.h", "lumen_progress.h"])
@pytest.mark.parametrize("lang", ["c", "c++"])
def test_headers_compile_on_their_own(header, lang):
    """Each public header parses alone as C and as C++ (no HIP headers
    needed), with warnings as errors."""
    import os
    import shutil
    import subprocess
    cc = shutil.which("gcc" if lang == "c" else "g++")
    if cc is None:
        pytest.skip("no host compiler")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    inc = os.path.join(root, "include")
    r = subprocess.run([cc, "-x", lang, "-fsyntax-only", "-Wall", "-Werror",
                        "-I", inc, os.path.join(inc, header)],
                       capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
