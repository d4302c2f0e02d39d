"""The copy-kernel timing hook (lumen_kv_ckpt_time_next_copy): the next copy
call's kernel stamps its own start and end on the caller's HIP events, and
its rows are the oracle's as without the hook."""
import numpy as np
import pytest
import torch

import bench
import oracle
import paper_2606_17787_amd.kvckpt as kv
from paper_2606_17787_amd import workloads as W
from paper_2606_17787_amd.workloads import CacheShape, NHD
from gpu_util import SENTINEL, d2h16, dev, h2d

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("via", ["plan", "ranges"])
@pytest.mark.parametrize("shape", [CacheShape(2, 2, 8, 4, NHD),
                                   CacheShape(3, 4, 64, 16, NHD)],
                         ids=["page-major", "token-major"])
def test_timed_copies_match_the_oracle(shape, via):
    rng = np.random.default_rng(91)
    R, nb, cols = 6, 40, 6
    bt = rng.permutation(nb)[:R * cols].astype(np.int32).reshape(R, cols)
    s = rng.integers(0, 20, R).astype(np.int32)
    e = (s + rng.integers(0, 30, R)).astype(np.int32)
    e = np.minimum(e, cols * shape.block_size).astype(np.int32)
    rows = int((e - s).sum())
    src = W.random_bits(rng, shape.pool_elems(nb))
    dst = W.random_bits(rng, shape.pool_elems(nb))
    st, want = oracle.pack(shape, nb, src, bt, s, e)
    assert st == oracle.OK
    want_dst = dst.copy()
    assert oracle.unpack(shape, nb, want_dst, bt, s, e, want) == oracle.OK

    d_s, d_e, d_bt = h2d(s), h2d(e), h2d(bt)
    ck = h2d(np.full(rows * shape.token_row_elems, SENTINEL, np.uint16))
    d_dst = h2d(dst)
    ws = kv.new_workspace(R, dev())
    status = torch.zeros(1, dtype=torch.int32, device=dev())
    ev = [bench.TimingEvent() for _ in range(4)]
    for i, pack in ((0, True), (2, False)):
        if via == "plan":
            kv.lumen_kv_ckpt_plan(d_s, d_e, ws)
        kv.lumen_kv_ckpt_time_next_copy(ev[i].ev, ev[i + 1].ev)
        cache, fn = ((h2d(src), kv.lumen_kv_ckpt_pack) if pack
                     else (d_dst, kv.lumen_kv_ckpt_unpack))
        if via == "plan":
            fn(shape, nb, cache, d_bt, ws, ck)
        else:
            fn = (kv.lumen_kv_ckpt_pack_ranges if pack
                  else kv.lumen_kv_ckpt_unpack_ranges)
            fn(shape, nb, cache, d_bt, d_s, d_e, ck, status)
    ev[3].synchronize()
    for i in (0, 2):
        ms = ev[i].elapsed_time(ev[i + 1])
        assert 0.0 < ms < 1000.0, ms
    assert np.array_equal(d2h16(ck).reshape(rows, -1), want)
    assert np.array_equal(d2h16(d_dst), want_dst)
    if via == "plan":
        assert kv.lumen_kv_ckpt_status(ws) == kv.LUMEN_OK
    else:
        assert int(status.item()) == kv.LUMEN_OK


def test_events_wait_for_a_launch_and_serve_one():
    """Arming, then a call the library refuses (a misaligned checkpoint):
    nothing is launched and the events stay unrecorded.  The next copy
    kernel takes them; the copies after it run untimed and leave them as
    they are.  (The failed query of the unrecorded events leaves an error
    pending in the runtime; the next copy must still report its own
    launch, LUMEN_OK.)"""
    shape = CacheShape(2, 2, 8, 4, NHD)
    rng = np.random.default_rng(92)
    nb = 8
    bt = np.array([[0, 1, 2]], np.int32)
    s, e = np.array([0], np.int32), np.array([12], np.int32)
    src = h2d(W.random_bits(rng, shape.pool_elems(nb)))
    d_s, d_e, d_bt = h2d(s), h2d(e), h2d(bt)
    row = shape.token_row_elems
    ck = torch.zeros(13 * row, dtype=torch.int16, device=dev())
    ws = kv.new_workspace(1, dev())
    kv.lumen_kv_ckpt_plan(d_s, d_e, ws)
    a, b = bench.TimingEvent(), bench.TimingEvent()
    kv.lumen_kv_ckpt_time_next_copy(a.ev, b.ev)
    with pytest.raises(kv.LumenError) as ex:
        kv.lumen_kv_ckpt_pack(shape, nb, src, d_bt, ws, ck[1:1 + 12 * row])
    assert ex.value.code == kv.LUMEN_ERR_MISALIGNED
    torch.cuda.synchronize()
    with pytest.raises(RuntimeError):
        a.elapsed_time(b)  # never recorded
    kv.lumen_kv_ckpt_pack(shape, nb, src, d_bt, ws, ck[:12 * row])
    b.synchronize()
    first = a.elapsed_time(b)
    assert 0.0 < first < 1000.0
    for _ in range(3):
        kv.lumen_kv_ckpt_pack(shape, nb, src, d_bt, ws, ck[:12 * row])
    torch.cuda.synchronize()
    assert a.elapsed_time(b) == first
    assert kv.lumen_kv_ckpt_status(ws) == kv.LUMEN_OK


def _leave_a_pending_error():
    """A failed runtime query of the caller's (elapsed time of events never
    recorded) leaves an error pending in this thread."""
    a, b = bench.TimingEvent(), bench.TimingEvent()
    with pytest.raises(RuntimeError):
        a.elapsed_time(b)


def test_calls_report_their_own_launches_after_a_pending_error():
    """Plan, pack, the one-launch copy and validate mode each report the
    outcome of their own launches, not an error an earlier, unrelated
    runtime call left pending."""
    shape = CacheShape(2, 2, 64, 4, NHD)
    rng = np.random.default_rng(93)
    nb = 8
    bt = np.array([[0, 1, 2], [3, 4, 5]], np.int32)
    s, e = np.array([0, 2], np.int32), np.array([12, 9], np.int32)
    rows = int((e - s).sum())
    src_h = W.random_bits(rng, shape.pool_elems(nb))
    src = h2d(src_h)
    d_s, d_e, d_bt = h2d(s), h2d(e), h2d(bt)
    ck = torch.zeros(rows * shape.token_row_elems, dtype=torch.int16,
                     device=dev())
    ws = kv.new_workspace(2, dev())
    _leave_a_pending_error()
    kv.lumen_kv_ckpt_plan(d_s, d_e, ws)
    _leave_a_pending_error()
    kv.lumen_kv_ckpt_pack(shape, nb, src, d_bt, ws, ck)
    _leave_a_pending_error()
    kv.lumen_kv_ckpt_validate_targets(shape, nb, d_bt, ws,
                                      kv.new_marks(nb, dev()))
    assert kv.lumen_kv_ckpt_status(ws) == kv.LUMEN_OK
    status = torch.zeros(1, dtype=torch.int32, device=dev())
    ck2 = torch.zeros_like(ck)
    _leave_a_pending_error()
    kv.lumen_kv_ckpt_pack_ranges(shape, nb, src, d_bt, d_s, d_e, ck2, status)
    torch.cuda.synchronize()
    assert int(status.item()) == kv.LUMEN_OK
    st, want = oracle.pack(shape, nb, src_h, bt, s, e)
    assert st == oracle.OK
    for got in (ck, ck2):
        assert np.array_equal(d2h16(got).reshape(rows, -1), want)
