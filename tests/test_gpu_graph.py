"""The checkpoint step (plan, pack, plan, unpack; or the two one-launch
copies that read the ranges) captured in a HIP graph and replayed: the
library issues only kernels, no memsets, so a capture holds the whole step.  Each replay follows eager work that changes the inputs
(new cache contents, a reset destination pool) and a synchronisation, and
is checked against the oracle on the same inputs."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_17787_amd.kvckpt as kv
from paper_2606_17787_amd import workloads as W

from gpu_util import d2h16, dev, h2d

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("make", [
    lambda: W.c2_llama8b(num_reqs=11, steps=2, median=200, clip_hi=400),
    lambda: W.c4_llama70b_tp8(num_reqs=9, median=150, clip_hi=500),
], ids=["decode-small", "tp8-small-page-major"])
@pytest.mark.parametrize("via", ["plan", "ranges"])
def test_captured_step_replays_match_oracle(make, via):
    w = make()
    sh = w.shape
    k = 0
    s, e = w.starts[k], w.ends[k]
    rows = w.step_tokens(k)
    rng = np.random.default_rng(61)
    src_h = W.random_bits(rng, sh.pool_elems(w.num_blocks))
    dst_h = W.random_bits(rng, sh.pool_elems(w.dst_num_blocks))
    src, dst = h2d(src_h), h2d(dst_h)
    d_s, d_e = h2d(s), h2d(e)
    bt, bt2 = h2d(w.block_tables), h2d(w.dst_block_tables)
    ws_a = kv.new_workspace(w.num_reqs, dev())
    ws_b = kv.new_workspace(w.num_reqs, dev())
    ck = torch.zeros(rows * sh.token_row_elems, dtype=torch.int16,
                     device=dev())

    status = torch.zeros(1, dtype=torch.int32, device=dev())

    def step():
        if via == "ranges":
            kv.lumen_kv_ckpt_pack_ranges(sh, w.num_blocks, src, bt, d_s, d_e,
                                         ck, status)
            kv.lumen_kv_ckpt_unpack_ranges(sh, w.dst_num_blocks, dst, bt2,
                                           d_s, d_e, ck, status)
            return
        kv.lumen_kv_ckpt_plan(d_s, d_e, ws_a)
        kv.lumen_kv_ckpt_pack(sh, w.num_blocks, src, bt, ws_a, ck)
        kv.lumen_kv_ckpt_plan(d_s, d_e, ws_b)
        kv.lumen_kv_ckpt_unpack(sh, w.dst_num_blocks, dst, bt2, ws_b, ck)

    def statuses_ok():
        assert kv.lumen_kv_ckpt_status(ws_a) == 0
        assert kv.lumen_kv_ckpt_status(ws_b) == 0
        assert int(status.item()) == 0

    # eager once (device state of the library initialised outside capture)
    step()
    torch.cuda.synchronize()
    statuses_ok()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    for rep in range(4):
        # eager work between replays: new cache contents, fresh destination
        new_src = W.random_bits(rng, sh.pool_elems(w.num_blocks))
        src.copy_(h2d(new_src))
        dst.copy_(h2d(dst_h))
        ck.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        statuses_ok()
        st, want_ck = oracle.pack(sh, w.num_blocks, new_src, w.block_tables,
                                  s, e)
        assert st == 0
        want_dst = dst_h.copy()
        assert oracle.unpack(sh, w.dst_num_blocks, want_dst,
                             w.dst_block_tables, s, e, want_ck) == 0
        assert np.array_equal(d2h16(ck).reshape(want_ck.shape), want_ck), rep
        assert np.array_equal(d2h16(dst), want_dst), rep
