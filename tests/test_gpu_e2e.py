"""The checkpoint pipeline of LUMEN on one GPU, end to end (Sec. 4.2 and
Sec. 4.3): serving steps grow every request's token history; the worker's
progress tracker turns that into ranges of new tokens; the rows are packed
on the GPU and copied to pinned host memory; a receiver appends each
request's rows to its checkpoint store and publishes the tags of pages that
became complete.  One step's transfer is cut short (forced from the host):
only its first rows arrive.  Recovery regenerates the tags from the token
histories, finds each request's longest checkpointed prefix, and restores
exactly those tokens from host memory into freshly allocated blocks.  The
restored pool must equal what the oracle computes straight from the
original cache: the restore of each request's first complete pages."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_17787_amd.kvckpt as kv
from oracle import tags as OT
from paper_2606_17787_amd import workloads as W
from paper_2606_17787_amd.progress import Progress
from paper_2606_17787_amd.tags import TagStore
from paper_2606_17787_amd.workloads import CacheShape, NHD

from gpu_util import d2h16, dev, h2d

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cut_fraction", [0.0, 0.37, 0.9])
def test_checkpoint_cut_stream_then_recover(cut_fraction):
    shape = CacheShape(2, 2, 64, 16, NHD)
    bs, re_ = shape.block_size, shape.token_row_elems
    rb = shape.token_row_bytes
    rng = np.random.default_rng(int(cut_fraction * 1000) + 7)
    R, steps = 12, 9
    prompt = rng.integers(20, 100, R)
    deltas = rng.integers(1, 17, (steps, R))
    final = prompt + deltas.sum(0)
    history = [rng.integers(0, 1 << 17, int(n)).astype(np.int32)
               for n in final]
    pages = -(-final // bs)
    cols = int(pages.max())
    nb = int(pages.sum()) + 7
    perm = rng.permutation(nb).astype(np.int32)
    bt = np.full((R, cols), -1, np.int32)
    k = 0
    for r in range(R):
        bt[r, :pages[r]] = perm[k:k + pages[r]]
        k += pages[r]
    src_h = W.random_bits(rng, shape.pool_elems(nb))
    src, d_bt = h2d(src_h), h2d(bt)

    progress, tags = Progress(), TagStore(bs)
    store = [np.zeros((int(n), re_), np.uint16) for n in final]
    stored = np.zeros(R, np.int64)
    lengths = prompt.copy()
    ps, cs = torch.cuda.Stream(), torch.cuda.Stream()
    staging = torch.empty(2 * 64 * rb, dtype=torch.uint8, device=dev())
    cut_step = steps - 1
    for step in range(steps):
        if step:
            lengths = lengths + deltas[step - 1]
        s, e = progress.ranges(np.arange(R), lengths)
        n = (e - s).astype(np.int64)
        total = int(n.sum())
        host = torch.zeros(max(total, 1) * rb, dtype=torch.uint8,
                           pin_memory=True)
        ws = kv.new_workspace(R, dev())
        d_s, d_e = h2d(s), h2d(e)
        torch.cuda.synchronize()
        kv.lumen_kv_ckpt_plan(d_s, d_e, ws, stream=ps)
        kv.lumen_kv_ckpt_pack_to_host(shape, nb, src, d_bt, ws, total,
                                      staging, 2, host, pack_stream=ps,
                                      copy_stream=cs)
        cs.synchronize()
        assert kv.lumen_kv_ckpt_status(ws, stream=ps) == 0
        rows = host.numpy()[:total * rb].view(np.uint16).reshape(total, re_)
        # the receiver: rows arrive in packed order; the cut step delivers
        # only its first `arrived` rows
        arrived = total if step != cut_step else int(total * cut_fraction)
        off = np.concatenate([[0], np.cumsum(n)[:-1]])
        for r in range(R):
            got = int(np.clip(arrived - off[r], 0, n[r]))
            assert s[r] == stored[r]
            store[r][s[r]:s[r] + got] = rows[off[r]:off[r] + got]
            before = stored[r] // bs
            stored[r] = s[r] + got
            tags.publish_pages(r, history[r][:stored[r]], before,
                               stored[r] // bs)

    # recovery: longest checkpointed prefix from the regenerated tags
    lens = lengths
    e_star = np.array([tags.longest_prefix(r, history[r][:lens[r]])
                       for r in range(R)], np.int64)
    ora = OT.TagStore(bs)
    for r in range(R):
        for i, tg in enumerate(OT.page_tags(history[r][:stored[r]].tolist(),
                                            bs)):
            ora.publish(r, i, tg)
        assert e_star[r] == ora.longest_prefix(r, history[r][:lens[r]].tolist())
    assert (e_star == (stored // bs) * bs).all()
    if cut_fraction < 0.5:
        assert (e_star < lens).any()  # something is left to recompute

    # restore the prefixes from host memory into fresh blocks
    bt2 = np.full((R, cols), -1, np.int32)
    perm2 = rng.permutation(nb).astype(np.int32)
    k = 0
    for r in range(R):
        bt2[r, :pages[r]] = perm2[k:k + pages[r]]
        k += pages[r]
    dst_h = W.random_bits(rng, shape.pool_elems(nb))
    zeros = np.zeros(R, np.int32)
    tot = int(e_star.sum())
    buf = np.concatenate([store[r][:e_star[r]] for r in range(R)])
    host = torch.empty(max(tot, 1) * rb, dtype=torch.uint8, pin_memory=True)
    if tot:
        host.numpy()[:tot * rb] = buf.view(np.uint8).reshape(-1)
    d_dst, d_bt2 = h2d(dst_h), h2d(bt2)
    d_z, d_es = h2d(zeros), h2d(e_star.astype(np.int32))
    ws = kv.new_workspace(R, dev())
    torch.cuda.synchronize()
    us = torch.cuda.Stream()
    kv.lumen_kv_ckpt_plan(d_z, d_es, ws, stream=us)
    kv.lumen_kv_ckpt_unpack_from_host(shape, nb, d_dst, d_bt2, ws, tot, host,
                                      staging, 2, copy_stream=cs,
                                      unpack_stream=us)
    us.synchronize()
    assert kv.lumen_kv_ckpt_status(ws, stream=us) == 0
    # the oracle, straight from the original cache
    st, want_rows = oracle.pack(shape, nb, src_h, bt, zeros, e_star)
    assert st == 0
    want = dst_h.copy()
    assert oracle.unpack(shape, nb, want, bt2, zeros, e_star, want_rows) == 0
    assert np.array_equal(d2h16(d_dst), want)
