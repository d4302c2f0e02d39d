"""The five workloads at their full sizes, on the GPU, in the launch
configuration the benchmark times (the library's default grid).

The oracle cannot hold 100+ GiB pools at once, so each check gathers the
physical blocks a chunk of requests touches into a compact host pool (a
consistent relabelling of blocks, which the oracle's pins show leaves the
checkpoint unchanged), runs the oracle there and compares element by element
with the rows the GPU wrote.  Every checkpoint row of every workload is
checked this way, and so is every restored token (packed back by the oracle
from the restored pool).  Properties that hold at any size add to it:
restore after checkpoint round-trips over every request on the GPU, and
sampled blocks and slots no request names are left byte-identical.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
import paper_2606_17787_amd.kvckpt as kv
from paper_2606_17787_amd import workloads as W

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def say(msg):
    print(msg, flush=True)


def fill_random(n, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    t = torch.empty(n, dtype=torch.int16, device=DEV)
    t.view(torch.uint8).random_(0, 256, generator=g)  # every 16-bit pattern
    return t


def slab_view(pool, shape, nb):
    """[L*2, NB, block_elems] view of a flat pool (either layout: a block is
    contiguous inside each (layer, K/V) slab)."""
    return pool.view(shape.num_layers * 2, nb, -1)


def gather_blocks(pool, shape, nb, blocks):
    """Host copy of the given physical blocks as a compact pool (flat
    uint16 in the same layout, blocks renumbered 0..len-1)."""
    idx = torch.from_numpy(np.asarray(blocks, np.int64)).to(DEV)
    sub = slab_view(pool, shape, nb).index_select(1, idx)
    return sub.contiguous().view(-1).cpu().numpy().view(np.uint16)


def compact_tables(bt, reqs, s, e, bs):
    """Blocks the requests' ranges touch, and their tables renumbered."""
    blocks, remap = [], {}
    sub = np.full((len(reqs), bt.shape[1]), -1, np.int32)
    for i, r in enumerate(reqs):
        if e[r] <= s[r]:
            continue
        for j in range(int(s[r]) // bs, (int(e[r]) - 1) // bs + 1):
            b = int(bt[r, j])
            if b not in remap:
                remap[b] = len(blocks)
                blocks.append(b)
            sub[i, j] = remap[b]
    return blocks, sub


def gpu_rows(ck_dev, shape, first_row, reqs, s, e):
    rows = ck_dev.view(-1, shape.token_row_elems)
    out = [rows[int(first_row[r]):int(first_row[r]) + int(e[r] - s[r])]
           for r in reqs]
    return torch.cat(out).cpu().numpy().view(np.uint16)


def check_unpack_sample(shape, before, after, nb, bt, s, e, ck_rows_host,
                        reqs, what):
    """`before`: compact host pool of the blocks (in `blocks` order) prior to
    the unpack; `after`: the same blocks gathered after it."""
    blocks, sub = compact_tables(bt, reqs, s, e, shape.block_size)
    want = before.copy()
    st = oracle.unpack(shape, len(blocks), want, sub, s[reqs], e[reqs],
                       ck_rows_host)
    assert st == oracle.OK
    if not np.array_equal(after, want):
        raise AssertionError(f"{what}: restored blocks differ at "
                             f"{int((after != want).sum())} elements")


def roundtrip_all(shape, nb, cache, bt, s, e, ck, row_base, chunk, what):
    """Re-pack every request from `cache` under `bt`, a chunk of requests at
    a time, and compare with the checkpoint rows `ck` (on the device)."""
    _, first, _ = oracle.plan(s, e, row_base)
    R = len(s)
    row_elems = shape.token_row_elems
    for r0 in range(0, R, chunk):
        r1 = min(R, r0 + chunk)
        n = int((e[r0:r1] - s[r0:r1]).sum())
        if n == 0:
            continue
        ws = kv.new_workspace(r1 - r0, DEV)
        kv.lumen_kv_ckpt_plan(torch.from_numpy(s[r0:r1]).to(DEV),
                              torch.from_numpy(e[r0:r1]).to(DEV), ws)
        tmp = torch.empty(n * row_elems, dtype=torch.int16, device=DEV)
        kv.lumen_kv_ckpt_pack(shape, nb, cache,
                              torch.from_numpy(np.ascontiguousarray(bt[r0:r1])).to(DEV),
                              ws, tmp)
        assert kv.lumen_kv_ckpt_status(ws) == 0
        ref = ck.view(-1, row_elems)[int(first[r0]):int(first[r0]) + n]
        assert torch.equal(tmp.view(-1, row_elems), ref), f"{what}: requests {r0}..{r1}"


def check_all_rows(shape, pool, nb, bt, s, e, ck, row_base, what,
                   chunk_bytes=1 << 30):
    """Every checkpoint row of a packed plan against the oracle.  The token
    ranges are cut into pieces, and consecutive pieces into chunks of about
    chunk_bytes of rows.  Per chunk, the blocks its pieces touch are
    gathered into a compact pinned host pool, the oracle (its C code, on the
    host's threads, one run of pieces each) writes the chunk's rows into a
    pinned buffer, and that buffer is compared on the device with the rows
    the GPU wrote (one contiguous run of the checkpoint)."""
    n = np.maximum(e.astype(np.int64) - s, 0)
    if int(n.sum()) == 0:
        return
    row_elems = shape.token_row_elems
    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    chunk_rows = max(threads, chunk_bytes // shape.token_row_bytes)
    piece = max(1, chunk_rows // threads)
    preq, ps, pe = [], [], []
    for r in range(len(s)):
        for t in range(int(s[r]), int(s[r]) + int(n[r]), piece):
            preq.append(r)
            ps.append(t)
            pe.append(min(t + piece, int(s[r]) + int(n[r])))
    preq = np.array(preq, np.int64)
    ps = np.array(ps, np.int32)
    pe = np.array(pe, np.int32)
    plen = (pe - ps).astype(np.int64)
    prow = row_base + np.concatenate([[0], np.cumsum(plen)[:-1]])
    rows_dev = ck.view(-1, row_elems)
    src_pin = out_pin = None
    with ThreadPoolExecutor(threads) as ex:
        i = 0
        while i < len(preq):
            j, rows = i, 0
            while j < len(preq) and (j == i or rows + plen[j] <= chunk_rows):
                rows += int(plen[j])
                j += 1
            blocks, sub = compact_tables(bt[preq[i:j]], np.arange(j - i),
                                         ps[i:j], pe[i:j], shape.block_size)
            idx = torch.from_numpy(np.asarray(blocks, np.int64)).to(DEV)
            gathered = slab_view(pool, shape, nb).index_select(1, idx)
            need = gathered.numel()
            if src_pin is None or src_pin.numel() < need:
                src_pin = torch.empty(need, dtype=torch.int16, pin_memory=True)
            src_pin[:need].copy_(gathered.view(-1))
            del gathered
            host = src_pin[:need].numpy().view(np.uint16)
            if out_pin is None or out_pin.numel() < rows * row_elems:
                out_pin = torch.empty(rows * row_elems, dtype=torch.int16,
                                      pin_memory=True)
            out = out_pin[:rows * row_elems].numpy().view(np.uint16).reshape(
                rows, row_elems)
            cuts = np.linspace(i, j, threads + 1).astype(int)

            def part(k):
                a, b = cuts[k], cuts[k + 1]
                if a >= b:
                    return
                lo = int(prow[a] - prow[i])
                hi = lo + int(plen[a:b].sum())
                st, _ = oracle.pack(shape, len(blocks), host, sub[a - i:b - i],
                                    ps[a:b], pe[a:b], ckpt=out[lo:hi])
                assert st == oracle.OK, (what, st)

            list(ex.map(part, range(threads)))
            want = out_pin[:rows * row_elems].to(DEV)
            got = rows_dev[int(prow[i]):int(prow[i]) + rows].reshape(-1)
            if not torch.equal(got, want):
                bad = torch.nonzero(got != want)[:3].flatten().tolist()
                raise AssertionError(
                    f"{what}: rows {int(prow[i])}..{int(prow[i]) + rows}: "
                    f"first differing elements {bad}")
            # one line per chunk, so that no phase of the host-side oracle
            # checks runs silently for long
            say(f"[fullsize] {what}: rows {int(prow[i])}..{int(prow[i]) + rows}"
                " equal the oracle")
            i = j


def sample(rng, R, k):
    return np.unique(np.concatenate([[0, R - 1], rng.choice(R, k, replace=False)]))


@pytest.fixture(autouse=True)
def free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("make,via", [(W.c2_llama8b, "ranges"),
                                      (W.c2_llama8b, "plan"),
                                      (W.c5_qwen_hnd, "plan")],
                         ids=["llama3-8b-decode-ranges",
                              "llama3-8b-decode-plan", "qwen-gqa-hnd"])
def test_incremental_full_size(make, via):
    """via: the copies issued as the benchmark's decode leg issues them (one
    launch per copy that plans from the ranges) or after a plan kernel."""
    w = make()
    sh = w.shape
    say(f"[fullsize] {w.name}: source pool {w.num_blocks} blocks")
    rng = np.random.default_rng(7)
    src = fill_random(sh.pool_elems(w.num_blocks), 11)
    dst = fill_random(sh.pool_elems(w.dst_num_blocks), 12)
    dst_before = dst.clone()
    rows = np.array([w.step_tokens(k) for k in range(w.num_steps)], np.int64)
    row_off = np.concatenate([[0], np.cumsum(rows)])
    arena = torch.empty(int(row_off[-1]) * sh.token_row_elems,
                        dtype=torch.int16, device=DEV)
    bt = torch.from_numpy(w.block_tables).to(DEV)
    btd = torch.from_numpy(w.dst_block_tables).to(DEV)
    ws = kv.new_workspace(w.num_reqs, DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    for k in range(w.num_steps):
        s, e = w.starts[k], w.ends[k]
        d_s, d_e = torch.from_numpy(s).to(DEV), torch.from_numpy(e).to(DEV)
        if via == "ranges":
            kv.lumen_kv_ckpt_pack_ranges(sh, w.num_blocks, src, bt, d_s, d_e,
                                         arena, status, int(row_off[k]))
            kv.lumen_kv_ckpt_unpack_ranges(sh, w.dst_num_blocks, dst, btd,
                                           d_s, d_e, arena, status,
                                           int(row_off[k]))
            assert int(status.item()) == kv.LUMEN_OK, f"step {k}"
        else:
            kv.lumen_kv_ckpt_plan(d_s, d_e, ws, int(row_off[k]))
            kv.lumen_kv_ckpt_pack(sh, w.num_blocks, src, bt, ws, arena)
            kv.lumen_kv_ckpt_unpack(sh, w.dst_num_blocks, dst, btd, ws, arena)
            assert kv.lumen_kv_ckpt_status(ws) == kv.LUMEN_OK, f"step {k}"
        check_all_rows(sh, src, w.num_blocks, w.block_tables, s, e, arena,
                       int(row_off[k]), f"{w.name} step {k}")
    say(f"[fullsize] {w.name}: restored pool re-packs to the checkpoint")
    # every restored token re-packs to its checkpoint row
    for k in range(w.num_steps):
        roundtrip_all(sh, w.dst_num_blocks, dst, w.dst_block_tables,
                      w.starts[k], w.ends[k],
                      arena, int(row_off[k]), 128, f"{w.name} step {k}")
    # and, read back by the oracle, every restored token equals its row
    # (every token is written by exactly one step)
    for k in range(w.num_steps):
        check_all_rows(sh, dst, w.dst_num_blocks, w.dst_block_tables,
                       w.starts[k], w.ends[k], arena, int(row_off[k]),
                       f"{w.name} restore of step {k}")
    # sampled requests' destination blocks, whole: written slots hold their
    # rows from every step, all other slots keep their bytes
    reqs = sample(rng, w.num_reqs, 14)
    s0, e_last = w.starts[0], w.ends[-1]
    blocks, _ = compact_tables(w.dst_block_tables, reqs, s0, e_last,
                               sh.block_size)
    before = gather_blocks(dst_before, sh, w.dst_num_blocks, blocks)
    after = gather_blocks(dst, sh, w.dst_num_blocks, blocks)
    firsts = [oracle.plan(w.starts[k], w.ends[k], int(row_off[k]))[1]
              for k in range(w.num_steps)]
    rows_dev = arena.view(-1, sh.token_row_elems)
    parts = [rows_dev[int(firsts[k][r]):int(firsts[k][r])
                      + int(w.ends[k][r] - w.starts[k][r])]
             for r in reqs for k in range(w.num_steps)]
    union_rows = torch.cat(parts).cpu().numpy().view(np.uint16)
    check_unpack_sample(sh, before, after, w.dst_num_blocks,
                        w.dst_block_tables, s0, e_last, union_rows, reqs,
                        f"{w.name} restore pool")


def test_restore_burst_full_size():
    w = W.c3_restore()
    sh = w.shape
    waves = W.restore_waves(w)
    assert len(waves) >= 2
    ctx = w.ends[0].astype(np.int64)
    max_rows = max(int(ctx[wv].sum()) for wv in waves)
    say(f"[fullsize] restore burst: {len(waves)} waves, {max_rows} rows max")
    # each pool block starts as a constant of its own; occupied blocks must
    # keep it
    NB = w.dst_num_blocks
    pool = torch.empty(sh.pool_elems(NB), dtype=torch.int16, device=DEV)
    fill = (torch.arange(NB, device=DEV, dtype=torch.int64) * 7919 % 65521
            - 32768).to(torch.int16)
    slab_view(pool, sh, NB).copy_(fill.view(1, NB, 1).expand(
        sh.num_layers * 2, NB, slab_view(pool, sh, NB).shape[2]))
    ck = fill_random(max_rows * sh.token_row_elems, 13)
    for wi, wv in enumerate(waves):
        s, e = w.starts[0][wv], w.ends[0][wv]
        bt = np.ascontiguousarray(w.dst_block_tables[wv])
        nrows = int(ctx[wv].sum())
        ws = kv.new_workspace(len(wv), DEV)
        kv.lumen_kv_ckpt_plan(torch.from_numpy(s).to(DEV),
                              torch.from_numpy(e).to(DEV), ws)
        view = ck[:nrows * sh.token_row_elems]
        kv.lumen_kv_ckpt_unpack(sh, NB, pool, torch.from_numpy(bt).to(DEV),
                                ws, view)
        assert kv.lumen_kv_ckpt_status(ws) == kv.LUMEN_OK
        roundtrip_all(sh, NB, pool, bt, s, e, view, 0, 4, f"wave {wi}")
        # every restored token, read back by the oracle
        check_all_rows(sh, pool, NB, bt, s, e, view, 0, f"wave {wi} restore")
        sv = slab_view(pool, sh, NB)
        # in every request's last block, the slots past its last token keep
        # the block's constant (ranges start at token 0, so only the last
        # block is partial)
        assert sh.order == "NHD" and not s.any()
        bs = sh.block_size
        part = [i for i in range(len(wv)) if int(e[i]) % bs]
        if part:
            last = torch.from_numpy(np.array(
                [bt[i, (int(e[i]) - 1) // bs] for i in part], np.int64)).to(DEV)
            cut = torch.tensor([int(e[i]) % bs for i in part], device=DEV)
            got = sv.index_select(1, last).view(sv.shape[0], len(part), bs, -1)
            past = (torch.arange(bs, device=DEV).view(1, 1, bs, 1)
                    >= cut.view(1, -1, 1, 1))
            assert bool(((got == fill[last].view(1, -1, 1, 1)) | ~past).all()), \
                f"wave {wi}: a slot past a request's last token changed"
        # occupied blocks keep their constant
        occ = torch.from_numpy(w.occupied).to(DEV)
        for c0 in range(0, occ.numel(), 1024):
            idx = occ[c0:c0 + 1024]
            got = sv.index_select(1, idx)
            assert bool((got == fill[idx].view(1, -1, 1)).all()), f"wave {wi}"
        # the next wave reuses the free list: put the constants back
        freed = torch.from_numpy(np.unique(bt[bt >= 0]).astype(np.int64)).to(DEV)
        for c0 in range(0, freed.numel(), 1024):
            idx = freed[c0:c0 + 1024]
            val = fill[idx].view(1, -1, 1).expand(sv.shape[0], -1, sv.shape[2])
            sv.index_copy_(1, idx, val.contiguous())


def test_tp8_shard_full_size_in_place():
    w = W.c4_llama70b_tp8()
    sh = w.shape
    say(f"[fullsize] tp8 shard: pool {w.num_blocks} blocks, {w.step_tokens(0)} rows")
    rng = np.random.default_rng(4)
    pool = fill_random(sh.pool_elems(w.num_blocks), 14)
    s, e = w.starts[0], w.ends[0]
    n = w.step_tokens(0)
    arena = torch.empty(n * sh.token_row_elems, dtype=torch.int16, device=DEV)
    ws = kv.new_workspace(w.num_reqs, DEV)
    kv.lumen_kv_ckpt_plan(torch.from_numpy(s).to(DEV), torch.from_numpy(e).to(DEV), ws)
    kv.lumen_kv_ckpt_pack(sh, w.num_blocks, pool,
                          torch.from_numpy(w.block_tables).to(DEV), ws, arena)
    assert kv.lumen_kv_ckpt_status(ws) == kv.LUMEN_OK
    check_all_rows(sh, pool, w.num_blocks, w.block_tables, s, e, arena, 0,
                   "tp8 pack")
    reqs = sample(rng, w.num_reqs, 5)
    # restore in place under a fresh permutation of the same pool
    blocks, _ = compact_tables(w.dst_block_tables, reqs, s, e, sh.block_size)
    before = gather_blocks(pool, sh, w.num_blocks, blocks)
    kv.lumen_kv_ckpt_unpack(sh, w.num_blocks, pool,
                            torch.from_numpy(w.dst_block_tables).to(DEV), ws,
                            arena)
    assert kv.lumen_kv_ckpt_status(ws) == kv.LUMEN_OK
    after = gather_blocks(pool, sh, w.num_blocks, blocks)
    _, first, _ = oracle.plan(s, e)
    rows_h = gpu_rows(arena, sh, first, reqs, s, e).reshape(-1, sh.token_row_elems)
    check_unpack_sample(sh, before, after, w.num_blocks, w.dst_block_tables,
                        s, e, rows_h, reqs, "tp8 unpack")
    roundtrip_all(sh, w.num_blocks, pool, w.dst_block_tables, s, e, arena, 0,
                  32, "tp8 round trip")
