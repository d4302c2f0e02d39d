"""Checks that pin the CPU oracle to facts outside the oracle itself.

The paper prints no worked example for the checkpoint path, so the oracle is
pinned by what the mathematics fixes:

* coordinate decoding: every pool element holds the mixed-radix code of its
  logical coordinate (layer, K/V, block, slot, head, dim), laid out by numpy's
  own transpose; each checkpoint element must decode to the coordinate the
  definition names (paged cache, Sec. 2.1; token ranges, Sec. 4.2), and the
  same for restore (Sec. 4.3) with checkpoint rows coded by their coordinate;
* a library special case: torch's advanced indexing over a shaped pool view
  (and index_put_ for restore) gives the same bytes;
* invariants: restore after checkpoint round-trips, bytes outside the named
  slots never change, checkpoints of successive deltas concatenate to the
  checkpoint of their union, token-major and head-major pools holding the same
  logical values give the same checkpoint, and relabelling physical blocks
  leaves the checkpoint unchanged;
* the row plan is an exclusive prefix sum (itertools.accumulate);
* error codes on crafted bad inputs.

Each pin is a plain function taking the oracle's ctypes library so that the
mutation test can run the same pins against an oracle with a planted mistake.
"""
from __future__ import annotations

import itertools
import math

import numpy as np
import torch

import oracle
from paper_2606_17787_amd.workloads import CacheShape, HND, NHD


# ---------------------------------------------------------------- helpers

def logical_dims(shape: CacheShape, nb: int):
    return (shape.num_layers, 2, nb, shape.block_size, shape.num_kv_heads,
            shape.head_dim)


def to_physical(logical: np.ndarray, order: str) -> np.ndarray:
    """[L,2,NB,bs,H,D] logical array -> flat pool in the given order."""
    if order == HND:
        logical = logical.transpose(0, 1, 2, 4, 3, 5)
    return np.ascontiguousarray(logical).reshape(-1)


def to_logical(flat: np.ndarray, shape: CacheShape, nb: int) -> np.ndarray:
    L, H, D, bs = (shape.num_layers, shape.num_kv_heads, shape.head_dim,
                   shape.block_size)
    if shape.order == HND:
        return flat.reshape(L, 2, nb, H, bs, D).transpose(0, 1, 2, 4, 3, 5)
    return flat.reshape(L, 2, nb, bs, H, D)


def word(shape):
    return oracle.word_dtype(shape)


def sentinel(shape):
    """A value no coordinate code takes: the word's maximum."""
    return np.iinfo(word(shape)).max


def coded_pool(shape: CacheShape, nb: int) -> np.ndarray:
    dims = logical_dims(shape, nb)
    n = math.prod(dims)
    assert n < sentinel(shape), "coordinate codes must fit the element"
    return to_physical(np.arange(n, dtype=word(shape)).reshape(dims),
                       shape.order)


def first_rows(start, end, row_base=0, req_row_base=None):
    """Each request's first checkpoint row: exclusive scan of the lengths."""
    n = [max(int(e) - int(s), 0) if int(s) >= 0 else 0
         for s, e in zip(start, end)]
    if req_row_base is not None:
        return [int(b) + int(s) for b, s in zip(req_row_base, start)]
    return list(itertools.accumulate(n, initial=row_base))[:len(n)]


def _signed(shape):
    """torch has no unsigned 16/32-bit tensors: move the bits as signed."""
    return {1: np.uint8, 2: np.int16, 4: np.int32}[shape.elem_bytes]


def random_words(rng, shape, n):
    w = word(shape)
    return rng.integers(0, np.iinfo(w).max, n, dtype=w, endpoint=True)


def torch_gather(shape: CacheShape, nb: int, flat: np.ndarray, bt, start,
                 end) -> np.ndarray:
    """Checkpoint rows by torch advanced indexing, in request order."""
    L, H, D, bs = (shape.num_layers, shape.num_kv_heads, shape.head_dim,
                   shape.block_size)
    t = torch.from_numpy(flat.view(_signed(shape)).copy())
    if shape.order == HND:
        view = t.view(L, 2, nb, H, bs, D).permute(2, 4, 0, 1, 3, 5)
    else:
        view = t.view(L, 2, nb, bs, H, D).permute(2, 3, 0, 1, 4, 5)
    parts = []
    for r in range(len(start)):
        tok = torch.arange(int(start[r]), int(end[r]))
        b = torch.from_numpy(np.asarray(bt[r], np.int64))[tok // bs]
        parts.append(view[b, tok % bs].reshape(len(tok), L * 2 * H * D))
    out = torch.cat(parts) if parts else torch.zeros(
        0, L * 2 * H * D, dtype=torch.from_numpy(np.zeros(1, _signed(shape))).dtype)
    return out.numpy().view(word(shape))


def torch_scatter(shape: CacheShape, nb: int, flat: np.ndarray, bt, start,
                  end, ckpt: np.ndarray) -> np.ndarray:
    L, H, D, bs = (shape.num_layers, shape.num_kv_heads, shape.head_dim,
                   shape.block_size)
    t = torch.from_numpy(flat.view(_signed(shape)).copy())
    if shape.order == HND:
        view = t.view(L, 2, nb, H, bs, D).permute(2, 4, 0, 1, 3, 5)
    else:
        view = t.view(L, 2, nb, bs, H, D).permute(2, 3, 0, 1, 4, 5)
    ck = torch.from_numpy(ckpt.view(_signed(shape)).reshape(-1, L, 2, H, D))
    row = 0
    for r in range(len(start)):
        tok = torch.arange(int(start[r]), int(end[r]))
        b = torch.from_numpy(np.asarray(bt[r], np.int64))[tok // bs]
        view.index_put_((b, tok % bs), ck[row:row + len(tok)])
        row += len(tok)
    return t.numpy().view(word(shape))


def random_table(rng, R, cols, nb, fill_all=True):
    perm = rng.permutation(nb)[:R * cols]
    bt = np.full((R, cols), -1, np.int32)
    bt.reshape(-1)[:perm.size] = perm
    return bt


# ------------------------------------------------------------------- pins

def pin_plan_prefix_sum(lib):
    rng = np.random.default_rng(11)
    for R in (0, 1, 2, 7, 64, 1000):
        s = rng.integers(0, 50, R).astype(np.int32)
        e = (s + rng.integers(0, 20, R)).astype(np.int32)
        for base in (0, 5, 1 << 33):
            st, fr, tot = oracle.plan(s, e, base, lib=lib)
            assert st == oracle.OK
            assert list(fr) == first_rows(s, e, base)
            assert tot == int((e.astype(np.int64) - s).sum())
        rb = rng.integers(0, 1 << 40, R)
        st, fr, _ = oracle.plan(s, e, 0, rb, lib=lib)
        assert st == oracle.OK and list(fr) == first_rows(s, e, 0, rb)
    # an invalid range contributes no rows and is a RANGE error
    st, fr, tot = oracle.plan([0, 5, 2], [3, 4, 6], 0, lib=lib)
    assert st == oracle.ERR_RANGE and list(fr) == [0, 3, 3] and tot == 7
    st, _, _ = oracle.plan([-1], [2], 0, lib=lib)
    assert st == oracle.ERR_RANGE


def check_decoded_pack(shape, nb, bt, s, e, lib, row_base=0):
    """Pack a coordinate-coded pool and decode every checkpoint element."""
    L, H, D, bs = (shape.num_layers, shape.num_kv_heads, shape.head_dim,
                   shape.block_size)
    pool = coded_pool(shape, nb)
    n = int(np.sum(np.asarray(e, np.int64) - np.asarray(s, np.int64)))
    rows = row_base + n + 1  # one spare row that must stay untouched
    ck = np.full((rows, L * 2 * H * D), sentinel(shape), word(shape))
    st, ck = oracle.pack(shape, nb, pool, bt, s, e, row_base, ckpt=ck,
                         lib=lib)
    assert st == oracle.OK, st
    dims = logical_dims(shape, nb)
    li, kvi, hi, di = np.meshgrid(np.arange(L), np.arange(2), np.arange(H),
                                  np.arange(D), indexing="ij")
    fr = first_rows(s, e, row_base)
    touched = np.zeros(rows, bool)
    for r in range(len(s)):
        for t in range(int(s[r]), int(e[r])):
            row = fr[r] + t - int(s[r])
            touched[row] = True
            got = ck[row].reshape(L, 2, H, D)
            assert int(got.max()) < math.prod(dims), "unwritten element"
            l, kv, b, slot, h, d = np.unravel_index(got.astype(np.int64), dims)
            assert np.array_equal(l, li) and np.array_equal(kv, kvi)
            assert np.array_equal(h, hi) and np.array_equal(d, di)
            assert np.all(b == bt[r][t // bs]) and np.all(slot == t % bs)
    assert np.all(ck[~touched] == sentinel(shape))


def check_decoded_unpack(shape, nb, bt, s, e, lib):
    """Unpack coordinate-coded checkpoint rows and decode every pool slot."""
    L, H, D, bs = (shape.num_layers, shape.num_kv_heads, shape.head_dim,
                   shape.block_size)
    n = int(np.sum(np.asarray(e, np.int64) - np.asarray(s, np.int64)))
    cdims = (n, L, 2, H, D)
    assert math.prod(cdims) < sentinel(shape)
    ck = np.arange(math.prod(cdims), dtype=word(shape)).reshape(n, L * 2 * H * D)
    pool = np.full(shape.pool_elems(nb), sentinel(shape), word(shape))
    st = oracle.unpack(shape, nb, pool, bt, s, e, ck, lib=lib)
    assert st == oracle.OK, st
    lg = to_logical(pool, shape, nb)
    li, kvi, hi, di = np.meshgrid(np.arange(L), np.arange(2), np.arange(H),
                                  np.arange(D), indexing="ij")
    named = np.zeros((nb, bs), bool)
    fr = first_rows(s, e)
    for r in range(len(s)):
        for t in range(int(s[r]), int(e[r])):
            b, slot = int(bt[r][t // bs]), t % bs
            named[b, slot] = True
            got = lg[:, :, b, slot]  # [L,2,H,D]
            assert int(got.max()) < math.prod(cdims), "unwritten slot"
            row, l, kv, h, d = np.unravel_index(got.astype(np.int64), cdims)
            assert np.all(row == fr[r] + t - int(s[r]))
            assert np.array_equal(l, li) and np.array_equal(kv, kvi)
            assert np.array_equal(h, hi) and np.array_equal(d, di)
    rest = lg.transpose(2, 3, 0, 1, 4, 5)[~named]
    assert np.all(rest == sentinel(shape))


TINY_SHAPES = [CacheShape(1, 1, 8, bs, o) for bs in (1, 2, 3) for o in (NHD, HND)] + \
    [CacheShape(2, 2, 8, 2, o) for o in (NHD, HND)] + \
    [CacheShape(1, 2, 16, 4, o) for o in (NHD, HND)] + \
    [CacheShape(2, 3, 4, 3, o, elem_bytes=4) for o in (NHD, HND)] + \
    [CacheShape(1, 1, 16, 1, o, elem_bytes=1) for o in (NHD, HND)]


def pin_bruteforce_decode(lib, exhaustive=True):
    """Every injective single-request table over a 4-block pool and every
    range 0 <= s <= e <= cols*bs; sampled two-request cases."""
    rng = np.random.default_rng(12)
    nb, cols = 4, 2
    for shape in TINY_SHAPES:
        bs = shape.block_size
        tables = list(itertools.permutations(range(nb), cols))
        if not exhaustive:
            tables = tables[::5]
        for tab in tables:
            bt = np.array([tab], np.int32)
            for s in range(cols * bs + 1):
                for e in range(s, cols * bs + 1):
                    check_decoded_pack(shape, nb, bt, [s], [e], lib)
                    check_decoded_unpack(shape, nb, bt, [s], [e], lib)
        for _ in range(40 if exhaustive else 8):
            bt = random_table(rng, 2, cols, nb)
            s = rng.integers(0, cols * bs + 1, 2)
            e = np.array([rng.integers(x, cols * bs + 1) for x in s])
            check_decoded_pack(shape, nb, bt, s, e, lib,
                               row_base=int(rng.integers(0, 3)))
            check_decoded_unpack(shape, nb, bt, s, e, lib)


def _random_case(rng, shape, R, nb, max_tok, incremental=False):
    bs = shape.block_size
    cols = -(-max_tok // bs)
    assert R * cols <= nb
    bt = random_table(rng, R, cols, nb)
    if incremental:
        s = rng.integers(0, max_tok, R)
        e = np.minimum(s + rng.integers(0, 2 * bs + 2, R), max_tok)
    else:
        s = np.zeros(R, np.int64)
        e = rng.integers(0, max_tok + 1, R)
    return bt, s.astype(np.int32), e.astype(np.int32)


MEDIUM_SHAPES = [CacheShape(3, 2, 16, 4, NHD), CacheShape(3, 2, 16, 4, HND),
                 CacheShape(2, 4, 8, 16, NHD), CacheShape(2, 4, 8, 16, HND),
                 CacheShape(1, 3, 24, 5, NHD), CacheShape(1, 3, 24, 5, HND),
                 CacheShape(2, 2, 32, 4, NHD, elem_bytes=1),
                 CacheShape(2, 3, 32, 4, HND, elem_bytes=1),
                 CacheShape(2, 2, 4, 4, NHD, elem_bytes=4),
                 CacheShape(1, 3, 8, 5, HND, elem_bytes=4)]


def pin_torch_indexing(lib):
    rng = np.random.default_rng(13)
    for shape in MEDIUM_SHAPES:
        for inc in (False, True):
            nb = 64
            bt, s, e = _random_case(rng, shape, 5, nb, 40, inc)
            pool = random_words(rng, shape, shape.pool_elems(nb))
            st, ck = oracle.pack(shape, nb, pool, bt, s, e, lib=lib)
            assert st == oracle.OK
            assert np.array_equal(ck, torch_gather(shape, nb, pool, bt, s, e))
            dst = random_words(rng, shape, shape.pool_elems(nb))
            bt2 = random_table(rng, *bt.shape, nb)
            want = torch_scatter(shape, nb, dst, bt2, s, e, ck)
            assert oracle.unpack(shape, nb, dst, bt2, s, e, ck,
                                 lib=lib) == oracle.OK
            assert np.array_equal(dst, want)


def pin_invariants(lib):
    rng = np.random.default_rng(14)
    for shape in MEDIUM_SHAPES:
        nb, R, max_tok = 96, 6, 60
        bs = shape.block_size
        bt, _, e_full = _random_case(rng, shape, R, nb, max_tok)
        pool = random_words(rng, shape, shape.pool_elems(nb))
        s_full = np.zeros(R, np.int32)
        st, full = oracle.pack(shape, nb, pool, bt, s_full, e_full, lib=lib)
        assert st == oracle.OK
        assert full.shape == (int(e_full.sum()), shape.token_row_elems)

        # deltas: split every range into 3 random consecutive pieces
        cuts = np.sort(rng.integers(0, e_full[:, None] + 1, (R, 2)), axis=1)
        bounds = np.concatenate([np.zeros((R, 1), np.int64), cuts,
                                 e_full[:, None]], axis=1)
        stride = max_tok + 1
        per_req = np.zeros((R * stride, shape.token_row_elems), word(shape))
        steps = []
        for k in range(3):
            s_k, e_k = bounds[:, k].astype(np.int32), bounds[:, k + 1].astype(np.int32)
            st, part = oracle.pack(shape, nb, pool, bt, s_k, e_k, lib=lib)
            assert st == oracle.OK
            steps.append(part)
            st, _ = oracle.pack(shape, nb, pool, bt, s_k, e_k,
                                req_row_base=np.arange(R) * stride,
                                ckpt=per_req, lib=lib)
            assert st == oracle.OK
        # per-request append rows == the full checkpoint, request by request
        fr = first_rows(s_full, e_full)
        for r in range(R):
            n = int(e_full[r])
            assert np.array_equal(per_req[r * stride:r * stride + n],
                                  full[fr[r]:fr[r] + n])
        # packed deltas, regrouped by request, == the full checkpoint
        regrouped = []
        for r in range(R):
            for k in range(3):
                frk = first_rows(bounds[:, k], bounds[:, k + 1])
                n = int(bounds[r, k + 1] - bounds[r, k])
                regrouped.append(steps[k][frk[r]:frk[r] + n])
        assert np.array_equal(np.concatenate(regrouped), full)

        # round trip into a fresh table; untouched bytes unchanged
        dst0 = random_words(rng, shape, shape.pool_elems(nb))
        bt2 = random_table(rng, R, bt.shape[1], nb)
        s2 = rng.integers(0, e_full + 1).astype(np.int32)
        st, ck = oracle.pack(shape, nb, pool, bt, s2, e_full, lib=lib)
        dst = dst0.copy()
        assert oracle.unpack(shape, nb, dst, bt2, s2, e_full, ck,
                             lib=lib) == oracle.OK
        st, back = oracle.pack(shape, nb, dst, bt2, s2, e_full, lib=lib)
        assert st == oracle.OK and np.array_equal(back, ck)
        lg0, lg1 = to_logical(dst0, shape, nb), to_logical(dst, shape, nb)
        named = np.zeros((nb, bs), bool)
        for r in range(R):
            for t in range(int(s2[r]), int(e_full[r])):
                named[bt2[r][t // bs], t % bs] = True
        a = lg0.transpose(2, 3, 0, 1, 4, 5)
        b = lg1.transpose(2, 3, 0, 1, 4, 5)
        assert np.array_equal(a[~named], b[~named])

        # the same logical values in the other layout give the same bytes
        other = CacheShape(shape.num_layers, shape.num_kv_heads,
                           shape.head_dim, bs,
                           NHD if shape.order == HND else HND,
                           shape.elem_bytes)
        lg = to_logical(pool, shape, nb)
        st, ck_other = oracle.pack(other, nb, to_physical(lg, other.order), bt,
                                   s_full, e_full, lib=lib)
        assert st == oracle.OK and np.array_equal(ck_other, full)

        # relabelling physical blocks consistently changes nothing
        pi = rng.permutation(nb)
        lg_perm = np.empty_like(lg)
        lg_perm[:, :, pi] = lg
        bt_perm = np.where(bt >= 0, pi[np.maximum(bt, 0)], -1).astype(np.int32)
        st, ck_perm = oracle.pack(shape, nb, to_physical(lg_perm, shape.order),
                                  bt_perm, s_full, e_full, lib=lib)
        assert st == oracle.OK and np.array_equal(ck_perm, full)


def pin_error_codes(lib):
    shape = CacheShape(2, 2, 8, 4, NHD)
    nb = 8
    pool = np.zeros(shape.pool_elems(nb), np.uint16)
    bt = np.array([[0, 1, 2], [3, 4, -1]], np.int32)

    def st_pack(s, e, bt=bt, rows=None, base=0, rb=None):
        # the buffer has slack past the stated capacity, so an oracle that
        # ignored the capacity would write there instead of out of bounds
        rows = 64 if rows is None else rows
        ck = np.zeros((rows + 8, shape.token_row_elems), np.uint16)
        return oracle.pack(shape, nb, pool, bt, s, e, row_base=base,
                           req_row_base=rb, ckpt=ck, ckpt_rows=rows,
                           lib=lib)[0]

    assert st_pack([0, 0], [12, 8]) == oracle.OK
    assert st_pack([0, 0], [13, 8]) == oracle.ERR_RANGE      # past the table
    assert st_pack([0, 0], [12, 9]) == oracle.ERR_BLOCK_ID   # -1 entry
    assert st_pack([3, 0], [2, 8]) == oracle.ERR_RANGE       # end < start
    assert st_pack([-1, 0], [2, 8]) == oracle.ERR_RANGE
    bad = np.array([[0, 8, 2], [3, 4, -1]], np.int32)
    assert st_pack([0, 0], [8, 1], bt=bad) == oracle.ERR_BLOCK_ID
    assert st_pack([0, 0], [5, 1], bt=bad) == oracle.ERR_BLOCK_ID
    assert st_pack([0, 0], [4, 1], bt=bad) == oracle.OK       # page 1 unread
    assert st_pack([0, 0], [12, 8], rows=20) == oracle.OK
    assert st_pack([0, 0], [12, 8], rows=19) == oracle.ERR_CAPACITY
    assert st_pack([0, 0], [12, 8], rows=25, base=5) == oracle.OK
    assert st_pack([0, 0], [12, 8], rows=25, base=6) == oracle.ERR_CAPACITY
    assert st_pack([2, 0], [4, 1], rows=100, rb=[-2, 0]) == oracle.OK
    assert st_pack([2, 0], [4, 1], rows=100, rb=[-3, 0]) == oracle.ERR_CAPACITY
    # the most negative code wins when several occur
    assert st_pack([0, 0], [13, 9], rows=1) == oracle.ERR_CAPACITY
    assert st_pack([5, 0], [4, 9]) == oracle.ERR_BLOCK_ID
    # nothing is written on error
    ck = np.full((30, shape.token_row_elems), 7, np.uint16)
    st, ck = oracle.pack(shape, nb, pool, bt, [0, 0], [12, 9], ckpt=ck,
                         lib=lib)
    assert st == oracle.ERR_BLOCK_ID and np.all(ck == 7)
    # empty requests are legal anywhere, even past the table
    assert st_pack([40, 3], [40, 3]) == oracle.OK


def validate_by_tokens(bs, nb, bt, start, end):
    """Validate-mode status written from its definition, token by token: a
    request's written pages are the pages of its tokens; a physical block
    named by two distinct (request, page) pairs is a duplicate."""
    codes = [oracle.OK]
    pages = set()
    for r, (s, e) in enumerate(zip(start, end)):
        if s < 0 or e < s:
            codes.append(oracle.ERR_RANGE)
            continue
        for t in range(s, e):
            j = t // bs
            if j >= len(bt[r]):
                codes.append(oracle.ERR_RANGE)
            elif not 0 <= bt[r][j] < nb:
                codes.append(oracle.ERR_BLOCK_ID)
            else:
                pages.add((r, j))
    for x, y in itertools.combinations(sorted(pages), 2):
        if bt[x[0]][x[1]] == bt[y[0]][y[1]]:
            codes.append(oracle.ERR_DUP_BLOCK)
    return min(codes)


def pin_validate_targets(lib, exhaustive=True):
    # every 2x2 table over entries {-1..3} with a pool of 3 blocks (entry 3
    # is outside it), against sampled ranges, for three block sizes
    nb, R, cols = 3, 2, 2
    rng = np.random.default_rng(23)
    for bs in (1, 2, 3):
        shape = CacheShape(1, 1, 8, bs, NHD)
        cap = cols * bs
        spans = [(s, e) for s in range(cap + 2) for e in range(s, cap + 2)]
        spans += [(-1, 2), (2, 1)]
        tables = list(itertools.product(range(-1, 4), repeat=R * cols))
        if not exhaustive:
            tables = [tables[i] for i in rng.choice(len(tables), 60, False)]
        for flat in tables:
            bt = np.array(flat, np.int32).reshape(R, cols)
            for _ in range(6):
                (s0, e0), (s1, e1) = (spans[i] for i in
                                      rng.choice(len(spans), 2))
                want = validate_by_tokens(bs, nb, bt.tolist(), [s0, s1],
                                          [e0, e1])
                got = oracle.validate_targets(shape, nb, bt, [s0, s1],
                                              [e0, e1], lib=lib)
                assert got == want, (bs, flat, (s0, e0, s1, e1), got, want)
    # larger cases: injective tables validate; one planted duplicate among
    # the written pages is caught, one among unwritten pages is not; and
    # whenever validation passes, unpack then pack round-trips
    for shape in MEDIUM_SHAPES[:4]:
        for trial in range(6):
            R, nb, max_tok = 9, 90, 37
            bt, s, e = _random_case(rng, shape, R, nb, max_tok,
                                    incremental=trial % 2 == 1)
            bs = shape.block_size
            assert oracle.validate_targets(shape, nb, bt, s, e,
                                           lib=lib) == oracle.OK
            written = [(r, j) for r in range(R) if e[r] > s[r]
                       for j in range(s[r] // bs, (e[r] - 1) // bs + 1)]
            unwritten = [(r, j) for r in range(R) for j in range(bt.shape[1])
                         if (r, j) not in set(written) and bt[r, j] >= 0]
            ck = random_words(rng, shape,
                              int((e - s).sum()) * shape.token_row_elems)
            pool = random_words(rng, shape, shape.pool_elems(nb))
            assert oracle.unpack(shape, nb, pool, bt, s, e, ck,
                                 lib=lib) == oracle.OK
            st, back = oracle.pack(shape, nb, pool, bt, s, e, lib=lib)
            assert st == oracle.OK and np.array_equal(back.reshape(-1), ck)
            if len(written) >= 2:
                a, b = (written[i] for i in rng.choice(len(written), 2, False))
                dup = bt.copy()
                dup[b] = dup[a]
                assert oracle.validate_targets(shape, nb, dup, s, e,
                                               lib=lib) == oracle.ERR_DUP_BLOCK
            if written and unwritten:
                a = written[rng.integers(len(written))]
                b = unwritten[rng.integers(len(unwritten))]
                dup = bt.copy()
                dup[b] = dup[a]
                assert oracle.validate_targets(shape, nb, dup, s, e,
                                               lib=lib) == oracle.OK


ALL_PINS = [pin_plan_prefix_sum, pin_bruteforce_decode, pin_torch_indexing,
            pin_invariants, pin_error_codes, pin_validate_targets]
