"""Draft-state alignment on the GPU against the oracle (LUMEN Sec. 4.4):
new KV lengths, replay counts, freed block lists and truncated tables
bit for bit, across request counts that span many wavefronts and scan
threads, mismatches anywhere (or nowhere), the capacity limit of the freed
list and requests with inconsistent lengths."""
import numpy as np
import pytest
import torch

from oracle import draft as D
import paper_2606_17787_amd.kvckpt as kv

from gpu_util import dev, h2d

pytestmark = pytest.mark.gpu


def case(rng, R, cols, bs, bt_extra=2):
    base = rng.integers(0, 50000, (R, cols)).astype(np.int32)
    draft, committed = base.copy(), base.copy()
    for r in range(R):
        p = int(rng.integers(0, cols + 8))
        if p < cols:
            committed[r, p:] = rng.integers(50000, 60000, cols - p)
    dl = rng.integers(0, cols + 1, R).astype(np.int32)
    cl = rng.integers(0, cols + 1, R).astype(np.int32)
    kl = rng.integers(0, cols + 1, R).astype(np.int32)
    btc = -(-cols // bs) + bt_extra
    bt = rng.permutation(R * btc + 9)[:R * btc].reshape(R, btc).astype(np.int32)
    bt[rng.random(bt.shape) < 0.05] = -1
    return draft, dl, committed, cl, kl, bt


def run_gpu(draft, dl, committed, cl, kl, bt, bs, cap):
    R = bt.shape[0]
    d_kl, d_bt = h2d(kl), h2d(bt)
    replay = torch.full((R,), -7, dtype=torch.int32, device=dev())
    freed = torch.full((max(cap, 1),), -9, dtype=torch.int32, device=dev())
    count = torch.zeros(1, dtype=torch.int64, device=dev())
    ws = kv.new_workspace(R, dev())
    kv.lumen_kv_draft_align(h2d(draft), h2d(dl), h2d(committed), h2d(cl),
                            d_kl, d_bt, bs, replay, freed[:cap], count, ws)
    st = kv.lumen_kv_ckpt_status(ws)
    return (st, d_kl.cpu().numpy(), replay.cpu().numpy(),
            freed.cpu().numpy(), d_bt.cpu().numpy(), int(count.item()))


@pytest.mark.parametrize("R", [1, 5, 64, 65, 300, 1025, 5000])
@pytest.mark.parametrize("bs", [1, 4, 16])
def test_draft_align_matches_oracle(R, bs):
    rng = np.random.default_rng(R * 31 + bs)
    cols = 150 if R <= 300 else 40
    draft, dl, committed, cl, kl, bt = case(rng, R, cols, bs)
    for cap in (10**7, 3):
        want = D.align(draft, dl, committed, cl, kl, bt, bs, cap)
        st, k, rp, fr, tab, tot = run_gpu(draft, dl, committed, cl, kl, bt,
                                          bs, cap)
        st_o, k_o, rp_o, fr_o, tab_o, tot_o = want
        assert st == st_o, (cap, st, st_o)
        assert np.array_equal(k, k_o)
        assert np.array_equal(rp, rp_o)
        assert tot == tot_o
        n = len(fr_o)
        assert np.array_equal(fr[:n], fr_o) and (fr[n:] == -9).all()
        assert np.array_equal(tab, tab_o)


def test_draft_align_range_errors_and_empty():
    rng = np.random.default_rng(2)
    draft, dl, committed, cl, kl, bt = case(rng, 6, 30, 4)
    dl[2] = 31            # past the draft array
    kl[4] = bt.shape[1] * 4 + 1   # past the table
    cl[5] = -1
    want = D.align(draft, dl, committed, cl, kl, bt, 4, 1000)
    got = run_gpu(draft, dl, committed, cl, kl, bt, 4, 1000)
    assert got[0] == want[0] == kv.LUMEN_ERR_RANGE
    for a, b in zip(got[1:3], want[1:3]):
        assert np.array_equal(a, b)
    assert np.array_equal(got[4], want[4])
    # no requests at all: nothing freed, OK
    ws = kv.new_workspace(0, dev())
    e = torch.zeros(0, dtype=torch.int32, device=dev())
    count = torch.full((1,), 5, dtype=torch.int64, device=dev())
    kv.lumen_kv_draft_align(e.view(0, 0), e, e.view(0, 0), e, e, e.view(0, 0),
                            4, e, e, count, ws)
    assert kv.lumen_kv_ckpt_status(ws) == 0 and count.item() == 0
