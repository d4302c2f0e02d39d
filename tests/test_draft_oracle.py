"""Draft-state alignment oracle (LUMEN Sec. 4.4) against its pins, on the
CPU: the first mismatch by an independent numpy route, the paper's own
scenario of accepted and rejected draft tokens, positional (not value)
matching, conservation of blocks, and closed forms for the freed pages.
Planted mistakes are caught."""
import numpy as np
import pytest

from oracle import draft as D


def first_mismatch_numpy(d, c, lim):
    ne = np.asarray(d[:lim]) != np.asarray(c[:lim])
    return int(np.argmax(ne)) if ne.any() else lim


def random_case(rng, R=9, cols=40, bs=4):
    dl = rng.integers(0, cols + 1, R)
    cl = rng.integers(0, cols + 1, R)
    base = rng.integers(0, 30, (R, cols))
    draft = base.copy()
    committed = base.copy()
    for r in range(R):   # diverge at a random position, or never
        p = int(rng.integers(0, cols + 5))
        if p < cols:
            committed[r, p:] = rng.integers(30, 60, cols - p)
    kl = np.minimum(rng.integers(0, cols + 1, R), cols)
    btc = -(-cols // bs)
    bt = rng.permutation(R * btc + 5)[:R * btc].reshape(R, btc).astype(np.int32)
    bt[rng.random(bt.shape) < 0.1] = -1
    return (draft.astype(np.int32), dl.astype(np.int32),
            committed.astype(np.int32), cl.astype(np.int32),
            kl.astype(np.int32), bt, bs)


def pin_draft(align):
    rng = np.random.default_rng(4)
    # the paper's scenario: a history of 37 committed tokens; the draft
    # model proposed K = 4 more; the target accepted 2 and corrected the 3rd
    hist = rng.integers(0, 1000, 37)
    prop = rng.integers(1000, 2000, 4)
    draft = np.concatenate([hist, prop])[None].astype(np.int32)
    committed = np.concatenate([hist, prop[:2], [5]])[None].astype(np.int32)
    bt = np.arange(11, dtype=np.int32)[None]
    st, kl, rp, freed, tab, tot = align(draft, [41], committed, [40], [41],
                                        bt, 4, 100)
    assert st == 0 and kl[0] == 39 and rp[0] == 1      # replay the correction
    # positions 0..38 stay: page 10 (positions 40..43) held position 40
    assert freed.tolist() == [10] and tot == 1 and tab[0, 10] == -1
    st, kl, rp, freed, tab, tot = align(draft, [41], committed, [40], [41],
                                        bt, 16, 100)
    assert kl[0] == 39 and freed.tolist() == [] and tot == 0
    # positional, not by value: the same tokens in another order differ at 2
    st, kl, rp, *_ = align(np.array([[5, 7, 5, 7]], np.int32), [4],
                           np.array([[5, 7, 7, 5]], np.int32), [4], [4],
                           np.array([[0]], np.int32), 4, 4)
    assert kl[0] == 2 and rp[0] == 2
    # random cases against the numpy route and closed forms
    for trial in range(200):
        draft, dl, committed, cl, kl0, bt, bs = random_case(rng)
        cap = int(rng.integers(0, 40))
        st, kl, rp, freed, tab, tot = align(draft, dl, committed, cl, kl0,
                                            bt, bs, cap)
        want_freed = []
        for r in range(bt.shape[0]):
            p = first_mismatch_numpy(draft[r], committed[r], min(dl[r], cl[r]))
            v = min(int(kl0[r]), p)
            assert kl[r] == v and rp[r] == cl[r] - v
            gone = range(-(-v // bs), -(-int(kl0[r]) // bs))
            want_freed += [int(bt[r, j]) for j in gone if bt[r, j] >= 0]
        assert tot == len(want_freed)
        assert freed.tolist() == want_freed[:cap]
        assert st == (0 if tot <= cap else D.ERR_CAPACITY)
        # no block lost or duplicated: listed + still in tables = before
        before = sorted(bt[bt >= 0].tolist())
        after = sorted(tab[tab >= 0].tolist() + freed.tolist())
        assert before == after
    # inconsistent lengths: RANGE, request untouched, others still aligned
    draft, dl, committed, cl, kl0, bt, bs = random_case(rng, R=3)
    dl[1] = draft.shape[1] + 1
    st, kl, rp, freed, tab, tot = align(draft, dl, committed, cl, kl0, bt,
                                        bs, 1000)
    assert st == D.ERR_RANGE and kl[1] == kl0[1] and (tab[1] == bt[1]).all()


def test_oracle_pins():
    pin_draft(D.align)


@pytest.mark.parametrize("mutant", ["mismatch_one_late", "floor_not_ceil",
                                    "replay_from_draft", "value_matching"])
def test_pins_catch_planted_mistakes(mutant, monkeypatch):
    real = D.align

    def wrapped(draft, dl, committed, cl, kl, bt, bs, cap):
        draft, committed = np.asarray(draft), np.asarray(committed)
        if mutant == "mismatch_one_late":
            # keeps the mismatched position itself as valid
            st, k, rp, fr, tab, tot = real(draft, dl, committed, cl, kl, bt,
                                           bs, cap)
            k, rp = k.copy(), rp.copy()
            for r in range(len(k)):
                lim = min(int(dl[r]), int(cl[r]), int(kl[r]))
                if k[r] < lim:
                    k[r] += 1
                    rp[r] -= 1
            return st, k, rp, fr, tab, tot
        if mutant == "floor_not_ceil":
            st, k, rp, fr, tab, tot = real(draft, dl, committed, cl, kl, bt,
                                           bs, cap)
            return st, k, rp, fr[:max(len(fr) - 1, 0)], tab, tot
        if mutant == "replay_from_draft":
            st, k, rp, fr, tab, tot = real(draft, dl, committed, cl, kl, bt,
                                           bs, cap)
            return st, k, np.asarray(dl) - k, fr, tab, tot
        # value matching: a token counts as matching if it occurs anywhere
        d2 = draft.copy()
        for r in range(d2.shape[0]):
            for i in range(d2.shape[1]):
                if d2[r, i] in committed[r]:
                    d2[r, i] = committed[r, i]
        return real(d2, dl, committed, cl, kl, bt, bs, cap)

    with pytest.raises(AssertionError):
        pin_draft(wrapped)
