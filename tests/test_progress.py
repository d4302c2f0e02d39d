"""Checkpoint progress (LUMEN Sec. 4.2): the oracle against its pins, then
the native tracker against the oracle, on the CPU.

Pins: over any sequence of growing histories the sent ranges of a request
tile [0, final length) without gap or overlap; a shorter history re-sends
from its new end; unknown requests start at 0; release forgets."""
import numpy as np
import pytest

from oracle import progress as O
from paper_2606_17787_amd import kvckpt as kv
from paper_2606_17787_amd import progress as N


def pin_progress(make):
    rng = np.random.default_rng(21)
    # growing histories: the ranges tile [0, final) exactly
    p = make()
    lens = {r: 0 for r in range(6)}
    covered = {r: [] for r in range(6)}
    for step in range(30):
        ids = sorted(rng.choice(6, int(rng.integers(1, 7)), replace=False))
        for r in ids:
            lens[r] += int(rng.integers(0, 20))
        s, e = p.ranges(ids, [lens[r] for r in ids])
        for r, a, b in zip(ids, s, e):
            covered[r].append((int(a), int(b)))
    for r in range(6):
        pos = 0
        for a, b in covered[r]:
            assert a == pos and b >= a
            pos = b
        assert pos == lens[r] and p.sent(r) == lens[r]
    # a history cut back (rejected speculative tokens) re-sends its tail
    p = make()
    p.ranges([1], [40])
    assert [list(x) for x in p.ranges([1], [33])] == [[33], [33]]
    assert [list(x) for x in p.ranges([1], [45])] == [[33], [45]]
    # unknown requests start at 0; release forgets
    assert [list(x) for x in p.ranges([9, 1], [5, 45])] == [[0, 45], [5, 45]]
    p.release(9)
    assert p.sent(9) == 0
    assert [list(x) for x in p.ranges([9], [7])] == [[0], [7]]


def test_oracle_pins():
    pin_progress(O.Progress)


@pytest.mark.parametrize("mutant", ["no_cut_back", "resend_all", "skip_one"])
def test_pins_catch_planted_mistakes(mutant, monkeypatch):
    real = O.Progress.ranges

    def ranges(self, ids, lengths):
        if mutant == "no_cut_back":
            s = [self.done.get(int(r), 0) for r in ids]
            for r, n in zip(ids, lengths):
                self.done[int(r)] = max(self.done.get(int(r), 0), int(n))
            return s, [int(n) for n in lengths]
        s, e = real(self, ids, lengths)
        if mutant == "resend_all":
            return [0] * len(s), e
        return [x + 1 if x < y else x for x, y in zip(s, e)], e

    monkeypatch.setattr(O.Progress, "ranges", ranges)
    with pytest.raises(AssertionError):
        pin_progress(O.Progress)


def test_native_passes_the_same_pins():
    pin_progress(N.Progress)


def test_native_matches_oracle_on_random_batches():
    rng = np.random.default_rng(5)
    a, b = N.Progress(), O.Progress()
    lens = {}
    for step in range(400):
        ids = rng.choice(50, int(rng.integers(0, 20)), replace=False)
        for r in ids:
            lens[r] = max(0, lens.get(r, 0) + int(rng.integers(-5, 30)))
        ln = [lens[r] for r in ids]
        sa, ea = a.ranges(ids, ln)
        sb, eb = b.ranges(ids, ln)
        assert sa.tolist() == sb and ea.tolist() == eb
        if rng.random() < 0.1 and lens:
            r = int(rng.choice(list(lens)))
            a.release(r)
            b.release(r)
            lens.pop(r)
    for r in range(50):
        assert a.sent(r) == b.sent(r)


def test_native_rejects_bad_batches():
    p = N.Progress()
    with pytest.raises(kv.LumenError):
        p.ranges([1, 1], [3, 4])
    with pytest.raises(kv.LumenError):
        p.ranges([1], [-1])
    assert p.sent(1) == 0  # nothing changed
