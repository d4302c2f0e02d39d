"""Checkpoint placement (Sec. 4.2, Eq. 1) and recovery scheduling (Sec. 4.3):
the oracle against its pins, then the native scheduler against the oracle,
on the CPU.

The paper prints no worked example for the scheduler, so the pins are
examples computed by hand from Eq. 1 and the rebalancing rule, special
cases that reduce to a plain minimum, and invariants of the rule (budgets
never exceeded, load conserved, no legal move left, smallest checkpoints
shed first).  Planted mistakes in the oracle are caught."""
import itertools

import numpy as np
import pytest

from oracle import sched as O
from paper_2606_17787_amd import kvckpt as kv
from paper_2606_17787_amd import sched as N


class OracleSched(O.Scheduler):
    def set_worker(self, w, q, queued=0, running=0):
        self.w[w].q, self.w[w].queued, self.w[w].running = q, queued, running

    def holder(self, r):
        return self.req[r].holder

    def reserved(self, w):
        return self.w[w].used


# ------------------------------------------------------------------ pins

def pin_hand_placement(make):
    # 3 workers, 100 B budgets, 10 B/s, lambda 1; q = 0.5, 0.1, 0.3
    s = make([100, 100, 100], 10.0, 1.0)
    for w, q in enumerate((0.5, 0.1, 0.3)):
        s.set_worker(w, q)
    # r1 (serving 0, 40 B): w1 0.1 + 40/10 = 4.1, w2 0.3 + 4 = 4.3 -> 1
    assert s.place(1, 0, 40) == 1
    # r2 (serving 0, 10 B): w1 0.1 + (40+10)/2/10 = 2.6, w2 0.3 + 1 = 1.3 -> 2
    assert s.place(2, 0, 10) == 2
    # r3 (serving 1, 70 B): w0 0.5 + 7 = 7.5, w2 0.3 + (10+70)/2/10 = 4.3 -> 2
    assert s.place(3, 1, 70) == 2
    # r4 (serving 2, 80 B): w1 has 60 B free, not in F; w0 0.5 + 8 -> 0
    assert s.place(4, 2, 80) == 0
    # r5 (serving 0, 50 B): w1 60 free -> 0.1 + (40+50)/2/10 = 4.6;
    # w2 has 20 free -> not in F -> 1
    assert s.place(5, 0, 50) == 1
    # r6 (serving 1, 30 B): w0 20 free, w2 20 free -> nobody
    assert s.place(6, 1, 30) == -1
    assert [s.reserved(w) for w in range(3)] == [80, 90, 80]
    s.release(5)
    assert [s.reserved(w) for w in range(3)] == [80, 40, 80]
    # worker 0 fails: r1 (holder 1) and r2 (holder 2) reuse; r4 loses its
    # holder (worker 0) but keeps running on worker 2
    out = s.recover([0])
    assert out == [(1, 1, True), (2, 2, True)]
    assert s.holder(4) == -1 and s.holder(3) == 2
    assert [s.reserved(w) for w in range(3)] == [0, 0, 70]


def pin_hand_rebalance(make):
    # 4 workers; worker 0 holds the checkpoints of 6 requests served by
    # worker 3; loads before the failure: w0 4, w1 1, w2 0 (queued+running)
    s = make([1000] * 4, 1.0, 0.0)
    s.set_worker(0, 0.0, 3, 1)
    s.set_worker(1, 1.0, 0, 1)
    s.set_worker(2, 1.0, 0, 0)
    s.set_worker(3, 9.0, 0, 6)
    for r in range(6):
        assert s.place(r, 3, 10) == 0   # lambda 0: lowest q among 0..2
        s.set_persisted(r, [50, 10, 40, 30, 20, 60][r])
    # dispatch: all 6 reuse on worker 0 -> loads w0 10, w1 1, w2 0;
    # average 11/3 = 3.67.  Moves (w0 sheds smallest persisted first):
    #  r1 (10) -> w2 [9,1,1]; r4 (20) -> w1 [8,2,1]; r3 (30) -> w2 [7,2,2];
    #  r2 (40) -> w1 [6,3,2]; r0 (50) -> w2 [5,3,3]; r5 (60) -> w1 [4,4,3]
    # w0 is at 4 > 3.67 but has nothing left to move -> stop
    out = s.recover([3])
    assert out == [(0, 2, False), (1, 2, False), (2, 1, False),
                   (3, 2, False), (4, 1, False), (5, 1, False)]


def pin_no_cycle(make):
    # loads [5, 4, 4] after dispatch against an average of 4.33: moving one
    # request would only swap roles, so nothing moves
    s = make([1000] * 4, 1.0, 0.0)
    s.set_worker(0, 0.0, 4, 0)
    s.set_worker(1, 1.0, 4, 0)
    s.set_worker(2, 1.0, 4, 0)
    s.set_worker(3, 9.0, 0, 1)
    assert s.place(7, 3, 5) == 0
    assert s.recover([3]) == [(7, 0, True)]


def pin_special_cases(make):
    rng = np.random.default_rng(3)
    for trial in range(30):
        nw = int(rng.integers(2, 7))
        budgets = rng.integers(0, 400, nw).tolist()
        lam = 0.0 if trial % 2 else 1e9
        s = make(budgets, 7.0, lam)
        qs = rng.random(nw).round(3).tolist()
        for w in range(nw):
            s.set_worker(w, qs[w])
        used = [0] * nw
        held = [[] for _ in range(nw)]
        for r in range(12):
            serving = int(rng.integers(0, nw))
            size = int(rng.integers(1, 120))
            feas = [w for w in range(nw)
                    if w != serving and budgets[w] - used[w] >= size]
            h = s.place(r, serving, size)
            if not feas:
                assert h == -1
                continue
            if lam == 0.0:   # Eq. 1 reduces to the least queueing delay
                want = min(feas, key=lambda w: (qs[w], w))
            else:            # restore pressure dominates
                want = min(feas, key=lambda w: (
                    (sum(held[w]) + size) / (len(held[w]) + 1), qs[w], w))
            assert h == want and h != serving
            used[h] += size
            held[h].append(size)
            assert s.reserved(h) == used[h] <= budgets[h]


def pin_rebalance_invariants(make):
    rng = np.random.default_rng(9)
    for trial in range(40):
        nw = int(rng.integers(2, 7))
        s = make([10**6] * nw, 1.0, float(rng.integers(0, 2)))
        base = {}
        for w in range(nw):
            qd, qq, rr = float(rng.random()), int(rng.integers(0, 6)), \
                int(rng.integers(0, 6))
            s.set_worker(w, qd, qq, rr)
            base[w] = qq + rr
        serving = {}
        for r in range(int(rng.integers(1, 25))):
            serving[r] = int(rng.integers(0, nw))
            s.place(r, serving[r], int(rng.integers(1, 100)))
            s.set_persisted(r, int(rng.integers(0, 1000)))
        holder = {r: s.holder(r) for r in serving}
        k = int(rng.integers(1, nw))
        failed = sorted(rng.choice(nw, k, replace=False).tolist())
        out = s.recover(failed)
        alive = [w for w in range(nw) if w not in failed]
        hit = sorted(r for r in serving if serving[r] in failed)
        assert [r for r, _, _ in out] == hit
        load = {w: base[w] for w in alive}
        for r, w, reuse in out:
            assert w in alive
            load[w] += 1
            if reuse:  # only at its own, surviving holder
                assert w == holder[r]
        avg = (sum(base[w] for w in alive) + len(hit)) / len(alive)
        # nothing left that the rule could legally move
        dst = min(alive, key=lambda w: (load[w], w))
        for src in alive:
            if load[src] > avg and any(w == src for _, w, _ in out):
                assert load[dst] + 1 >= load[src]


def pin_all(make):
    pin_hand_placement(make)
    pin_hand_rebalance(make)
    pin_no_cycle(make)
    pin_special_cases(make)
    pin_rebalance_invariants(make)


def test_oracle_pins():
    pin_all(OracleSched)


def _mutant(name, monkeypatch):
    real_pressure = O.Scheduler.pressure
    if name == "pressure_ignores_new_request":
        monkeypatch.setattr(O.Scheduler, "pressure", lambda self, w, r: (
            (sum(self.w[w].held.values()) / max(len(self.w[w].held), 1))
            / self.bw))
    elif name == "pressure_not_averaged":
        monkeypatch.setattr(O.Scheduler, "pressure", lambda self, w, r: (
            (sum(self.w[w].held.values()) + r) / self.bw))
    elif name == "serving_worker_allowed":
        real_place = O.Scheduler.place

        def place(self, request, serving, reserved):
            return real_place(self, request, -1, reserved)
        monkeypatch.setattr(O.Scheduler, "place", place)
    elif name == "largest_checkpoint_moves_first":
        src = O.Scheduler.recover

        def recover(self, failed):
            for rq in self.req.values():
                rq.persisted = -rq.persisted
            return src(self, failed)
        monkeypatch.setattr(O.Scheduler, "recover", recover)
    elif name == "dead_holder_reused":
        real_recover = O.Scheduler.recover

        def recover(self, failed):
            keep = {r: rq.holder for r, rq in self.req.items()}
            out = real_recover(self, failed)
            return [(r, keep[r] if keep[r] >= 0 else w, keep[r] >= 0)
                    for r, w, _ in out]
        monkeypatch.setattr(O.Scheduler, "recover", recover)


@pytest.mark.parametrize("mutant", ["pressure_ignores_new_request",
                                    "pressure_not_averaged",
                                    "serving_worker_allowed",
                                    "largest_checkpoint_moves_first",
                                    "dead_holder_reused"])
def test_pins_catch_planted_mistakes(mutant, monkeypatch):
    _mutant(mutant, monkeypatch)
    with pytest.raises(AssertionError):
        pin_all(OracleSched)


# -------------------------------------------------- native vs the oracle

def test_native_passes_the_same_pins():
    pin_all(N.Scheduler)


def test_native_matches_oracle_on_random_histories():
    rng = np.random.default_rng(2025)
    for trial in range(80):
        nw = int(rng.integers(1, 9))
        budgets = rng.integers(0, 2000, nw).tolist()
        bw, lam = float(rng.choice([1.0, 26e9, 3.0])), \
            float(rng.choice([0.0, 0.5, 1.0, 4.0]))
        a, b = N.Scheduler(budgets, bw, lam), OracleSched(budgets, bw, lam)
        live, nxt = set(), 0
        for step in range(int(rng.integers(5, 60))):
            op = int(rng.integers(0, 10))
            if op < 5:
                serving = int(rng.integers(0, nw))
                size = int(rng.integers(0, 600))
                if not b.w[serving].alive:
                    continue
                assert a.place(nxt, serving, size) == b.place(nxt, serving,
                                                              size)
                live.add(nxt)
                nxt += 1
            elif op == 5 and live:
                r = int(rng.choice(sorted(live)))
                a.release(r)
                b.release(r)
                live.discard(r)
            elif op == 6 and live:
                r = int(rng.choice(sorted(live)))
                n = int(rng.integers(0, 10**6))
                a.set_persisted(r, n)
                b.set_persisted(r, n)
            elif op == 7:
                w = int(rng.integers(0, nw))
                q = float(rng.random() * 3)
                qq, rr = int(rng.integers(0, 9)), int(rng.integers(0, 9))
                a.set_worker(w, q, qq, rr)
                b.set_worker(w, q, qq, rr)
            elif op == 8:
                k = int(rng.integers(1, nw + 1))
                failed = sorted(rng.choice(nw, k, replace=False).tolist())
                assert a.recover(failed) == b.recover(failed), trial
            for w in range(nw):
                assert a.reserved(w) == b.reserved(w)
            for r in live:
                assert a.holder(r) == b.holder(r)


def test_native_argument_errors():
    with pytest.raises(kv.LumenError):
        N.Scheduler([], 1.0)
    with pytest.raises(kv.LumenError):
        N.Scheduler([10], 0.0)
    s = N.Scheduler([10, 10], 1.0)
    with pytest.raises(kv.LumenError):
        s.place(1, 5, 1)          # unknown serving worker
    s.place(1, 0, 1)
    with pytest.raises(kv.LumenError):
        s.place(1, 0, 1)          # the request already has a holder
    with pytest.raises(kv.LumenError):
        s.release(99)
    with pytest.raises(kv.LumenError):
        s.recover([7])
