"""CPU oracle for LUMEN's scheduling decisions (checkpoint placement,
recovery dispatch, load rebalancing).

TEST INFRASTRUCTURE ONLY: imported by the tests, never by the library, with
which it shares no code.

What it computes:
  * Placement (Sec. 4.2, checkpoint placement, Eq. 1).  Each active request
    r has one checkpoint holder.  The candidates F(r) are the workers whose
    free host memory can take r's reserved checkpoint footprint (sized from
    the maximum context length), excluding the worker serving r.  Worker w
    scores q_w + lambda * p_w(r).  q_w is its queueing delay.  p_w(r) is the
    mean reserved footprint of the checkpoints w would hold with r added,
    divided by a fixed host-to-GPU bandwidth.  The holder minimises the
    score; the footprint is reserved on assignment and released when the
    request completes.
  * Recovery dispatch (Sec. 4.3).  An interrupted request goes to its
    checkpoint holder for KV reuse.  If the holder has failed too, the
    request is recomputed on the least-loaded surviving worker.
  * Load rebalancing (Sec. 4.3, average-based request-count rule).  A
    worker's load is its queued + running + newly assigned interrupted
    requests; the average is taken after the initial dispatch.  The most
    congested worker sheds its assigned interrupted requests to the
    least-loaded worker, smallest checkpointed size first, and loads are
    recomputed after every move, until no worker exceeds the average.  A
    moved request loses its checkpoint and is recomputed.
  * Several failures (Sec. 4.3, multi-worker failures) are one recovery
    event over all their interrupted requests.

Readings where the paper is silent:
  * ties go to the lowest worker index (placement, least-loaded choices);
  * F(r) empty: the request gets no checkpoint and is recomputed if its
    worker fails;
  * with integer loads the rule as stated need not terminate ([5, 4, 4]
    against an average of 4.33 would move one request back and forth), so
    a request moves only if the target's load plus one stays below the
    source's load; among overloaded workers the most loaded one holding a
    movable request goes first (ties: lowest index);
  * interrupted requests are dispatched in increasing request id;
  * the movable requests of a worker are the interrupted requests assigned
    to it; a request that is already recomputed counts as checkpointed size
    0, so it moves before any request that would reuse a checkpoint;
  * a surviving request whose holder failed keeps running without a
    checkpoint (its reservation is gone with the holder);
  * once recovered, a request's old checkpoint is released (it now runs on
    its holder, or has been recomputed), and the caller places a new one;
  * with no survivor at all, a request is reported with worker -1 and stays
    on its failed worker, so the next recovery event reports it again.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple


@dataclass
class Worker:
    limit: int                 # host-memory budget for checkpoints, bytes
    q: float = 0.0             # queueing delay, seconds
    queued: int = 0
    running: int = 0
    alive: bool = True
    used: int = 0              # reserved bytes
    held: Dict[int, int] = field(default_factory=dict)  # request -> bytes


@dataclass
class Request:
    serving: int
    reserved: int
    holder: int = -1
    persisted: int = 0         # checkpointed bytes so far


class Scheduler:
    def __init__(self, limits: List[int], h2d_bytes_per_s: float,
                 lam: float = 1.0):
        self.w = [Worker(limit=int(x)) for x in limits]
        self.bw = float(h2d_bytes_per_s)
        self.lam = float(lam)
        self.req: Dict[int, Request] = {}

    # ---------------------------------------------------------- placement
    def pressure(self, w: int, reserved: int) -> float:
        held = self.w[w].held
        mean = (sum(held.values()) + reserved) / (len(held) + 1)
        return mean / self.bw

    def place(self, request: int, serving: int, reserved: int) -> int:
        best, best_score = -1, None
        for i, wk in enumerate(self.w):
            if i == serving or not wk.alive:
                continue
            if wk.limit - wk.used < reserved:
                continue
            score = wk.q + self.lam * self.pressure(i, reserved)
            if best_score is None or score < best_score:
                best, best_score = i, score
        self.req[request] = Request(serving=serving, reserved=reserved,
                                    holder=best)
        if best >= 0:
            self.w[best].used += reserved
            self.w[best].held[request] = reserved
        return best

    def set_persisted(self, request: int, nbytes: int) -> None:
        self.req[request].persisted = nbytes

    def release(self, request: int) -> None:
        r = self.req.pop(request)
        if r.holder >= 0 and request in self.w[r.holder].held:
            self.w[r.holder].used -= r.reserved
            del self.w[r.holder].held[request]

    # ----------------------------------------------------------- recovery
    def load(self, w: int, assigned: Dict[int, List[int]]) -> int:
        wk = self.w[w]
        return wk.queued + wk.running + len(assigned.get(w, []))

    def recover(self, failed: List[int]) -> List[Tuple[int, int, bool]]:
        """Returns (request, worker, reuse) for every interrupted request,
        in increasing request id."""
        for f in failed:
            self.w[f].alive = False
        # checkpoints held by failed workers are lost
        for f in failed:
            for rq in list(self.w[f].held):
                self.req[rq].holder = -1
            self.w[f].held.clear()
            self.w[f].used = 0
        alive = [i for i, wk in enumerate(self.w) if wk.alive]
        interrupted = sorted(r for r, rq in self.req.items()
                             if not self.w[rq.serving].alive)
        assigned: Dict[int, List[int]] = {}
        reuse: Dict[int, bool] = {}
        where: Dict[int, int] = {}
        for r in interrupted:
            h = self.req[r].holder
            if h >= 0 and self.w[h].alive:
                tgt, ok = h, True
            elif alive:
                tgt = min(alive, key=lambda i: (self.load(i, assigned), i))
                ok = False
            else:  # no survivor at all
                tgt, ok = -1, False
            assigned.setdefault(tgt, []).append(r)
            reuse[r], where[r] = ok, tgt
        # rebalancing against the average after the initial dispatch
        if alive:
            avg = sum(self.load(i, assigned) for i in alive) / len(alive)
            while True:
                loads = {i: self.load(i, assigned) for i in alive}
                dst = min(alive, key=lambda i: (loads[i], i))
                moved = False
                for src in sorted(alive, key=lambda i: (-loads[i], i)):
                    if loads[src] <= avg:
                        break
                    movable = [r for r in assigned.get(src, [])]
                    if not movable or loads[dst] + 1 >= loads[src]:
                        continue
                    r = min(movable, key=lambda x: (
                        self.req[x].persisted if reuse[x] else 0, x))
                    assigned[src].remove(r)
                    assigned.setdefault(dst, []).append(r)
                    reuse[r], where[r] = False, dst
                    moved = True
                    break
                if not moved:
                    break
        for r in interrupted:
            rq = self.req[r]
            if rq.holder >= 0:
                wk = self.w[rq.holder]
                wk.used -= rq.reserved
                del wk.held[r]
            rq.holder = -1
            if where[r] >= 0:
                rq.serving = where[r]
            rq.persisted = 0
        return [(r, where[r], reuse[r]) for r in interrupted]
