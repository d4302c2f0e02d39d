"""CPU oracle for checkpoint progress.

TEST INFRASTRUCTURE ONLY: imported by the tests, never by the library.

What it computes (LUMEN Sec. 4.2, incremental checkpoint pipeline): workers
track checkpoint progress and send only the KV that is new since the last
checkpoint.  Per request, `sent` is the number of leading tokens already
handed to the pipeline; a batch whose KV covers `length` tokens sends
[min(sent, length), length) and then sent = length.  A shorter history
(rejected speculative tokens) lowers sent, so the rewritten tail is sent
again.
"""
from __future__ import annotations

from typing import Dict, Sequence, Tuple


class Progress:
    def __init__(self):
        self.done: Dict[int, int] = {}

    def ranges(self, ids: Sequence[int],
               lengths: Sequence[int]) -> Tuple[list, list]:
        ids, lengths = [int(x) for x in ids], [int(x) for x in lengths]
        if len(set(ids)) != len(ids) or any(n < 0 for n in lengths):
            raise ValueError("repeated id or negative length")
        start, end = [], []
        for r, n in zip(ids, lengths):
            start.append(min(self.done.get(r, 0), n))
            end.append(n)
            self.done[r] = n
        return start, end

    def sent(self, request: int) -> int:
        return self.done.get(request, 0)

    def release(self, request: int) -> None:
        self.done.pop(request, None)
