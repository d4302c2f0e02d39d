"""CPU oracle for draft-state alignment.

TEST INFRASTRUCTURE ONLY: imported by the tests, never by the library.

What it computes (LUMEN Sec. 4.4, draft-state alignment): after each
decode step the paired surviving worker sends the newly committed tokens of
every mirror request.  The recovering worker compares them with its local
draft tokens position by position (not by value: tokens recur); its draft
KV stays valid only up to the first mismatched position.  From there on the
draft KV is truncated and the remaining committed tokens are replayed
through the draft model.

Readings, where the paper gives no data layout:
  * per request: draft tokens d[0, draft_len), committed tokens
    c[0, committed_len), and the draft KV computed for positions
    [0, kv_len) in the pages of a block table (page j holds positions
    [j*bs, (j+1)*bs));
  * p = the first i < min(draft_len, committed_len) with d[i] != c[i], or
    that minimum when there is none; the KV stays valid for
    valid = min(kv_len, p) positions, and committed_len - valid committed
    tokens are replayed;
  * truncation frees the pages the valid prefix no longer reaches, pages
    ceil(valid/bs) .. ceil(kv_len/bs) - 1: their table entries become -1
    and their block ids (entries < 0 are skipped) are listed in request
    order, then page order;
  * a request whose lengths are inconsistent (negative, past its arrays, or
    kv_len past its table) is a RANGE error and is left unchanged, with
    nothing to replay;
  * if more than freed_cap pages are freed (CAPACITY), only the first
    freed_cap are listed and cleared; the others stay in their tables, so
    no block is lost.
"""
from __future__ import annotations

import numpy as np

OK, ERR_RANGE, ERR_CAPACITY = 0, -5, -7


def align(draft, draft_len, committed, committed_len, kv_len, block_tables,
          block_size, freed_cap):
    """Returns (status, new_kv_len, replay, freed, tables, total): freed
    lists at most freed_cap block ids, total counts them all, and tables is
    the truncated copy of block_tables."""
    draft = np.asarray(draft)
    committed = np.asarray(committed)
    bt = np.array(block_tables, dtype=np.int32, copy=True)
    R = bt.shape[0]
    new_len = np.array(kv_len, dtype=np.int32, copy=True)
    replay = np.zeros(R, np.int32)
    freed = []
    total = 0
    status = OK
    for r in range(R):
        dl, cl, kl = int(draft_len[r]), int(committed_len[r]), int(kv_len[r])
        if (dl < 0 or cl < 0 or kl < 0 or dl > draft.shape[1]
                or cl > committed.shape[1] or kl > bt.shape[1] * block_size):
            status = min(status, ERR_RANGE)
            continue
        lim = min(dl, cl)
        p = lim
        for i in range(lim):
            if draft[r, i] != committed[r, i]:
                p = i
                break
        valid = min(kl, p)
        new_len[r] = valid
        replay[r] = cl - valid
        for j in range(-(-valid // block_size), -(-kl // block_size)):
            if bt[r, j] >= 0:
                total += 1
                if len(freed) < freed_cap:
                    freed.append(int(bt[r, j]))
                    bt[r, j] = -1
    if total > freed_cap:
        status = min(status, ERR_CAPACITY)
    return status, new_len, replay, np.array(freed, np.int32), bt, total
