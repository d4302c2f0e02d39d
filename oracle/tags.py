"""CPU oracle for page tags and the longest checkpointed prefix.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the library, with which it shares no
code.

What it computes (LUMEN Sec. 4.2, page tags; Sec. 4.3, KV-reuse recovery):
  * Page i of a request holds tokens [i*bs, (i+1)*bs).  Its tag pairs a hash
    of the token IDs stored in the page with the page's end position, the
    request's token count after the page, (i+1)*bs.
  * A tag is regenerated from the token history alone, so any worker can
    recompute it.
  * A page becomes visible in the checkpoint store only once its payload has
    been received completely; a transfer cut short leaves it invisible.
  * Recovery regenerates the tags of pages 0, 1, ... and stops at the first
    page that is not visible or whose stored tag differs: the pages before
    it are the longest contiguous checkpointed prefix, and the tokens after
    it are recomputed by a partial prefill.

Readings (the paper names neither the hash nor partial pages):
  * hash = BLAKE2b with an 8-byte digest (RFC 7693, unkeyed) over the page's
    token IDs as little-endian int32, read as a little-endian uint64;
  * only complete pages carry tags, so the reusable prefix is a whole number
    of pages, and a partial last page is recomputed with the suffix.
"""
from __future__ import annotations

import hashlib
from typing import Dict, Iterable, List, Tuple

import numpy as np

Tag = Tuple[int, int]  # (hash, end position)


def page_hash(token_ids: Iterable[int]) -> int:
    """BLAKE2b-64 of the token IDs (little-endian int32)."""
    data = np.asarray(list(token_ids), dtype="<i4").tobytes()
    return int.from_bytes(hashlib.blake2b(data, digest_size=8).digest(),
                          "little")


def page_tags(tokens, block_size: int, first_page: int = 0,
              last_page: int | None = None) -> List[Tag]:
    """Tags of the complete pages first_page .. last_page - 1 (default: every
    complete page) of a token history."""
    tokens = list(tokens)
    complete = len(tokens) // block_size
    last = complete if last_page is None else last_page
    if not 0 <= first_page <= last <= complete:
        raise ValueError("pages must be complete pages of the history")
    out = []
    for i in range(first_page, last):
        page = tokens[i * block_size:(i + 1) * block_size]
        out.append((page_hash(page), (i + 1) * block_size))
    return out


class TagStore:
    """A holder's checkpoint store, reduced to what recovery reads: the tag
    of every page that has been received completely, per request."""

    def __init__(self, block_size: int):
        self.block_size = block_size
        self.pages: Dict[int, Dict[int, Tag]] = {}

    def publish(self, request: int, page: int, tag: Tag) -> None:
        """Called once page `page` of `request` has fully arrived."""
        self.pages.setdefault(request, {})[page] = tag

    def release(self, request: int) -> None:
        self.pages.pop(request, None)

    def longest_prefix(self, request: int, tokens) -> int:
        """Tokens of the longest contiguous checkpointed prefix."""
        have = self.pages.get(request, {})
        tags = page_tags(tokens, self.block_size)
        n = 0
        while n < len(tags) and have.get(n) == tags[n]:
            n += 1
        return n * self.block_size


def received_pages(received_tokens: int, block_size: int) -> int:
    """Pages wholly inside a received prefix of token rows."""
    return received_tokens // block_size
