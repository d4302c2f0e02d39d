"""Page tags and the longest checkpointed prefix (LUMEN Sec. 4.2, page tags;
Sec. 4.3, KV-reuse recovery): the oracle against its pins, then the native
store against the oracle, on the CPU.

Pins of the oracle: its hash primitive reproduces RFC 7693's worked example;
tag end positions have a closed form; a page's tag depends on its own
tokens only; the longest prefix equals a brute-force maximum over candidate
prefix lengths, and has closed forms for a transfer cut at any byte and for
a history that changed at any token.  Planted mistakes in the oracle are
caught by these pins."""
import hashlib
import itertools
import os
import threading

import numpy as np
import pytest

from oracle import tags as O
from paper_2606_17787_amd import kvckpt as kv
from paper_2606_17787_amd import tags as T

GOLDEN = os.path.join(os.path.dirname(__file__), "golden",
                      "blake2b_rfc7693.txt")


# ------------------------------------------------------------ oracle pins

def test_hash_primitive_matches_rfc7693_example():
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        msg, digest = line.split()
        assert hashlib.blake2b(msg.encode()).hexdigest() == digest


def prefix_by_max(tag_of, have, tokens, bs):
    """Longest prefix as a maximum over candidate lengths k: every page
    below k is published with the tag regenerated from the history."""
    complete = len(tokens) // bs
    best = 0
    for k in range(complete + 1):
        if all(have.get(i) == tag_of(tokens, i) for i in range(k)):
            best = k
    return best * bs


def pin_tags(page_tags, store_cls):
    rng = np.random.default_rng(8)
    # end positions: (i + 1) * bs for every complete page, none for a tail
    for bs in (1, 3, 16):
        for n in (0, 1, bs - 1, bs, 5 * bs + 2):
            tok = rng.integers(0, 50000, n).tolist()
            tags = page_tags(tok, bs)
            assert [e for _, e in tags] == [(i + 1) * bs
                                           for i in range(n // bs)]
    # locality: changing one token changes the tag of its page only
    bs = 4
    tok = rng.integers(0, 50000, 6 * bs).tolist()
    base = page_tags(tok, bs)
    for pos in range(len(tok)):
        t2 = list(tok)
        t2[pos] += 1
        new = page_tags(t2, bs)
        changed = [i for i in range(6) if new[i] != base[i]]
        assert changed == [pos // bs], (pos, changed)
    # the same tokens at another position: same hash, different end
    rep = tok[:bs] * 3
    tags = page_tags(rep, bs)
    assert len({h for h, _ in tags}) == 1 and len({e for _, e in tags}) == 3
    # longest prefix vs a brute-force maximum, every publish subset of a
    # 4-page history, with and without one foreign page
    hist = rng.integers(0, 50000, 4 * bs + 2).tolist()
    other = rng.integers(0, 50000, 4 * bs).tolist()
    tag_of = lambda t, i: page_tags(t, bs)[i]
    for mask in range(16):
        for foreign in (None, 0, 2):
            st = store_cls(bs)
            have = {}
            for i in range(4):
                if mask >> i & 1:
                    tg = tag_of(other if foreign == i else hist, i)
                    st.publish(7, i, tg)
                    have[i] = tg
            assert st.longest_prefix(7, hist) == prefix_by_max(
                tag_of, have, hist, bs), (mask, foreign)
            assert st.longest_prefix(8, hist) == 0
    # a transfer cut after b bytes of token rows: floor(floor(b/row)/bs) pages
    row = 96
    for cut in range(0, 4 * bs * row + 1, 37):
        st = store_cls(bs)
        got_rows = cut // row
        for i in range(O.received_pages(got_rows, bs)):
            st.publish(1, i, tag_of(hist, i))
        assert st.longest_prefix(1, hist) == (got_rows // bs) * bs
    # a history that changed at token p (rejected draft tokens): the pages
    # before p's page survive, later ones no longer match
    for p in range(len(hist)):
        st = store_cls(bs)
        for i in range(4):
            st.publish(3, i, tag_of(hist, i))
        h2 = list(hist)
        h2[p] = h2[p] + 1
        assert st.longest_prefix(3, h2) == min(p // bs, 4) * bs
    # release forgets everything
    st = store_cls(bs)
    st.publish(5, 0, tag_of(hist, 0))
    st.release(5)
    assert st.longest_prefix(5, hist) == 0


class OracleStore(O.TagStore):
    def publish(self, request, page, tag):
        super().publish(request, page, tag)


def test_oracle_pins():
    pin_tags(O.page_tags, OracleStore)


@pytest.mark.parametrize("mutant", ["end_is_start", "page_shifted",
                                    "prefix_skips_gap", "whole_tail_page"])
def test_pins_catch_planted_mistakes(mutant, monkeypatch):
    real_tags, real_prefix = O.page_tags, O.TagStore.longest_prefix

    def tags_end_is_start(tokens, bs, first=0, last=None):
        return [(h, e - bs) for h, e in real_tags(tokens, bs, first, last)]

    def tags_page_shifted(tokens, bs, first=0, last=None):
        t = list(tokens)
        out = []
        for i in range(len(t) // bs):
            out.append((O.page_hash(t[i * bs + 1:(i + 1) * bs + 1]),
                        (i + 1) * bs))
        return out

    def prefix_skips_gap(self, request, tokens):
        have = self.pages.get(request, {})
        tags = O.page_tags(tokens, self.block_size)
        return sum(have.get(i) == tg for i, tg in enumerate(tags)) * \
            self.block_size

    def tags_whole_tail(tokens, bs, first=0, last=None):
        t = list(tokens)
        n = -(-len(t) // bs)
        return [(O.page_hash(t[i * bs:(i + 1) * bs]), (i + 1) * bs)
                for i in range(n)]

    if mutant == "end_is_start":
        monkeypatch.setattr(O, "page_tags", tags_end_is_start)
    elif mutant == "page_shifted":
        monkeypatch.setattr(O, "page_tags", tags_page_shifted)
    elif mutant == "prefix_skips_gap":
        monkeypatch.setattr(O.TagStore, "longest_prefix", prefix_skips_gap)
    else:
        monkeypatch.setattr(O, "page_tags", tags_whole_tail)
    with pytest.raises(AssertionError):
        pin_tags(O.page_tags, OracleStore)


# ------------------------------------------------ native store vs oracle

class NativeStore(T.TagStore):
    def publish(self, request, page, tag):
        super().publish(request, page, tag[0], tag[1])


def native_tags(tokens, bs):
    return [(int(h), int(e)) for h, e in T.lumen_page_tags(tokens, bs)]


def test_native_passes_the_same_pins():
    pin_tags(native_tags, NativeStore)


@pytest.mark.parametrize("bs", [1, 2, 7, 16, 32, 33, 64, 100])
def test_native_tags_match_oracle(bs):
    rng = np.random.default_rng(bs)
    for n in (0, 1, bs - 1, bs, 3 * bs + 1, 17 * bs):
        tok = rng.integers(-2**31, 2**31, n, dtype=np.int64).astype(np.int32)
        complete = n // bs
        for a, b in ((0, complete), (complete // 2, complete),
                     (complete, complete)):
            got = T.lumen_page_tags(tok, bs, a, b)
            want = O.page_tags(tok.tolist(), bs, a, b)
            assert [(int(h), int(e)) for h, e in got] == want


def test_native_argument_errors():
    tok = np.arange(10, dtype=np.int32)
    for args in ((tok, 0), (tok, 4, 0, 3), (tok, 4, 2, 1), (tok, 4, -1, 1)):
        with pytest.raises(kv.LumenError):
            T.lumen_page_tags(*args)
    st = T.TagStore(4)
    with pytest.raises(kv.LumenError):
        st.publish(1, 0, 123, 5)      # end must be (page + 1) * block_size
    with pytest.raises(kv.LumenError):
        st.publish(1, -1, 123, 0)
    with pytest.raises(kv.LumenError):
        st.publish_pages(1, tok, 0, 3)  # page 2 is not complete
    # page indices past INT32_MAX are refused before (page + 1) * block_size
    # is formed or any page vector grows
    for page in ((1 << 31), (1 << 62), (1 << 63) - 1):
        with pytest.raises(kv.LumenError) as e:
            st.publish(1, page, 123, ((page + 1) * 4) % (1 << 63))
        assert e.value.code == kv.LUMEN_ERR_INVALID_ARG
    assert st.pages(1) == 0
    with pytest.raises(kv.LumenError):
        T.TagStore(0)


def test_native_store_random_scenarios_match_oracle():
    """Random sequences of transfers (in order, out of order, cut short),
    histories that diverge, and releases, on both stores."""
    rng = np.random.default_rng(2024)
    for trial in range(60):
        bs = int(rng.choice([1, 4, 16, 32]))
        nat, ora = T.TagStore(bs), O.TagStore(bs)
        hist = {r: rng.integers(0, 1 << 17, int(rng.integers(0, 12 * bs)))
                .astype(np.int32) for r in range(5)}
        for _ in range(40):
            r = int(rng.integers(0, 5))
            h = hist[r]
            complete = len(h) // bs
            op = rng.integers(0, 5)
            if op <= 1 and complete:
                a = int(rng.integers(0, complete))
                b = int(rng.integers(a, complete + 1))
                nat.publish_pages(r, h, a, b)
                for i, tg in enumerate(O.page_tags(h.tolist(), bs, a, b)):
                    ora.publish(r, a + i, tg)
            elif op == 2 and len(h):
                p = int(rng.integers(0, len(h)))
                h = h.copy()
                h[p] ^= 1 + int(rng.integers(0, 1000))
                hist[r] = h
            elif op == 3:
                nat.release(r)
                ora.release(r)
            for q in range(5):
                assert nat.longest_prefix(q, hist[q]) == \
                    ora.longest_prefix(q, hist[q].tolist()), (trial, q)
                assert nat.pages(q) == len(ora.pages.get(q, {}))


def test_native_store_concurrent_publish_and_lookup():
    """Receivers publish pages of disjoint requests from several threads
    while a reader looks prefixes up; the final answers equal the oracle's
    and every answer seen on the way is a whole number of pages no longer
    than the final one."""
    bs = 16
    rng = np.random.default_rng(5)
    hist = {r: rng.integers(0, 1 << 17, 64 * bs + 5).astype(np.int32)
            for r in range(8)}
    nat = T.TagStore(bs)
    seen = {r: [] for r in hist}
    stop = threading.Event()

    def receiver(rs):
        for r in rs:
            for p in range(64):
                nat.publish_pages(r, hist[r], p, p + 1)

    def reader():
        while not stop.is_set():
            for r in hist:
                seen[r].append(nat.longest_prefix(r, hist[r]))

    rd = threading.Thread(target=reader)
    rd.start()
    ws = [threading.Thread(target=receiver, args=(rs,))
          for rs in ([0, 1], [2, 3], [4, 5], [6, 7])]
    for t in ws:
        t.start()
    for t in ws:
        t.join()
    stop.set()
    rd.join()
    for r in hist:
        assert nat.longest_prefix(r, hist[r]) == 64 * bs
        assert all(v % bs == 0 and v <= 64 * bs for v in seen[r])
        assert seen[r] == sorted(seen[r])  # pages only ever arrive
