"""Seeded synthetic inputs for the paged-KV checkpoint path.

This module only draws inputs: cache shapes, per-request context lengths,
per-step token ranges, and block tables built from random permutations of a
block pool. It holds none of the checkpoint arithmetic (no row offsets, no
gathers, no scatters), so both the CPU oracle's tests and the GPU path's
tests and benchmark can draw the same inputs from it without sharing any of
the method's code.

The five workloads follow the serving shapes the checkpoint path is measured
on: a tiny cache for exhaustive checks, a Llama-3-8B-shaped decode loop with
incremental deltas, a failure-restore burst into a fragmented pool, one
tensor-parallel rank's shard of a Llama-3-70B-shaped cache, and a Qwen-style
GQA cache in head-major layout.  The paper measures on serving traces and
model weights that are not available here; these seeded inputs stand in for
them with the same cache shapes and context-length mixes.

Block tables use -1 for pages a request never touches.  Draw order inside a
generator is fixed (context lengths, then deltas, then permutations) so a
seed reproduces every array bit for bit with numpy's PCG64.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import List, Optional, Tuple

import numpy as np

NHD = "NHD"  # cache [L][2][NB][block_size][H][D]
HND = "HND"  # cache [L][2][NB][H][block_size][D]


@dataclasses.dataclass(frozen=True)
class CacheShape:
    num_layers: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    order: str = NHD
    elem_bytes: int = 2

    @property
    def token_row_elems(self) -> int:
        """Elements in one token's checkpoint row (all layers, K and V)."""
        return self.num_layers * 2 * self.num_kv_heads * self.head_dim

    @property
    def token_row_bytes(self) -> int:
        return self.token_row_elems * self.elem_bytes

    def pool_elems(self, num_blocks: int) -> int:
        return (self.num_layers * 2 * num_blocks * self.block_size
                * self.num_kv_heads * self.head_dim)

    def pool_dims(self, num_blocks: int) -> Tuple[int, ...]:
        L, H, D, bs = (self.num_layers, self.num_kv_heads, self.head_dim,
                       self.block_size)
        if self.order == NHD:
            return (L, 2, num_blocks, bs, H, D)
        return (L, 2, num_blocks, H, bs, D)


@dataclasses.dataclass
class Workload:
    """One seeded workload: a source pool, per-step ranges, a destination."""
    name: str
    seed: int
    shape: CacheShape
    ctx: np.ndarray                   # int64 [R]: tokens present before step 0
    num_blocks: int                   # source pool size in blocks
    block_tables: np.ndarray          # int32 [R, cols] into the source pool
    starts: List[np.ndarray]          # per step, int32 [R]
    ends: List[np.ndarray]            # per step, int32 [R]
    dst_num_blocks: int               # destination pool size in blocks
    dst_block_tables: np.ndarray      # int32 [R, cols'] into the destination
    in_place: bool = False            # destination pool is the source pool
    occupied: Optional[np.ndarray] = None  # destination blocks held by others
    description: str = ""

    @property
    def num_reqs(self) -> int:
        return int(self.ctx.shape[0])

    @property
    def num_steps(self) -> int:
        return len(self.starts)

    def step_tokens(self, k: int) -> int:
        return int((self.ends[k].astype(np.int64)
                    - self.starts[k].astype(np.int64)).sum())

    def step_bytes_each_way(self, k: int) -> int:
        return self.step_tokens(k) * self.shape.token_row_bytes

    def fingerprint(self) -> str:
        h = hashlib.sha256()
        h.update(repr(dataclasses.astuple(self.shape)).encode())
        for a in ([self.ctx, self.block_tables, self.dst_block_tables]
                  + self.starts + self.ends
                  + ([self.occupied] if self.occupied is not None else [])):
            h.update(np.ascontiguousarray(a).tobytes())
        h.update(f"{self.num_blocks},{self.dst_num_blocks}".encode())
        return h.hexdigest()


def _ceil_div(a, b):
    return -(-a // b)


def _tables_from_perm(perm: np.ndarray, first_page: np.ndarray,
                      end_page: np.ndarray, cols: int) -> np.ndarray:
    """Request r takes the next (end_page[r] - first_page[r]) entries of perm
    for its pages first_page[r] .. end_page[r]-1; other entries are -1."""
    R = first_page.shape[0]
    bt = np.full((R, cols), -1, dtype=np.int32)
    pos = 0
    for r in range(R):
        n = int(end_page[r] - first_page[r])
        bt[r, first_page[r]:end_page[r]] = perm[pos:pos + n]
        pos += n
    assert pos <= perm.shape[0]
    return bt


def _lognormal_ctx(rng, R, median, sigma, lo, hi):
    x = rng.lognormal(np.log(median), sigma, R)
    return np.clip(np.rint(x), lo, hi).astype(np.int64)


def full_pack(name: str, seed: int, shape: CacheShape, ctx: np.ndarray,
              rng: np.random.Generator, pool_blocks: Optional[int] = None,
              in_place: bool = False, description: str = "") -> Workload:
    """Every request's whole context [0, ctx) is checkpointed in one step."""
    bs = shape.block_size
    pages = _ceil_div(ctx, bs)
    need = int(pages.sum())
    nb = need if pool_blocks is None else int(pool_blocks)
    assert nb >= need
    cols = int(pages.max()) if ctx.size else 1
    zeros = np.zeros_like(pages)
    bt = _tables_from_perm(rng.permutation(nb).astype(np.int32), zeros,
                           pages, cols)
    dst_nb = nb  # a fresh pool of the same size, or the same pool in place
    dst_bt = _tables_from_perm(rng.permutation(dst_nb).astype(np.int32),
                               zeros, pages, cols)
    s = np.zeros(ctx.shape[0], np.int32)
    e = ctx.astype(np.int32)
    return Workload(name, seed, shape, ctx, nb, bt, [s], [e], dst_nb, dst_bt,
                    in_place=in_place, description=description)


def incremental(name: str, seed: int, shape: CacheShape, ctx: np.ndarray,
                rng: np.random.Generator, steps: int, dmin: int, dmax: int,
                description: str = "") -> Workload:
    """Each step checkpoints every request's newest dmin..dmax tokens.

    The source pool holds every request's whole final context; the
    destination pool holds only the pages the steps touch."""
    R = ctx.shape[0]
    bs = shape.block_size
    deltas = rng.integers(dmin, dmax + 1, (steps, R)).astype(np.int64)
    cum = np.concatenate([np.zeros((1, R), np.int64), np.cumsum(deltas, 0)])
    final = ctx + cum[-1]
    pages = _ceil_div(final, bs)
    nb = int(pages.sum())
    cols = int(pages.max())
    bt = _tables_from_perm(rng.permutation(nb).astype(np.int32),
                           np.zeros_like(pages), pages, cols)
    first = ctx // bs
    dst_nb = int((pages - first).sum())
    dst_bt = _tables_from_perm(rng.permutation(dst_nb).astype(np.int32),
                               first, pages, cols)
    starts = [(ctx + cum[k]).astype(np.int32) for k in range(steps)]
    ends = [(ctx + cum[k + 1]).astype(np.int32) for k in range(steps)]
    return Workload(name, seed, shape, ctx, nb, bt, starts, ends, dst_nb,
                    dst_bt, description=description)


def restore_burst(name: str, seed: int, shape: CacheShape, ctx: np.ndarray,
                  rng: np.random.Generator, pool_blocks: int,
                  occupied_frac: float, description: str = "") -> Workload:
    """Interrupted requests restored from contiguous checkpoints into a pool
    that other requests already hold in part; free blocks are handed out in
    shuffled order.  The source side is the contiguous checkpoint itself, so
    block_tables is empty and num_blocks is 0."""
    R = ctx.shape[0]
    bs = shape.block_size
    n_occ = int(round(occupied_frac * pool_blocks))
    occupied = np.sort(rng.choice(pool_blocks, n_occ, replace=False))
    mask = np.ones(pool_blocks, bool)
    mask[occupied] = False
    free = rng.permutation(np.nonzero(mask)[0]).astype(np.int32)
    pages = _ceil_div(ctx, bs)
    cols = int(pages.max())
    dst_bt = np.full((R, cols), -1, dtype=np.int32)
    # Blocks are handed out in request order; a request whose pages no
    # longer fit starts a new wave that reuses the free list from the top.
    pos = 0
    for r in range(R):
        n = int(pages[r])
        if pos + n > free.shape[0]:
            pos = 0
        dst_bt[r, :n] = free[pos:pos + n]
        pos += n
    s = np.zeros(R, np.int32)
    e = ctx.astype(np.int32)
    return Workload(name, seed, shape, ctx, 0, np.zeros((R, 0), np.int32),
                    [s], [e], pool_blocks, dst_bt, occupied=occupied,
                    description=description)


def restore_waves(w: Workload) -> List[np.ndarray]:
    """Request indices of each restore wave: consecutive requests whose pages
    fit the free list together (the same rule restore_burst hands blocks
    out by)."""
    bs = w.shape.block_size
    n_free = w.dst_num_blocks - (0 if w.occupied is None else w.occupied.size)
    pages = _ceil_div(w.ctx, bs)
    waves, cur, used = [], [], 0
    for r in range(w.num_reqs):
        n = int(pages[r])
        if used + n > n_free:
            waves.append(np.array(cur, np.int64))
            cur, used = [], 0
        cur.append(r)
        used += n
    if cur:
        waves.append(np.array(cur, np.int64))
    return waves


# --------------------------------------------------------------------------
# The five workloads at their full sizes.  The `scale_*` keywords shrink a
# workload (fewer requests and steps, shorter contexts) while keeping its
# cache shape, for checks the CPU oracle must finish in seconds.

SHAPE_TINY = CacheShape(2, 2, 64, 16, NHD)
SHAPE_LLAMA3_8B = CacheShape(32, 8, 128, 16, NHD)
SHAPE_LLAMA3_70B_TP8 = CacheShape(80, 1, 128, 16, NHD)
SHAPE_QWEN_GQA_HND = CacheShape(28, 4, 128, 32, HND)


def c1_tiny(seed: int = 1) -> Workload:
    rng = np.random.default_rng(seed)
    ctx = rng.integers(100, 301, 8).astype(np.int64)
    w = full_pack("tiny", seed, SHAPE_TINY, ctx, rng, pool_blocks=512,
                  description="2 layers, 2 KV heads, head_dim 64, block 16; "
                  "8 requests of 100-300 tokens in a 512-block pool; full "
                  "pack, then unpack into a fresh permutation")
    return w


def c2_llama8b(seed: int = 2, num_reqs: int = 256, steps: int = 100,
               median: float = 2048, clip_hi: int = 16384) -> Workload:
    rng = np.random.default_rng(seed)
    ctx = _lognormal_ctx(rng, num_reqs, median, 0.75, min(128, clip_hi),
                         clip_hi)
    return incremental("llama3-8b-decode", seed, SHAPE_LLAMA3_8B, ctx, rng,
                       steps, 1, 16,
                       description="Llama-3-8B-shaped cache (32 layers, 8 KV "
                       "heads, head_dim 128, block 16); 256 requests, "
                       "lognormal contexts (median 2048, sigma 0.75, clipped "
                       "to [128,16384]); each of 100 steps checkpoints every "
                       "request's newest 1-16 tokens")


def c3_restore(seed: int = 3, num_reqs: int = 64, ctx_lo: int = 4096,
               ctx_hi: int = 32768, pool_blocks: int = 65536) -> Workload:
    rng = np.random.default_rng(seed)
    ctx = rng.integers(ctx_lo, ctx_hi + 1, num_reqs).astype(np.int64)
    return restore_burst("restore-burst", seed, SHAPE_LLAMA3_8B, ctx, rng,
                         pool_blocks, 0.6,
                         description="Llama-3-8B shape; 64 interrupted "
                         "requests of 4096-32768 tokens restored from "
                         "contiguous checkpoints into a 65536-block pool that "
                         "is 60% occupied; free blocks handed out shuffled, "
                         "in waves that fit the free list")


def c4_llama70b_tp8(seed: int = 4, num_reqs: int = 512,
                    median: float = 4096, clip_hi: int = 32768) -> Workload:
    rng = np.random.default_rng(seed)
    ctx = _lognormal_ctx(rng, num_reqs, median, 0.75, min(128, clip_hi),
                         clip_hi)
    need = int(_ceil_div(ctx, 16).sum())
    nb = int(np.ceil(1.05 * need))
    return full_pack("llama3-70b-tp8-shard", seed, SHAPE_LLAMA3_70B_TP8, ctx,
                     rng, pool_blocks=nb, in_place=True,
                     description="one TP=8 rank of a Llama-3-70B-shaped cache "
                     "(80 layers, 1 KV head, head_dim 128, block 16); 512 "
                     "requests, lognormal contexts (median 4096, sigma 0.75, "
                     "clipped to [128,32768]); full pack, unpack in place "
                     "under a fresh permutation, packed rows streamed to "
                     "pinned host memory")


def c5_qwen_hnd(seed: int = 5, num_reqs: int = 1024, steps: int = 16,
                median: float = 1024, clip_hi: int = 16384) -> Workload:
    rng = np.random.default_rng(seed)
    ctx = _lognormal_ctx(rng, num_reqs, median, 0.75, min(32, clip_hi),
                         clip_hi)
    return incremental("qwen-gqa-hnd", seed, SHAPE_QWEN_GQA_HND, ctx, rng,
                       steps, 1, 64,
                       description="Qwen-style GQA cache in head-major layout "
                       "(28 layers, 4 KV heads, head_dim 128, block 32) with "
                       "token-major checkpoints; 1024 requests, lognormal "
                       "contexts (median 1024, sigma 0.75); each of 16 steps "
                       "checkpoints every request's newest 1-64 tokens")


WORKLOADS = {
    "tiny": c1_tiny,
    "llama3-8b-decode": c2_llama8b,
    "restore-burst": c3_restore,
    "llama3-70b-tp8-shard": c4_llama70b_tp8,
    "qwen-gqa-hnd": c5_qwen_hnd,
}


# --------------------------------------------------------------------------
# Cache contents.  Values are drawn as raw 16-bit patterns so that a copy
# that converts through float (and so changes NaN payloads or -0) is caught.

def random_bits(rng: np.random.Generator, n: int) -> np.ndarray:
    """n uniformly random 16-bit patterns (every bf16 class appears)."""
    return rng.integers(0, 1 << 16, n, dtype=np.uint16)


_WORDS = {1: np.uint8, 2: np.uint16, 4: np.uint32}


def random_words(rng: np.random.Generator, n: int,
                 elem_bytes: int = 2) -> np.ndarray:
    """n uniformly random bit patterns of elem_bytes bytes each (1: 8-bit
    caches, 2: bf16/fp16, 4: fp32)."""
    w = _WORDS[elem_bytes]
    return rng.integers(0, np.iinfo(w).max, n, dtype=w, endpoint=True)


def normal_bf16_bits(rng: np.random.Generator, n: int) -> np.ndarray:
    """n ~N(0,1) values rounded to bf16 (round to nearest even), as bits."""
    x = rng.standard_normal(n, dtype=np.float32).view(np.uint32)
    lsb = (x >> 16) & 1
    return ((x + 0x7FFF + lsb) >> 16).astype(np.uint16)
