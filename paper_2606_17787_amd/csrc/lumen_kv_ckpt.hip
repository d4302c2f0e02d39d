// Paged KV-cache checkpoint pack / restore unpack for MI355X (gfx950).
//
// The operations and layouts are specified in include/lumen_kv_ckpt.h.  This
// file holds the kernels (row plan, token-major gather and scatter, with
// the plan read from a workspace or scanned from the ranges in the same
// launch, page-major gather, restore-target validation, draft-state
// alignment), the staging pipelines to and from pinned host memory, and the
// C ABI.
//
// Work decomposition.  A checkpoint is a sequence of token rows, each
// [L][2][H][D] elements of E bytes (E = 1, 2 or 4; the copy moves raw bits
// and never looks at values).  The copy is split into units of
// (token row, layer): one unit is the K and V of one token in one layer,
// 2*H*D*E bytes, contiguous on the checkpoint side.  Units are numbered in
// checkpoint order, u = packed_row * L + layer, and the grid's wavefronts
// split [0, total_units) into equal contiguous spans, so every wavefront
// moves the same number of bytes whatever the mix of request lengths.  The
// grid is oversubscribed (hundreds of wavefronts per CU, about one unit each
// on a decode step): wavefronts that share a workload still run at very
// different speeds on this chip, and short-lived ones let the hardware
// dispatcher hand the remaining work to whichever CU frees a slot first,
// where a grid of resident long-lived wavefronts ends on its slowest one.
// Small checkpoints with short units get fewer, longer-lived wavefronts (at
// least 4 KiB each, while that leaves 16 per CU), since there a wavefront
// per unit makes wavefront dispatch the bound.
// Inside its span a wavefront walks token rows in order: the
// request, its block-table entry and the checkpoint row of each token are
// wave-uniform and live in scalar registers; the 64 lanes then move the
// token's units as 16-byte vectors.  On the checkpoint side those vectors
// are one contiguous run; on the cache side they are runs of H*D*E bytes
// (token-major cache) or D*E bytes (head-major cache), each a whole number
// of 128-byte lines for the serving shapes, so every access is full-line and
// no LDS staging is needed for the head-major transpose.
//
// Where the walk finds its plan.  Either a plan kernel has written it into
// a caller's workspace (the row prefix of every request), or the copy
// reads the token ranges themselves: each workgroup then scans them into
// LDS before its wavefronts start, which saves the plan kernel's launch and
// the wait for it; there, where units are long, each wavefront copies two
// spans so that one scan serves both.

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <stdint.h>
#include <stdlib.h>

#include <mutex>
#include <vector>

#include "lumen_kv_ckpt.h"

namespace {

// Tuning knobs (compile-time): threads per workgroup of the copy kernels,
// 16-byte vectors each lane keeps in flight, and non-temporal hints on the
// loads (bit 0) and stores (bit 1) of the gather and of the scatter.
#ifndef LUMEN_KV_CKPT_BLOCK_THREADS
#define LUMEN_KV_CKPT_BLOCK_THREADS 256
#endif
#ifndef LUMEN_KV_CKPT_UNROLL
#define LUMEN_KV_CKPT_UNROLL 4
#endif
#ifndef LUMEN_KV_CKPT_PACK_NT
#define LUMEN_KV_CKPT_PACK_NT 3
#endif
#ifndef LUMEN_KV_CKPT_UNPACK_NT
#define LUMEN_KV_CKPT_UNPACK_NT 3
#endif
// Wavefronts per CU in the copy grid (the environment variable of the same
// name overrides it at run time).  Measured on the decode workload: 32 per
// CU, about one resident round, gives 5.25 TB/s on the gather; 384 gives
// 5.7-5.8 TB/s; far beyond one unit per wave, idle waves cost dispatch time.
#ifndef LUMEN_KV_CKPT_WAVES_PER_CU
#define LUMEN_KV_CKPT_WAVES_PER_CU 384
#endif
// The same for units (one token's K and V of one layer) shorter than 4 KiB,
// unless the environment sets the count: measured on the head-major Qwen
// steps (2 KiB units, about ten per wavefront at 384), 768 per CU gathers
// 5% faster.
#ifndef LUMEN_KV_CKPT_SHORT_UNIT_WAVES_PER_CU
#define LUMEN_KV_CKPT_SHORT_UNIT_WAVES_PER_CU 768
#endif
// Fewest bytes a wave of the copy grid is sized for (0: no such bound), and
// the grid size per CU below which that bound does not cut.
#ifndef LUMEN_KV_CKPT_MIN_WAVE_BYTES
#define LUMEN_KV_CKPT_MIN_WAVE_BYTES 4096
#endif
#ifndef LUMEN_KV_CKPT_MIN_WAVES_PER_CU
#define LUMEN_KV_CKPT_MIN_WAVES_PER_CU 16
#endif
// Spans of the copy grid that each wavefront of the one-launch range walk
// copies when a (row, layer) unit is 4 KiB or more (the grid then has that
// many times fewer wavefronts than spans; wavefront w takes spans w, w + n,
// ...).  Each wavefront's set-up scans the ranges, and on the decode
// workload (4 KiB units, about one unit per span) two spans per wavefront
// gave 190.7 against 204.6 us per step with one.  With shorter units (2 KiB,
// head-major Qwen steps, several units per span) two spans per wavefront
// were slower (703 against 657 us per pack), so those keep one.  Plans
// read from a workspace set up in a few loads, and keep one span each.
#ifndef LUMEN_KV_CKPT_RANGE_SPANS_PER_WAVE
#define LUMEN_KV_CKPT_RANGE_SPANS_PER_WAVE 2
#endif
// Double-buffer the batches of a row segment (1) or not (0).
#ifndef LUMEN_KV_CKPT_PIPELINE
#define LUMEN_KV_CKPT_PIPELINE 1
#endif
// Waves per SIMD the register allocation of the copy kernels must allow
// (0: compiler's choice).
#ifndef LUMEN_KV_CKPT_WAVES_PER_EU
#define LUMEN_KV_CKPT_WAVES_PER_EU 0
#endif
#if LUMEN_KV_CKPT_WAVES_PER_EU > 0
#define LUMEN_COPY_OCCUPANCY \
  __attribute__((amdgpu_waves_per_eu(LUMEN_KV_CKPT_WAVES_PER_EU)))
#else
#define LUMEN_COPY_OCCUPANCY
#endif

constexpr int kWave = 64;
constexpr int kBlockThreads = LUMEN_KV_CKPT_BLOCK_THREADS;
constexpr int kWavesPerBlock = kBlockThreads / kWave;
constexpr int kPlanThreads = 1024;
constexpr int kUnroll = LUMEN_KV_CKPT_UNROLL;
constexpr int kDefaultWavesPerCU = LUMEN_KV_CKPT_WAVES_PER_CU;
constexpr int64_t kMinWaveBytes = LUMEN_KV_CKPT_MIN_WAVE_BYTES;
constexpr int64_t kMinWavesPerCU = LUMEN_KV_CKPT_MIN_WAVES_PER_CU;

// Workspace layout (device memory, caller-owned):
//   WsHeader, then int64 prefix[R+1], int64 first_row[R], int32 start[R],
//   int64 items[R+1] (page items, written by the page-major pack).
struct WsHeader {
  int64_t total_rows;  // sum of the valid requests' token counts
  int32_t num_reqs;
  int32_t err;  // most negative device-side status since the plan
  int64_t total_items;  // (request, page) items of the plan, page-major pack
  int64_t reserved[5];
};
static_assert(sizeof(WsHeader) == 64, "header size");

constexpr size_t align16(size_t x) { return (x + 15) & ~size_t(15); }

struct WsView {
  WsHeader *hdr;
  int64_t *prefix;
  int64_t *first_row;
  int32_t *start;
  int64_t *items;
};

WsView ws_view(void *ws, int32_t R) {
  char *p = static_cast<char *>(ws);
  WsView v;
  v.hdr = reinterpret_cast<WsHeader *>(p);
  size_t off = sizeof(WsHeader);
  v.prefix = reinterpret_cast<int64_t *>(p + off);
  off = align16(off + sizeof(int64_t) * (size_t(R) + 1));
  v.first_row = reinterpret_cast<int64_t *>(p + off);
  off = align16(off + sizeof(int64_t) * size_t(R));
  v.start = reinterpret_cast<int32_t *>(p + off);
  off = align16(off + sizeof(int32_t) * size_t(R));
  v.items = reinterpret_cast<int64_t *>(p + off);
  return v;
}

constexpr size_t ws_bytes(int32_t R) {
  size_t off = sizeof(WsHeader);
  off = align16(off + sizeof(int64_t) * (size_t(R) + 1));
  off = align16(off + sizeof(int64_t) * size_t(R));
  off = align16(off + sizeof(int32_t) * size_t(R));
  off = align16(off + sizeof(int64_t) * (size_t(R) + 1));
  return off;
}

// Division by a run-time constant d >= 1 with a multiply-high, valid for
// dividends below 2^31 (round-up reciprocal of Granlund and Montgomery,
// "Division by invariant integers using multiplication", PLDI 1994).
struct FastDiv {
  uint32_t d, mul, shift;
};

FastDiv make_fastdiv(uint32_t d) {
  uint32_t l = 0;
  while ((uint64_t(1) << l) < d) ++l;
  FastDiv f;
  f.d = d;
  f.shift = l;
  f.mul = uint32_t(((uint64_t(1) << 32) * ((uint64_t(1) << l) - d)) / d + 1);
  return f;
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv &f) {
  return (__umulhi(n, f.mul) + n) >> f.shift;
}

// Geometry shared by the gather and the scatter.
struct Geom {
  int64_t slab_bytes;   // stride of one (layer, K/V) slab: NB*bs*H*D*E
  int64_t block_bytes;  // stride of one block inside a slab: bs*H*D*E
  int64_t row_bytes;    // one checkpoint row: L*2*H*D*E
  int64_t num_blocks;
  int64_t ckpt_rows;    // rows the checkpoint buffer (window) holds
  int64_t win_first;    // checkpoint row held by buffer row 0
  int64_t row_lo;       // packed rows [row_lo, row_hi) of the plan are copied
  int64_t row_hi;
  int32_t num_layers;
  int32_t page_layers;  // page-major pack: layers per unit
  int32_t block_size;
  int32_t slot_bytes;   // stride of one slot: H*D*E (NHD) or D*E (HND)
  int32_t head_bytes;   // HND: stride of one head, bs*D*E
  int32_t unit_vecs;    // 16-byte vectors per (token, layer): 2*H*D*E/16
  int32_t bt_cols;
  int32_t num_reqs;
  int64_t spans;        // spans the units are split into (0: one per wave)
  int64_t max_rows;     // rows one launch walks at most: max units / L
  FastDiv div_unit;     // by unit_vecs
  FastDiv div_kv;       // by H*D*E/16, vectors of one (token, layer, K/V)
  FastDiv div_head;     // by D*E/16, vectors of one head
  FastDiv div_bs;       // by block_size
};

__device__ __forceinline__ void record_error(int32_t *err, int code) {
  if ((threadIdx.x & (kWave - 1)) == 0) atomicMin(err, code);
}

// Byte offset, relative to (block, slot) of layer 0 / K, of vector `vv` of a
// token's checkpoint row segment (vv counts 16-byte vectors from the start of
// the row: layer-major, then K/V, then head, then dim).
template <bool kHeadMajor>
__device__ __forceinline__ int64_t cache_vec_offset(uint32_t vv,
                                                    const Geom &g) {
  const uint32_t l = fdiv(vv, g.div_unit);
  const uint32_t w = vv - l * uint32_t(g.unit_vecs);
  const uint32_t kv = fdiv(w, g.div_kv);
  const uint32_t x = w - kv * g.div_kv.d;
  int64_t off = int64_t(l * 2 + kv) * g.slab_bytes;
  if (kHeadMajor) {
    const uint32_t h = fdiv(x, g.div_head);
    const uint32_t y = x - h * g.div_head.d;
    off += int64_t(h) * g.head_bytes + int64_t(y) * 16;
  } else {
    off += int64_t(x) * 16;
  }
  return off;
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// 16-byte load / store.  The buffer between them is a uint4 struct: an
// array of clang vector types in copy_batch makes the register allocator
// keep far more live values (256 VGPRs instead of about 70).
template <bool kNt>
__device__ __forceinline__ uint4 load16(const uint8_t *p) {
  if (kNt) {
    const u32x4 v =
        __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
  }
  return *reinterpret_cast<const uint4 *>(p);
}

template <bool kNt>
__device__ __forceinline__ void store16(uint8_t *p, const uint4 &v) {
  if (kNt)
    __builtin_nontemporal_store(u32x4{v.x, v.y, v.z, v.w},
                                reinterpret_cast<u32x4 *>(p));
  else
    *reinterpret_cast<uint4 *>(p) = v;
}

// Loads and stores of one batch: kUnroll 16-byte vectors per lane, the
// lanes of a wavefront covering kWave consecutive vectors per step.  kPred
// guards the last, partial batch of a row segment.
template <bool kPack>
constexpr int nt_policy() {
  // Measured on the decode workload, each kernel in a loop of its own:
  // non-temporal loads and stores are fastest for both directions.
  return kPack ? LUMEN_KV_CKPT_PACK_NT : LUMEN_KV_CKPT_UNPACK_NT;
}

template <bool kPack, bool kHeadMajor, bool kPred>
__device__ __forceinline__ void load_batch(uint4 (&buf)[kUnroll],
                                           const uint8_t *__restrict__ src,
                                           int64_t cache_tok, int64_t ckpt_off,
                                           uint32_t vbase, int32_t v0,
                                           int32_t nvec, int lane,
                                           const Geom &g) {
#pragma unroll
  for (int k = 0; k < kUnroll; ++k) {
    const int32_t v = v0 + k * kWave + lane;
    buf[k] = make_uint4(0, 0, 0, 0);
    if (!kPred || v < nvec) {
      const int64_t off =
          kPack ? cache_tok + cache_vec_offset<kHeadMajor>(vbase + v, g)
                : ckpt_off + int64_t(v) * 16;
      buf[k] = load16<(nt_policy<kPack>() & 1) != 0>(src + off);
    }
  }
}

template <bool kPack, bool kHeadMajor, bool kPred>
__device__ __forceinline__ void store_batch(const uint4 (&buf)[kUnroll],
                                            uint8_t *__restrict__ dst,
                                            int64_t cache_tok, int64_t ckpt_off,
                                            uint32_t vbase, int32_t v0,
                                            int32_t nvec, int lane,
                                            const Geom &g) {
#pragma unroll
  for (int k = 0; k < kUnroll; ++k) {
    const int32_t v = v0 + k * kWave + lane;
    if (!kPred || v < nvec) {
      const int64_t off =
          kPack ? ckpt_off + int64_t(v) * 16
                : cache_tok + cache_vec_offset<kHeadMajor>(vbase + v, g);
      store16<(nt_policy<kPack>() & 2) != 0>(dst + off, buf[k]);
    }
  }
}

// Copies vectors [0, nvec) of a row segment.  With LUMEN_KV_CKPT_PIPELINE the
// full batches are double-buffered: the loads of batch i+1 are issued before
// the stores of batch i, so a wavefront never waits for its own stores
// before loading again and keeps two batches of loads in flight.
template <bool kPack, bool kHeadMajor>
__device__ __forceinline__ void copy_segment(const uint8_t *__restrict__ src,
                                             uint8_t *__restrict__ dst,
                                             int64_t cache_tok,
                                             int64_t ckpt_off, uint32_t vbase,
                                             int32_t nvec, int lane,
                                             const Geom &g) {
  constexpr int32_t kBatch = kWave * kUnroll;
  const int32_t nfull = nvec / kBatch;
  uint4 a[kUnroll];
#if LUMEN_KV_CKPT_PIPELINE
  if (nfull > 0) {
    uint4 b[kUnroll];
    load_batch<kPack, kHeadMajor, false>(a, src, cache_tok, ckpt_off, vbase,
                                         0, nvec, lane, g);
    int32_t i = 0;
    while (true) {
      if (i + 1 < nfull)
        load_batch<kPack, kHeadMajor, false>(b, src, cache_tok, ckpt_off,
                                             vbase, (i + 1) * kBatch, nvec,
                                             lane, g);
      store_batch<kPack, kHeadMajor, false>(a, dst, cache_tok, ckpt_off,
                                            vbase, i * kBatch, nvec, lane, g);
      if (++i >= nfull) break;
      if (i + 1 < nfull)
        load_batch<kPack, kHeadMajor, false>(a, src, cache_tok, ckpt_off,
                                             vbase, (i + 1) * kBatch, nvec,
                                             lane, g);
      store_batch<kPack, kHeadMajor, false>(b, dst, cache_tok, ckpt_off,
                                            vbase, i * kBatch, nvec, lane, g);
      if (++i >= nfull) break;
    }
  }
#else
  for (int32_t i = 0; i < nfull; ++i) {
    load_batch<kPack, kHeadMajor, false>(a, src, cache_tok, ckpt_off, vbase,
                                         i * kBatch, nvec, lane, g);
    store_batch<kPack, kHeadMajor, false>(a, dst, cache_tok, ckpt_off, vbase,
                                          i * kBatch, nvec, lane, g);
  }
#endif
  if (nfull * kBatch < nvec) {
    load_batch<kPack, kHeadMajor, true>(a, src, cache_tok, ckpt_off, vbase,
                                        nfull * kBatch, nvec, lane, g);
    store_batch<kPack, kHeadMajor, true>(a, dst, cache_tok, ckpt_off, vbase,
                                         nfull * kBatch, nvec, lane, g);
  }
}

// Index of the block-table entry holding token t of request r.  A page past
// the table is clamped to the table's last column (so the load stays in
// bounds and can be issued unconditionally) and reported through `past`.
__device__ __forceinline__ int64_t entry_index(int32_t r, int64_t t,
                                               const Geom &g, bool &past) {
  const uint32_t page = fdiv(uint32_t(t), g.div_bs);
  past = page >= uint32_t(g.bt_cols);
  return int64_t(r) * g.bt_cols + min(page, uint32_t(g.bt_cols - 1));
}

// Status of a token row, checked in the documented order: page inside the
// block table (RANGE), entry a block of the pool (BLOCK_ID), checkpoint row
// inside the buffer (CAPACITY).
__device__ __forceinline__ int row_status(bool past, int32_t entry,
                                          int64_t crow, const Geom &g) {
  if (past) return LUMEN_ERR_RANGE;
  if (entry < 0 || entry >= g.num_blocks) return LUMEN_ERR_BLOCK_ID;
  if (crow < 0 || crow >= g.ckpt_rows) return LUMEN_ERR_CAPACITY;
  return LUMEN_OK;
}

// Where the copy walk finds a token row's request, source token and
// checkpoint row.  WsWalk reads the plan a plan kernel wrote into the
// workspace; RangeWalk reads the ranges themselves, each workgroup scanning
// their token counts into LDS, so the copy needs no plan launch before it.  Both give the same rows: the packed rows of request r start at
// row_base plus the tokens of the valid requests before it; per-request rows
// start at req_row_base[r] + start[r]; invalid ranges count no tokens.
struct WsWalk {
  const WsHeader *hdr;
  const int64_t *prefix;
  const int64_t *first_row;
  const int32_t *start;

  __device__ __forceinline__ WsWalk(const void *p0, const void *p1,
                                    const void *p2, const void *p3, int64_t)
      : hdr(static_cast<const WsHeader *>(p0)),
        prefix(static_cast<const int64_t *>(p1)),
        first_row(static_cast<const int64_t *>(p2)),
        start(static_cast<const int32_t *>(p3)) {}

  // Total token rows of the plan; false when the plan does not match the
  // launch (the wavefront then stops).
  __device__ __forceinline__ bool init(const Geom &g, int lane, int64_t gw,
                                       int32_t *err, int64_t &total) {
    if (hdr->num_reqs != g.num_reqs) {
      if (gw == 0) record_error(err, LUMEN_ERR_INVALID_ARG);
      return false;
    }
    total = hdr->total_rows;
    return true;
  }

  // Request r owning token row `row` (row < total), the end of its rows,
  // its token and its checkpoint buffer row.  The owner is the last request
  // whose prefix does not exceed the row (empty requests share their
  // successor's prefix and are skipped by taking the last).  A 64-way
  // search, one vector load per level, keeps the chain of dependent loads
  // before the first copy short (two levels up to 4096 requests).
  __device__ __forceinline__ void locate(int64_t row, int lane, const Geom &g,
                                         int32_t &r, int64_t &row_end,
                                         int64_t &t, int64_t &crow) const {
    int32_t lo = 0, n = g.num_reqs;
    while (n > 1) {
      const int32_t step = (n + kWave - 1) / kWave;
      const int32_t off = lane * step;
      const int64_t p = off < n ? prefix[lo + off] : INT64_MAX;
      const int32_t c = __popcll(__ballot(p <= row));  // >= 1: prefix[lo] <= row
      lo += (c - 1) * step;
      n = min(step, n - (c - 1) * step);
    }
    r = lo;
    const int64_t p0 = prefix[r];
    row_end = prefix[r + 1];
    t = start[r] + (row - p0);
    crow = first_row[r] + (row - p0) - g.win_first;  // buffer row
  }

  // The next request with rows after r2, whose first row is row + 1; one
  // exists because row + 1 < total.  The bound keeps the walk inside the
  // plan even if a caller has overwritten the workspace (a valid plan never
  // reaches it).
  __device__ __forceinline__ void next(int64_t row, const Geom &g,
                                       int32_t &r2, int64_t &row_end2,
                                       int64_t &t2, int64_t &crow2) const {
    do {
      ++r2;
    } while (r2 + 1 < g.num_reqs && prefix[r2 + 1] == row + 1);
    row_end2 = prefix[r2 + 1];
    t2 = start[r2];
    crow2 = first_row[r2] - g.win_first;
  }
};

__device__ __forceinline__ int64_t readlane64(int64_t x, int src_lane) {
  const uint32_t lo =
      __builtin_amdgcn_readlane(int(uint32_t(uint64_t(x))), src_lane);
  const uint32_t hi =
      __builtin_amdgcn_readlane(int(uint32_t(uint64_t(x) >> 32)), src_lane);
  return int64_t((uint64_t(hi) << 32) | lo);
}

// x plus its copy from the lane that the DPP control selects (0 where that
// lane is outside the source row, or the row is masked off), in 64 bits.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ int64_t add_dpp(int64_t x) {
  const int lo = int(uint32_t(uint64_t(x)));
  const int hi = int(uint32_t(uint64_t(x) >> 32));
  const uint32_t ylo = __builtin_amdgcn_update_dpp(0, lo, kCtrl, kRowMask,
                                                   0xf, true);
  const uint32_t yhi = __builtin_amdgcn_update_dpp(0, hi, kCtrl, kRowMask,
                                                   0xf, true);
  return x + int64_t((uint64_t(yhi) << 32) | ylo);
}

// Inclusive sum over lanes 0..lane of a full wavefront: shifts by 1, 2, 4
// and 8 lanes inside each row of 16, then each row's total broadcast to the
// rows after it (row_bcast:15 to rows 1 and 3, row_bcast:31 to rows 2 and
// 3).  Cross-lane moves are DPP operand modifiers, with no trip through
// LDS.
__device__ __forceinline__ int64_t wave_inclusive_sum(int64_t x) {
  constexpr int kRowShr = 0x110, kRowBcast15 = 0x142, kRowBcast31 = 0x143;
  x = add_dpp<kRowShr + 1, 0xf>(x);
  x = add_dpp<kRowShr + 2, 0xf>(x);
  x = add_dpp<kRowShr + 4, 0xf>(x);
  x = add_dpp<kRowShr + 8, 0xf>(x);
  x = add_dpp<kRowBcast15, 0xa>(x);
  x = add_dpp<kRowBcast31, 0xc>(x);
  return x;
}

__device__ __forceinline__ bool range_ok(int32_t s, int32_t e) {
  return s >= 0 && e >= s;
}

// Dynamic LDS of the copy kernel (used by RangeWalk only).
extern __shared__ __align__(16) int64_t copy_lds[];

struct RangeWalk {
  const int32_t *start;
  const int32_t *end;
  const int64_t *req_row_base;  // null: packed rows from row_base
  int64_t row_base;
  // Exclusive prefix of the requests' token counts, prefix[0..R], in LDS:
  // the workgroup scans the ranges once for its wavefronts.
  const int64_t *prefix;

  __device__ __forceinline__ RangeWalk(const void *p0, const void *p1,
                                       const void *p2, const void *,
                                       int64_t base)
      : start(static_cast<const int32_t *>(p0)),
        end(static_cast<const int32_t *>(p1)),
        req_row_base(static_cast<const int64_t *>(p2)),
        row_base(base),
        prefix(copy_lds) {}

  // Thread k of the workgroup sums the token counts of a contiguous chunk
  // of requests (writing each count to LDS); a wavefront scan and the
  // wavefronts' totals give each chunk its start; each thread then turns
  // its counts into prefixes in place.  An invalid range counts no tokens
  // and is reported once per launch (RANGE), by workgroup 0.
  __device__ __forceinline__ bool init(const Geom &g, int lane, int64_t,
                                       int32_t *err, int64_t &total) {
    int64_t *pre = copy_lds;
    int64_t *wave_tot = copy_lds + g.num_reqs + 1;  // [kWavesPerBlock]
    const int tid = threadIdx.x, wave = tid / kWave;
    const int32_t R = g.num_reqs;
    const int32_t per = (R + kBlockThreads - 1) / kBlockThreads;
    const int32_t lo = min(R, tid * per), hi = min(R, lo + per);
    int64_t local = 0;
    int bad = 0;
#pragma unroll 4
    for (int32_t i = lo; i < hi; ++i) {
      const int32_t s = start[i], e = end[i];
      const bool ok = range_ok(s, e);
      const int64_t n = ok ? int64_t(e) - s : 0;
      bad |= !ok;
      pre[i] = n;
      local += n;
    }
    const int64_t incl = wave_inclusive_sum(local);
    if (lane == kWave - 1) wave_tot[wave] = incl;
    __syncthreads();
    int64_t base = 0;
    total = 0;
#pragma unroll
    for (int w = 0; w < kWavesPerBlock; ++w) {
      const int64_t x = wave_tot[w];
      if (w < wave) base += x;
      total += x;
    }
    int64_t run = base + incl - local;
    for (int32_t i = lo; i < hi; ++i) {
      const int64_t n = pre[i];
      pre[i] = run;
      run += n;
    }
    if (tid == 0) pre[R] = total;
    if (__syncthreads_or(bad) && blockIdx.x == 0 && wave == 0)
      record_error(err, LUMEN_ERR_RANGE);
    return true;
  }

  // As WsWalk::locate, over the prefix in LDS.
  __device__ __forceinline__ void locate(int64_t row, int lane, const Geom &g,
                                         int32_t &r, int64_t &row_end,
                                         int64_t &t, int64_t &crow) const {
    int32_t lo = 0, n = g.num_reqs;
    while (n > 1) {
      const int32_t step = (n + kWave - 1) / kWave;
      const int32_t off = lane * step;
      const int64_t p = off < n ? prefix[lo + off] : INT64_MAX;
      const int32_t c = __popcll(__ballot(p <= row));  // >= 1: prefix[lo] <= row
      lo += (c - 1) * step;
      n = min(step, n - (c - 1) * step);
    }
    r = lo;
    const int64_t p0 = readlane64(prefix[r], 0);
    row_end = readlane64(prefix[r + 1], 0);
    const int32_t s = start[r];
    t = s + (row - p0);
    crow = (req_row_base ? req_row_base[r] + s : row_base + p0) +
           (row - p0) - g.win_first;
  }

  // As WsWalk::next, over the prefix in LDS.
  __device__ __forceinline__ void next(int64_t row, const Geom &g,
                                       int32_t &r2, int64_t &row_end2,
                                       int64_t &t2, int64_t &crow2) const {
    do {
      ++r2;
    } while (r2 + 1 < g.num_reqs &&
             readlane64(prefix[r2 + 1], 0) == row + 1);
    row_end2 = readlane64(prefix[r2 + 1], 0);
    t2 = start[r2];
    crow2 = (req_row_base ? req_row_base[r2] + t2 : row_base + row + 1) -
            g.win_first;
  }
};

// One kernel for both directions.  kPack: cache -> checkpoint;
// otherwise checkpoint -> cache.  The walk's arrays come in as separate
// __restrict__ arguments (p0..p3, in the order of the walk's constructor):
// only then may the compiler read them with scalar loads, which the
// stores of the copy could otherwise clobber.
template <bool kPack, bool kHeadMajor, class Walk>
__global__ __launch_bounds__(kBlockThreads) LUMEN_COPY_OCCUPANCY void copy_rows_kernel(
    const uint8_t *__restrict__ src, uint8_t *__restrict__ dst,
    const int32_t *__restrict__ block_tables, const void *__restrict__ p0,
    const void *__restrict__ p1, const void *__restrict__ p2,
    const void *__restrict__ p3, int64_t row_base, int32_t *err, Geom g) {
  Walk walk(p0, p1, p2, p3, row_base);
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int64_t gw = int64_t(blockIdx.x) * kWavesPerBlock + wave;
  const int64_t nw = int64_t(gridDim.x) * kWavesPerBlock;

  int64_t total;
  if (!walk.init(g, lane, gw, err, total)) return;
  const int64_t L = g.num_layers;
  const int64_t row_a = min(g.row_lo, total), row_b = min(g.row_hi, total);
  // More rows than a launch walks: refused as a whole (nothing copied).
  if (row_b - row_a > g.max_rows) {
    if (gw == 0) record_error(err, LUMEN_ERR_TOO_MANY);
    return;
  }
  const int64_t units = (row_b - row_a) * L;
  // The units are split into V equal spans; wave gw copies spans gw,
  // gw + nw, ... (one span per wave unless the launch asks for fewer waves
  // than spans, so that each wave's set-up serves several).
  const int64_t V = g.spans > 0 ? g.spans : nw;
  for (int64_t v = gw; v < V; v += nw) {
    int64_t u = row_a * L + units * v / V;
    const int64_t u_end = row_a * L + units * (v + 1) / V;
    if (u >= u_end) continue;

    // First token row of the span and its request.
    int64_t row = u / L;
    int32_t l0 = int32_t(u - row * L);
    int32_t r;
    int64_t row_end, t, crow;
    walk.locate(row, lane, g, r, row_end, t, crow);
    if (g.bt_cols == 0) {  // every page lies past an empty table
      record_error(err, LUMEN_ERR_RANGE);
      return;
    }
    bool past;
    int32_t b = block_tables[entry_index(r, t, g, past)];

    while (true) {
      const int32_t nl = int32_t(min(int64_t(g.num_layers - l0), u_end - u));
      const bool more = u + nl < u_end;
      const int code = row_status(past, b, crow, g);
      // Cache side: (block, slot) of layer 0 / K; checkpoint side: the span's
      // first unit in this row.
      const uint32_t slot = uint32_t(t) - fdiv(uint32_t(t), g.div_bs) *
                                              uint32_t(g.block_size);
      const int64_t cache_tok =
          int64_t(b) * g.block_bytes + int64_t(slot) * g.slot_bytes;
      const int64_t ckpt_off =
          crow * g.row_bytes + int64_t(l0) * g.unit_vecs * 16;
      // Materialise this row's addresses here: otherwise the compiler sinks
      // their arithmetic below the next row's block-table load, and the wait
      // for this row's entry then also waits for that load.
      asm volatile("" ::"s"(cache_tok), "s"(ckpt_off) : "memory");

      // Position and block-table entry of the next row.  The entry is loaded
      // unconditionally (clamped index), after every use of this row's entry
      // and before this row's copy, and first used after that copy: the scalar
      // load overlaps with the copy instead of stalling the next row.
      int32_t r2 = r;
      int64_t row_end2 = row_end, t2 = t + 1, crow2 = crow + 1;
      if (more && row + 1 == row_end)
        walk.next(row, g, r2, row_end2, t2, crow2);
      bool past2;
      const int32_t b2 = block_tables[entry_index(r2, t2, g, past2)];

      if (code != LUMEN_OK) {
        record_error(err, code);
      } else {
        copy_segment<kPack, kHeadMajor>(src, dst, cache_tok, ckpt_off,
                                        uint32_t(l0) * uint32_t(g.unit_vecs),
                                        nl * g.unit_vecs, lane, g);
      }
      if (!more) break;
      u += nl;
      l0 = 0;
      ++row;
      r = r2;
      row_end = row_end2;
      t = t2;
      crow = crow2;
      b = b2;
      past = past2;
    }
  }
}

// Page-major pack, step 1: the plan's (request, page) items.  Request r's
// rows [start, start + n) touch pages start/bs .. (start+n-1)/bs; one
// workgroup scans those counts into items[R+1] (cross-lane shuffles within
// each wavefront, once more across the wavefronts' totals).
__global__ __launch_bounds__(kPlanThreads) void item_scan_kernel(
    WsHeader *hdr, const int64_t *__restrict__ prefix,
    const int32_t *__restrict__ start, int64_t *items, int32_t R,
    int32_t block_size) {
  constexpr int kWaves = kPlanThreads / kWave;
  __shared__ int64_t wave_sum[kWaves];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wid = tid / kWave;
  const int32_t per = (R + kPlanThreads - 1) / kPlanThreads;
  const int32_t lo = min(R, tid * per);
  const int32_t hi = min(R, lo + per);
  auto count = [&](int32_t i) -> int64_t {
    const int64_t n = prefix[i + 1] - prefix[i];
    if (n <= 0) return 0;
    const int64_t s = start[i];
    return (s + n - 1) / block_size - s / block_size + 1;
  };
  int64_t local = 0;
  for (int32_t i = lo; i < hi; ++i) local += count(i);
  int64_t x = local;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int64_t y = __shfl_up(x, d, kWave);
    if (lane >= d) x += y;
  }
  if (lane == kWave - 1) wave_sum[wid] = x;
  __syncthreads();
  if (wid == 0) {
    int64_t v = lane < kWaves ? wave_sum[lane] : 0;
#pragma unroll
    for (int d = 1; d < kWaves; d <<= 1) {
      const int64_t y = __shfl_up(v, d, kWave);
      if (lane >= d) v += y;
    }
    if (lane < kWaves) wave_sum[lane] = v;
  }
  __syncthreads();
  int64_t run = (wid > 0 ? wave_sum[wid - 1] : 0) + x - local;
  for (int32_t i = lo; i < hi; ++i) {
    items[i] = run;
    run += count(i);
  }
  if (tid == 0) {
    items[R] = wave_sum[kWaves - 1];
    hdr->total_items = wave_sum[kWaves - 1];
  }
}

// Last index r in [0, n) with pre[r] <= x, for pre non-decreasing with
// pre[0] <= x: a 64-way search, one vector load per level.
__device__ __forceinline__ int32_t find_owner(const int64_t *__restrict__ pre,
                                              int32_t n, int64_t x,
                                              int lane) {
  int32_t lo = 0;
  while (n > 1) {
    const int32_t step = (n + kWave - 1) / kWave;
    const int32_t off = lane * step;
    const int64_t p = off < n ? pre[lo + off] : INT64_MAX;
    const int32_t c = __popcll(__ballot(p <= x));
    lo += (c - 1) * step;
    n = min(step, n - (c - 1) * step);
  }
  return lo;
}

// Where the page-major pack finds its plan: the (request, page) items and
// each request's rows.  WsPages reads the workspace (the plan kernel's row
// prefix and the item scan's items); RangePages scans the ranges into LDS,
// the token and page counts of every request side by side.
struct WsPages {
  const WsHeader *hdr;
  const int64_t *prefix;
  const int64_t *first_row;
  const int32_t *start;
  const int64_t *items;

  __device__ __forceinline__ WsPages(const void *p0, const void *p1,
                                     const void *p2, const void *p3,
                                     const void *p4, int64_t)
      : hdr(static_cast<const WsHeader *>(p0)),
        prefix(static_cast<const int64_t *>(p1)),
        first_row(static_cast<const int64_t *>(p2)),
        start(static_cast<const int32_t *>(p3)),
        items(static_cast<const int64_t *>(p4)) {}

  // Total items and token rows of the plan; false when the plan does not
  // match the launch.
  __device__ __forceinline__ bool init(const Geom &g, int64_t gw,
                                       int32_t *err, int64_t &total,
                                       int64_t &rows_total) {
    if (hdr->num_reqs != g.num_reqs) {
      if (gw == 0) record_error(err, LUMEN_ERR_INVALID_ARG);
      return false;
    }
    total = hdr->total_items;
    rows_total = hdr->total_rows;
    return true;
  }
  __device__ __forceinline__ const int64_t *item_prefix() const {
    return items;
  }
  __device__ __forceinline__ int64_t item0(int32_t r) const {
    return items[r];
  }
  // Request r's first token, token count and checkpoint row of its first
  // token (r has rows: it owns an item).
  __device__ __forceinline__ void request(int32_t r, const Geom &,
                                          int64_t &s, int64_t &n,
                                          int64_t &first) const {
    s = start[r];
    n = prefix[r + 1] - prefix[r];
    first = first_row[r];
  }
};

struct RangePages {
  const int32_t *start;
  const int32_t *end;
  const int64_t *req_row_base;  // null: packed rows from row_base
  int64_t row_base;
  const int64_t *rows;   // LDS: exclusive prefix of token counts, [R+1]
  const int64_t *items;  // LDS: exclusive prefix of page counts, [R+1]

  __device__ __forceinline__ RangePages(const void *p0, const void *p1,
                                        const void *p2, const void *,
                                        const void *, int64_t base)
      : start(static_cast<const int32_t *>(p0)),
        end(static_cast<const int32_t *>(p1)),
        req_row_base(static_cast<const int64_t *>(p2)),
        row_base(base),
        rows(nullptr),
        items(nullptr) {}

  // As RangeWalk::init, for the token and the page counts at once.
  __device__ __forceinline__ bool init(const Geom &g, int64_t,
                                       int32_t *err, int64_t &total,
                                       int64_t &rows_total) {
    const int32_t R = g.num_reqs;
    int64_t *pr = copy_lds;
    int64_t *pi = copy_lds + (R + 1);
    int64_t *wave_tot = copy_lds + 2 * (R + 1);  // [2][kWavesPerBlock]
    rows = pr;
    items = pi;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int32_t per = (R + kBlockThreads - 1) / kBlockThreads;
    const int32_t lo = min(R, tid * per), hi = min(R, lo + per);
    int64_t ln = 0, lp = 0;
    int bad = 0;
#pragma unroll 4
    for (int32_t i = lo; i < hi; ++i) {
      const int32_t s = start[i], e = end[i];
      const bool ok = range_ok(s, e);
      const int64_t n = ok ? int64_t(e) - s : 0;
      // pages (s + n - 1)/bs - s/bs + 1 of a non-empty range; s + n - 1
      // < 2^31, in the fast division's range
      const int64_t np =
          n > 0 ? int64_t(fdiv(uint32_t(s + n - 1), g.div_bs)) -
                      int64_t(fdiv(uint32_t(s), g.div_bs)) + 1
                : 0;
      bad |= !ok;
      pr[i] = n;
      pi[i] = np;
      ln += n;
      lp += np;
    }
    const int64_t in_n = wave_inclusive_sum(ln);
    const int64_t in_p = wave_inclusive_sum(lp);
    if (lane == kWave - 1) {
      wave_tot[wave] = in_n;
      wave_tot[kWavesPerBlock + wave] = in_p;
    }
    __syncthreads();
    int64_t bn = 0, bp = 0, tn = 0, tp = 0;
#pragma unroll
    for (int w = 0; w < kWavesPerBlock; ++w) {
      const int64_t xn = wave_tot[w], xp = wave_tot[kWavesPerBlock + w];
      if (w < wave) {
        bn += xn;
        bp += xp;
      }
      tn += xn;
      tp += xp;
    }
    int64_t rn = bn + in_n - ln, rp = bp + in_p - lp;
    for (int32_t i = lo; i < hi; ++i) {
      const int64_t n = pr[i], np = pi[i];
      pr[i] = rn;
      pi[i] = rp;
      rn += n;
      rp += np;
    }
    if (tid == 0) {
      pr[R] = tn;
      pi[R] = tp;
    }
    if (__syncthreads_or(bad) && blockIdx.x == 0 && wave == 0)
      record_error(err, LUMEN_ERR_RANGE);
    total = tp;
    rows_total = tn;
    return true;
  }
  __device__ __forceinline__ const int64_t *item_prefix() const {
    return items;
  }
  __device__ __forceinline__ int64_t item0(int32_t r) const {
    return readlane64(items[r], 0);
  }
  __device__ __forceinline__ void request(int32_t r, const Geom &g,
                                          int64_t &s, int64_t &n,
                                          int64_t &first) const {
    s = start[r];
    const int64_t p0 = readlane64(rows[r], 0);
    n = readlane64(rows[r + 1], 0) - p0;
    first = req_row_base ? req_row_base[r] + s : row_base + p0;
  }
};

// Page-major pack, step 2, for token-major caches whose per-token run
// (H*D*E bytes per layer and K/V) is short: the unit is one (item, layer),
// the item's tokens of one page.  Its K run and V run are each one
// contiguous stretch of the block (nt * H*D*E bytes), read whole, and each
// token's piece is written to its own checkpoint row.  Units are numbered
// layers fastest and dealt to the wavefronts round-robin, so at any moment
// the grid works on a dense window of consecutive pages (reads) and of
// consecutive checkpoint rows (writes).  Measured on the 70B TP=8 shard
// (256-byte runs): 6.28 TB/s, where contiguous spans per wavefront scatter
// the concurrent writes over the whole checkpoint and reach 5.1 TB/s, and
// the token-major walk 5.35 TB/s.
template <class Pages>
__global__ __launch_bounds__(kBlockThreads) LUMEN_COPY_OCCUPANCY void
pack_pages_kernel(const uint8_t *__restrict__ cache, uint8_t *__restrict__ ckpt,
                  const int32_t *__restrict__ block_tables,
                  const void *__restrict__ p0, const void *__restrict__ p1,
                  const void *__restrict__ p2, const void *__restrict__ p3,
                  const void *__restrict__ p4, int64_t row_base, int32_t *err,
                  Geom g) {
  Pages pages(p0, p1, p2, p3, p4, row_base);
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int64_t gw = int64_t(blockIdx.x) * kWavesPerBlock + wave;
  const int64_t nw = int64_t(gridDim.x) * kWavesPerBlock;
  int64_t total_items, total_rows;
  if (!pages.init(g, gw, err, total_items, total_rows)) return;
  // The limit of the token-major walk, on the same rows.
  if (total_rows > g.max_rows) {
    if (gw == 0) record_error(err, LUMEN_ERR_TOO_MANY);
    return;
  }
  const int64_t *items = pages.item_prefix();
  const int32_t G = g.page_layers;
  const int64_t groups = (g.num_layers + G - 1) / G;
  const int64_t units = total_items * groups;
  const int32_t tok = g.slot_bytes;  // H*D*E
  const int32_t vpt = tok / 16;
  for (int64_t u = gw; u < units; u += nw) {
    const int64_t item = u / groups;
    const int32_t l_first = int32_t(u - item * groups) * G;
    const int32_t l_end = min(l_first + G, g.num_layers);
    const int32_t r = find_owner(items, g.num_reqs, item, lane);
    int64_t s, n, first;
    pages.request(r, g, s, n, first);
    const int64_t e = s + n;
    const int64_t j = s / g.block_size + (item - pages.item0(r));
    const int64_t t_lo = max(s, j * g.block_size);
    const int64_t t_hi = min(e, (j + 1) * g.block_size);
    const int32_t nt = int32_t(t_hi - t_lo);
    const int64_t row0 = first + (t_lo - s) - g.win_first;
    // The item's rows are consecutive: the ones inside the buffer are the
    // tokens [ta, tb) of the page; the others are CAPACITY errors and only
    // they are skipped.
    const int64_t ta64 = row0 < 0 ? -row0 : 0;
    const int64_t room = g.ckpt_rows - row0;
    const int32_t ta = int32_t(min(ta64, int64_t(nt)));
    const int32_t tb = int32_t(max(min(room, int64_t(nt)), int64_t(ta)));
    if (j >= g.bt_cols) {
      record_error(err, LUMEN_ERR_RANGE);
      continue;
    }
    const int32_t b = block_tables[int64_t(r) * g.bt_cols + j];
    if (b < 0 || b >= g.num_blocks) {
      record_error(err, LUMEN_ERR_BLOCK_ID);
      continue;
    }
    if (ta > 0 || tb < nt) record_error(err, LUMEN_ERR_CAPACITY);
    const int64_t blk = int64_t(b) * g.block_bytes +
                        (t_lo - j * g.block_size) * int64_t(tok);
    const int32_t nv = tb * vpt;  // vectors of the K (or V) run to copy
    for (int32_t l = l_first; l < l_end; ++l) {
      const uint8_t *k_run = cache + int64_t(l * 2) * g.slab_bytes + blk;
      const uint8_t *v_run = k_run + g.slab_bytes;
      for (int32_t v0 = ta * vpt; v0 < nv; v0 += kWave * kUnroll) {
        uint4 ka[kUnroll], va[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
          const int32_t v = v0 + k * kWave + lane;
          ka[k] = make_uint4(0, 0, 0, 0);
          va[k] = make_uint4(0, 0, 0, 0);
          if (v < nv) {
            ka[k] = load16<(nt_policy<true>() & 1) != 0>(k_run + int64_t(v) * 16);
            va[k] = load16<(nt_policy<true>() & 1) != 0>(v_run + int64_t(v) * 16);
          }
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
          const int32_t v = v0 + k * kWave + lane;
          if (v < nv) {
            const uint32_t t = fdiv(uint32_t(v), g.div_kv);
            const int64_t w = int64_t(v) - int64_t(t) * vpt;
            uint8_t *q = ckpt + (row0 + t) * g.row_bytes +
                         int64_t(l * 2) * tok + w * 16;
            store16<(nt_policy<true>() & 2) != 0>(q, ka[k]);
            store16<(nt_policy<true>() & 2) != 0>(q + tok, va[k]);
          }
        }
      }
    }
  }
}

// Row plan: one workgroup scans the per-request token counts.  Each thread
// sums a contiguous chunk of requests; the per-thread sums are scanned with
// cross-lane shuffles inside each wavefront and once more across the
// wavefronts' totals, so only two workgroup barriers are needed.
__global__ __launch_bounds__(kPlanThreads) void plan_kernel(
    const int32_t *__restrict__ d_start, const int32_t *__restrict__ d_end,
    int32_t R, int64_t row_base, const int64_t *__restrict__ req_row_base,
    WsHeader *hdr, int64_t *prefix, int64_t *first_row, int32_t *start,
    int32_t *err) {
  constexpr int kWaves = kPlanThreads / kWave;
  __shared__ int64_t wave_sum[kWaves];
  __shared__ int bad;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wid = tid / kWave;
  const int32_t per = (R + kPlanThreads - 1) / kPlanThreads;
  const int32_t lo = min(R, tid * per);
  const int32_t hi = min(R, lo + per);
  int64_t local = 0;
  int my_bad = 0;
  for (int32_t i = lo; i < hi; ++i) {
    const int32_t s = d_start[i], e = d_end[i];
    if (s < 0 || e < s) my_bad = 1; else local += int64_t(e) - s;
  }
  // Inclusive scan of the per-thread sums within the wavefront.
  int64_t x = local;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int64_t y = __shfl_up(x, d, kWave);
    if (lane >= d) x += y;
  }
  if (lane == kWave - 1) wave_sum[wid] = x;
  if (tid == 0) bad = 0;
  __syncthreads();
  if (my_bad) atomicOr(&bad, 1);
  if (wid == 0) {  // inclusive scan of the wavefront totals
    int64_t v = lane < kWaves ? wave_sum[lane] : 0;
#pragma unroll
    for (int d = 1; d < kWaves; d <<= 1) {
      const int64_t y = __shfl_up(v, d, kWave);
      if (lane >= d) v += y;
    }
    if (lane < kWaves) wave_sum[lane] = v;
  }
  __syncthreads();
  int64_t run = (wid > 0 ? wave_sum[wid - 1] : 0) + x - local;  // exclusive
  for (int32_t i = lo; i < hi; ++i) {
    const int32_t s = d_start[i], e = d_end[i];
    const bool ok = !(s < 0 || e < s);
    const int64_t n = ok ? int64_t(e) - s : 0;
    prefix[i] = run;
    first_row[i] = req_row_base ? req_row_base[i] + s : row_base + run;
    start[i] = ok ? s : 0;
    run += n;
  }
  if (tid == 0) {
    const int64_t total = wave_sum[kWaves - 1];
    prefix[R] = total;
    hdr->total_rows = total;
    hdr->num_reqs = R;
    hdr->err = LUMEN_OK;
    *err = bad ? LUMEN_ERR_RANGE : LUMEN_OK;  // the header's word, or the
                                              // caller's status word
  }
}

// Validate mode, step 1: clear the mark bits (a kernel rather than a memset,
// so that the call can be captured in a graph).
__global__ __launch_bounds__(kBlockThreads) void clear_marks_kernel(
    uint4 *__restrict__ marks, int64_t n16) {
  const int64_t stride = int64_t(gridDim.x) * kBlockThreads;
  for (int64_t i = int64_t(blockIdx.x) * kBlockThreads + threadIdx.x; i < n16;
       i += stride)
    marks[i] = make_uint4(0, 0, 0, 0);
}

// Validate mode, step 2: one workgroup per request (grid-strided) walks the
// pages the unpack of its planned range writes, pages start/bs through
// (end-1)/bs, and sets one mark bit per physical block.  The atomic OR
// returns the previous word, so of two pages naming one block exactly one
// sees the bit already set, whatever the order.
__global__ __launch_bounds__(kBlockThreads) void validate_kernel(
    const int32_t *__restrict__ block_tables, const WsHeader *__restrict__ hdr,
    const int64_t *__restrict__ prefix, const int32_t *__restrict__ start,
    uint32_t *marks, int32_t *err, int32_t num_reqs, int32_t bt_cols,
    int32_t block_size, int64_t num_blocks) {
  if (hdr->num_reqs != num_reqs) {
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicMin(err, LUMEN_ERR_INVALID_ARG);
    return;
  }
  for (int32_t r = blockIdx.x; r < num_reqs; r += gridDim.x) {
    const int64_t n = prefix[r + 1] - prefix[r];
    if (n == 0) continue;
    const int64_t s = start[r];
    const int64_t first = s / block_size, last = (s + n - 1) / block_size;
    for (int64_t j = first + threadIdx.x; j <= last; j += kBlockThreads) {
      int code = LUMEN_OK;
      if (j >= bt_cols) {
        code = LUMEN_ERR_RANGE;
      } else {
        const int32_t b = block_tables[int64_t(r) * bt_cols + j];
        if (b < 0 || b >= num_blocks) {
          code = LUMEN_ERR_BLOCK_ID;
        } else {
          const uint32_t bit = 1u << (b & 31);
          if (atomicOr(&marks[b >> 5], bit) & bit) code = LUMEN_ERR_DUP_BLOCK;
        }
      }
      if (code != LUMEN_OK) atomicMin(err, code);
    }
  }
}

// Draft-state alignment, step 1: one wavefront per request (grid-strided)
// finds the first position where the draft and committed tokens differ,
// 1024 positions per round, truncates the request's KV length to it, and
// counts the allocated table entries of the pages the shorter KV no longer
// reaches.  Per request it leaves in the workspace the count (-1 for a
// request with inconsistent lengths, which is left unchanged) and the page
// span [lo, hi) packed into one int64.
__global__ __launch_bounds__(kBlockThreads) void draft_match_kernel(
    const int32_t *__restrict__ draft, int32_t draft_cols,
    const int32_t *__restrict__ draft_len,
    const int32_t *__restrict__ committed, int32_t committed_cols,
    const int32_t *__restrict__ committed_len, int32_t *kv_len,
    const int32_t *__restrict__ block_tables, int32_t bt_cols,
    int32_t block_size, int32_t num_reqs, int32_t *replay, int64_t *count,
    int64_t *span) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t gw = int64_t(blockIdx.x) * kWavesPerBlock + threadIdx.x / kWave;
  const int64_t nw = int64_t(gridDim.x) * kWavesPerBlock;
  for (int64_t r = gw; r < num_reqs; r += nw) {
    const int32_t dl = draft_len[r], cl = committed_len[r], kl = kv_len[r];
    if (dl < 0 || cl < 0 || kl < 0 || dl > draft_cols ||
        cl > committed_cols || int64_t(kl) > int64_t(bt_cols) * block_size) {
      if (lane == 0) {
        count[r] = -1;
        span[r] = 0;
        replay[r] = 0;
      }
      continue;
    }
    const int32_t lim = min(dl, cl);
    const int32_t *d = draft + r * draft_cols;
    const int32_t *c = committed + r * committed_cols;
    // kMatch positions per lane per round, all loads in flight together;
    // the round's first mismatch is the minimum over the lanes.
    constexpr int kMatch = 16;
    int32_t p = lim;
    for (int32_t base = 0; base < lim; base += kWave * kMatch) {
      int32_t dv[kMatch], cv[kMatch];
#pragma unroll
      for (int k = 0; k < kMatch; ++k) {
        const int32_t i = base + k * kWave + lane;
        dv[k] = i < lim ? d[i] : 0;
        cv[k] = i < lim ? c[i] : 0;
      }
      int32_t mine = INT32_MAX;
#pragma unroll
      for (int k = kMatch - 1; k >= 0; --k)
        if (dv[k] != cv[k]) mine = base + k * kWave + lane;
#pragma unroll
      for (int off = kWave / 2; off > 0; off >>= 1)
        mine = min(mine, __shfl_xor(mine, off, kWave));
      if (mine != INT32_MAX) {  // wave-uniform after the reduction
        p = mine;
        break;
      }
    }
    const int32_t valid = min(kl, p);
    const int32_t lo = (valid + block_size - 1) / block_size;
    const int32_t hi = (kl + block_size - 1) / block_size;
    int64_t n = 0;
    const int32_t *row = block_tables + r * bt_cols;
    for (int32_t j = lo + lane; j - lane < hi; j += kWave)
      n += __popcll(__ballot(j < hi && row[j] >= 0));
    if (lane == 0) {
      kv_len[r] = valid;
      replay[r] = cl - valid;
      count[r] = n;
      span[r] = (int64_t(lo) << 32) | int64_t(hi);
    }
  }
}

// Draft-state alignment, step 2: one workgroup scans the per-request counts
// (as the row plan does), lists the freed block ids in request order, then
// page order, clears their table entries, and writes the status of this
// call into the workspace's error word (a new epoch).
__global__ __launch_bounds__(kPlanThreads) void draft_free_kernel(
    int32_t *block_tables, int32_t bt_cols, int32_t R,
    const int64_t *__restrict__ count, const int64_t *__restrict__ span,
    int32_t *freed, int64_t freed_cap, int64_t *freed_count,
    WsHeader *hdr) {
  constexpr int kWaves = kPlanThreads / kWave;
  __shared__ int64_t wave_sum[kWaves];
  __shared__ int bad;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wid = tid / kWave;
  const int32_t per = (R + kPlanThreads - 1) / kPlanThreads;
  const int32_t lo = min(R, tid * per);
  const int32_t hi = min(R, lo + per);
  int64_t local = 0;
  int my_bad = 0;
  for (int32_t i = lo; i < hi; ++i) {
    const int64_t n = count[i];
    if (n < 0) my_bad = 1; else local += n;
  }
  int64_t x = local;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int64_t y = __shfl_up(x, d, kWave);
    if (lane >= d) x += y;
  }
  if (lane == kWave - 1) wave_sum[wid] = x;
  if (tid == 0) bad = 0;
  __syncthreads();
  if (my_bad) atomicOr(&bad, 1);
  if (wid == 0) {
    int64_t v = lane < kWaves ? wave_sum[lane] : 0;
#pragma unroll
    for (int d = 1; d < kWaves; d <<= 1) {
      const int64_t y = __shfl_up(v, d, kWave);
      if (lane >= d) v += y;
    }
    if (lane < kWaves) wave_sum[lane] = v;
  }
  __syncthreads();
  int64_t off = (wid > 0 ? wave_sum[wid - 1] : 0) + x - local;  // exclusive
  for (int32_t i = lo; i < hi; ++i) {
    if (count[i] <= 0) continue;
    const int32_t a = int32_t(span[i] >> 32), b = int32_t(span[i] & 0xffffffff);
    int32_t *row = block_tables + int64_t(i) * bt_cols;
    for (int32_t j = a; j < b; ++j) {
      const int32_t blk = row[j];
      if (blk < 0) continue;
      if (off < freed_cap) {  // an entry is cleared only once it is listed
        freed[off] = blk;
        row[j] = -1;
      }
      ++off;
    }
  }
  if (tid == 0) {
    const int64_t total = wave_sum[kWaves - 1];
    *freed_count = total;
    hdr->total_rows = 0;  // no copy plan in the workspace any more
    hdr->num_reqs = -1;
    int st = bad ? LUMEN_ERR_RANGE : LUMEN_OK;
    if (total > freed_cap) st = min(st, LUMEN_ERR_CAPACITY);
    hdr->err = st;
  }
}

// ------------------------------------------------------------- host side

constexpr int kMaxDevices = 64;

// Plan workspace of lumen_kv_ckpt_pack_noalloc, for callers that cannot
// allocate: one copy per device, held until the process ends, sized for
// kNoAllocMaxReqs requests.  Host code must not use this name as an address
// (it is a host-side stand-in); each device's address comes from
// hipGetSymbolAddress at that device's set-up.
constexpr int32_t kNoAllocMaxReqs = LUMEN_KV_CKPT_NOALLOC_MAX_REQS;
// The range walk keeps a prefix of 8 bytes per request in each
// workgroup's LDS (32 KiB at the limit).
constexpr int32_t kRangesMaxReqs = LUMEN_KV_CKPT_RANGES_MAX_REQS;
constexpr int64_t kMaxUnits = LUMEN_KV_CKPT_MAX_UNITS;
// The page-major pack over the ranges keeps two prefixes (tokens and
// pages) in LDS; above this many requests the range path packs
// token-major instead.
constexpr int32_t kRangesPageMaxReqs = 2048;
static_assert(sizeof(int64_t) * (2 * (kRangesPageMaxReqs + 1) +
                                 2 * kWavesPerBlock) <= 64 * 1024,
              "page-major range walk LDS");
static_assert(sizeof(int64_t) * (kRangesMaxReqs + 1 + kWavesPerBlock) <=
                  64 * 1024, "range walk LDS");
constexpr size_t kScratchBytes = ws_bytes(kNoAllocMaxReqs);
static __device__ __align__(256) uint8_t scratch[kScratchBytes];
constexpr int32_t kMaxSlots = 64;  // ring slots of a staging pipeline
constexpr size_t kMaxRings = 16;   // staging rings remembered per device
// Direct host copies: default and largest workgroup counts.  Measured on
// MI355X, kernels moving 16-byte vectors to or from pinned host memory
// reach the link rate (about 57 GB/s to the device, 55-56 GB/s to the
// host) from 32-64 workgroups of 256 threads on; more only hold CU slots.
constexpr int32_t kDirectWorkgroups = 64;
constexpr int32_t kMaxDirectWorkgroups = 4096;

struct DeviceInfo {
  std::once_flag once;
  int cus = 0;
  hipEvent_t order_event = nullptr;
  std::mutex event_mu;
  // Events of the staging pipelines, two per ring slot, created on first
  // use and kept for the life of the process.  pipe_mu is held while a
  // pipeline enqueues, so two calls never interleave records and waits on
  // the same event.
  std::mutex pipe_mu;
  std::vector<hipEvent_t> pipe_events;
  // Staging rings of recent pipeline calls (pipe_mu held): per ring, an
  // event recorded on the stream that last read or wrote it, once that
  // call's work on the ring has been enqueued.  The next call on the same
  // ring orders its first use after that event.
  struct Ring {
    const void *staging = nullptr;
    hipEvent_t idle = nullptr;
    bool recorded = false;
  };
  std::vector<Ring> rings;
  size_t ring_next = 0;  // entry reused once kMaxRings are known
  // This device's copy of `scratch` (null if its address could not be had).
  void *scratch = nullptr;
};
DeviceInfo g_dev[kMaxDevices];

int waves_per_cu(int64_t unit_bytes) {
  static int env = [] {
    const char *e = getenv("LUMEN_KV_CKPT_WAVES_PER_CU");
    const int v = e ? atoi(e) : 0;
    return v > 0 && v <= 4096 ? v : 0;
  }();
  if (env > 0) return env;
  return unit_bytes < 4096 ? LUMEN_KV_CKPT_SHORT_UNIT_WAVES_PER_CU
                           : kDefaultWavesPerCU;
}

// Page-major pack for token-major caches whose per-token run is at most
// this many bytes (measured on the Llama-3-70B TP=8 shard, 256-byte runs:
// 6.28 TB/s page-major against 5.35 TB/s token-major).  The environment
// variable LUMEN_KV_CKPT_PAGE_MAJOR overrides: 0 never, 1 for every
// token-major pack.
constexpr int32_t kPageMajorMaxRun = 512;

int page_layers() {
  static int v = [] {
    const char *e = getenv("LUMEN_KV_CKPT_PAGE_LAYERS");
    const int x = e ? atoi(e) : 1;
    return x >= 1 && x <= 1024 ? x : 1;
  }();
  return v;
}

bool use_page_major(int64_t run_bytes) {
  static int mode = [] {
    const char *e = getenv("LUMEN_KV_CKPT_PAGE_MAJOR");
    return e ? atoi(e) : -1;
  }();
  if (mode == 0) return false;
  if (mode == 1) return true;
  return run_bytes <= kPageMajorMaxRun;
}

int current_device(DeviceInfo **info) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return LUMEN_ERR_HIP;
  DeviceInfo &d = g_dev[dev];
  std::call_once(d.once, [&] {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount,
                              dev) == hipSuccess)
      d.cus = cus;
    hipEvent_t ev = nullptr;
    if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) == hipSuccess)
      d.order_event = ev;
    // Device `dev` is current here, so this is its copy of the array.
    void *ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) == hipSuccess)
      d.scratch = ptr;
    else
      (void)hipGetLastError();  // only the allocation-free call needs it
  });
  if (d.cus <= 0 || !d.order_event) return LUMEN_ERR_HIP;
  *info = &d;
  return LUMEN_OK;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// Takes an error that an earlier runtime call of this thread left pending
// (the caller's, say a failed event query), so that the check after this
// call's launches reports their own outcome only.
void clear_pending_error() { (void)hipGetLastError(); }

int check_layout(const lumen_kv_layout *lay) {
  if (!lay) return LUMEN_ERR_INVALID_ARG;
  if (lay->num_layers <= 0 || lay->num_kv_heads <= 0 || lay->head_dim <= 0 ||
      lay->block_size <= 0 || lay->num_blocks < 0)
    return LUMEN_ERR_INVALID_ARG;
  if (lay->elem_bytes != 1 && lay->elem_bytes != 2 && lay->elem_bytes != 4)
    return LUMEN_ERR_UNSUPPORTED;
  if (lay->cache_order != LUMEN_CACHE_NHD && lay->cache_order != LUMEN_CACHE_HND)
    return LUMEN_ERR_UNSUPPORTED;
  if ((int64_t(lay->head_dim) * lay->elem_bytes) % 16 != 0)
    return LUMEN_ERR_UNSUPPORTED;
  // Vector indices within a row and token positions are 32-bit.
  const int64_t row_bytes = int64_t(lay->num_layers) * 2 * lay->num_kv_heads *
                            lay->head_dim * lay->elem_bytes;
  if (row_bytes / 16 >= (int64_t(1) << 31)) return LUMEN_ERR_UNSUPPORTED;
  // Slot and head strides are 32-bit.
  const int64_t d_bytes = int64_t(lay->head_dim) * lay->elem_bytes;
  if (d_bytes * lay->num_kv_heads >= (int64_t(1) << 31) ||
      d_bytes * lay->block_size >= (int64_t(1) << 31))
    return LUMEN_ERR_UNSUPPORTED;
  return LUMEN_OK;
}

// A buffer may be null only when it is empty; the device checks then keep
// every access away from it.
int check_copy_buffers(const lumen_kv_layout *lay, const void *cache,
                       const void *ckpt, const int32_t *bt, int32_t bt_cols,
                       int64_t ckpt_rows) {
  if ((!cache && lay->num_blocks > 0) || (!ckpt && ckpt_rows > 0) ||
      (!bt && bt_cols > 0))
    return LUMEN_ERR_INVALID_ARG;
  if (!aligned16(cache) || !aligned16(ckpt)) return LUMEN_ERR_MISALIGNED;
  return LUMEN_OK;
}

// Events for the next copy kernel of this thread (lumen_kv_ckpt_time_next_copy).
struct Timing {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
  bool armed = false;
};
thread_local Timing next_timing;

Timing take_timing() {
  const Timing t = next_timing;
  next_timing = Timing{};
  return t;
}

// A kernel launch that carries the timing events when they are armed
// (hipExtLaunchKernel stamps the kernel's own start and end on them).
#define LUMEN_LAUNCH(tm, kernel, grid, block, lds, s, ...)                    \
  do {                                                                       \
    if ((tm).armed)                                                          \
      hipExtLaunchKernelGGL(kernel, grid, block, uint32_t(lds), s,           \
                            (tm).start, (tm).stop, 0, __VA_ARGS__);          \
    else                                                                     \
      hipLaunchKernelGGL(kernel, grid, block, lds, s, __VA_ARGS__);          \
  } while (0)

// max_waves > 0 caps the grid (a copy whose checkpoint side is host memory
// across the host link needs a few hundred wavefronts, not the HBM grid) and
// keeps the token-major walk, whose checkpoint accesses are sequential.
template <class Walk>
void launch_rows(bool pack, bool hnd, unsigned blocks, size_t lds,
                 hipStream_t s, const Timing &tm, const uint8_t *in,
                 uint8_t *out, const int32_t *bt, const void *p0,
                 const void *p1, const void *p2, const void *p3,
                 int64_t row_base, int32_t *err, const Geom &g) {
  const dim3 grid(blocks), block(kBlockThreads);
  if (pack) {
    if (hnd)
      LUMEN_LAUNCH(tm, (copy_rows_kernel<true, true, Walk>), grid, block, lds,
                   s, in, out, bt, p0, p1, p2, p3, row_base, err, g);
    else
      LUMEN_LAUNCH(tm, (copy_rows_kernel<true, false, Walk>), grid, block,
                   lds, s, in, out, bt, p0, p1, p2, p3, row_base, err, g);
  } else {
    if (hnd)
      LUMEN_LAUNCH(tm, (copy_rows_kernel<false, true, Walk>), grid, block,
                   lds, s, in, out, bt, p0, p1, p2, p3, row_base, err, g);
    else
      LUMEN_LAUNCH(tm, (copy_rows_kernel<false, false, Walk>), grid, block,
                   lds, s, in, out, bt, p0, p1, p2, p3, row_base, err, g);
  }
}

// The ranges of a one-launch copy.
struct Ranges {
  const int32_t *start;
  const int32_t *end;
  const int64_t *req_row_base;
  int64_t row_base;
};

// Copies the rows of a plan: the workspace's (ws) or, with `ranges`, the
// ranges themselves in a single launch (ws unused, err_word required).
int launch_copy(bool pack, const lumen_kv_layout *lay, const void *src,
                void *dst, const int32_t *bt, int32_t bt_cols,
                int32_t num_reqs, void *ws, int64_t row_lo, int64_t row_hi,
                int64_t win_first, int64_t ckpt_rows, lumen_stream_t stream,
                int64_t max_waves = 0, int32_t *err_word = nullptr,
                const Ranges *ranges = nullptr) {
  int st = check_layout(lay);
  if (st != LUMEN_OK) return st;
  if (num_reqs < 0 || bt_cols < 0 || ckpt_rows < 0) return LUMEN_ERR_INVALID_ARG;
  if (row_lo < 0 || row_hi < row_lo || win_first < 0) return LUMEN_ERR_INVALID_ARG;
  if (ranges) {
    if (!err_word) return LUMEN_ERR_INVALID_ARG;
  } else {
    if (!ws) return LUMEN_ERR_INVALID_ARG;
    if (!aligned16(ws)) return LUMEN_ERR_MISALIGNED;
  }
  if (num_reqs == 0 || row_hi == row_lo) return LUMEN_OK;
  st = check_copy_buffers(lay, pack ? src : dst, pack ? dst : src, bt,
                          bt_cols, ckpt_rows);
  if (st != LUMEN_OK) return st;
  DeviceInfo *dev = nullptr;
  st = current_device(&dev);
  if (st != LUMEN_OK) return st;

  const int64_t H = lay->num_kv_heads, D = lay->head_dim;
  const int64_t bs = lay->block_size;
  const int64_t d_bytes = D * lay->elem_bytes;
  Geom g;
  g.block_bytes = bs * H * d_bytes;
  g.slab_bytes = lay->num_blocks * g.block_bytes;
  g.row_bytes = int64_t(lay->num_layers) * 2 * H * d_bytes;
  g.num_blocks = lay->num_blocks;
  g.ckpt_rows = ckpt_rows;
  g.win_first = win_first;
  g.row_lo = row_lo;
  g.row_hi = row_hi;
  g.page_layers = page_layers();
  g.num_layers = lay->num_layers;
  g.block_size = lay->block_size;
  const bool hnd = lay->cache_order == LUMEN_CACHE_HND;
  g.slot_bytes = int32_t(hnd ? d_bytes : H * d_bytes);
  g.head_bytes = int32_t(hnd ? bs * d_bytes : 0);
  g.unit_vecs = int32_t(2 * H * d_bytes / 16);
  g.bt_cols = bt_cols;
  g.num_reqs = num_reqs;
  g.max_rows = kMaxUnits / lay->num_layers;
  g.div_unit = make_fastdiv(uint32_t(g.unit_vecs));
  g.div_kv = make_fastdiv(uint32_t(H * d_bytes / 16));
  g.div_head = make_fastdiv(uint32_t(d_bytes / 16));
  g.div_bs = make_fastdiv(uint32_t(bs));

  WsView v = ranges ? WsView{} : ws_view(ws, num_reqs);
  int32_t *err = err_word ? err_word : &v.hdr->err;
  // Oversubscribed grid (waves_per_cu per CU, by unit size), never more
  // waves than the checkpoint buffer could hold units: a wave whose span is
  // empty still costs a dispatch, so a checkpoint buffer sized to the rows
  // of the plan keeps small launches from paying for idle waves.
  int64_t waves = int64_t(dev->cus) * waves_per_cu(g.row_bytes / lay->num_layers);
  const int64_t cap_rows = ckpt_rows < row_hi - row_lo ? ckpt_rows
                                                       : row_hi - row_lo;
  const int64_t max_units = cap_rows * int64_t(lay->num_layers);
  if (max_waves > 0 && max_waves < waves) waves = max_waves;
  if (max_units < waves) waves = max_units > 0 ? max_units : 1;
  // Nor more waves than the buffer holds kMinWaveBytes pieces: where units
  // are a few hundred bytes (one KV head per GPU), a wave per unit of a
  // small checkpoint would leave the launch bound by wave dispatch.  Below
  // kMinWavesPerCU waves per CU the bound does not cut, so that a tiny
  // checkpoint still has enough waves in flight to hide memory latency.
  if (kMinWaveBytes > 0 && cap_rows <= (INT64_MAX / 2) / g.row_bytes) {
    int64_t pieces = (cap_rows * g.row_bytes + kMinWaveBytes - 1) /
                     kMinWaveBytes;
    const int64_t floor_waves = int64_t(dev->cus) * kMinWavesPerCU;
    if (pieces < floor_waves) pieces = floor_waves;
    if (pieces < waves) waves = pieces > 0 ? pieces : 1;
  }
  const unsigned blocks = unsigned((waves + kWavesPerBlock - 1) / kWavesPerBlock);
  // Token-major walk over the ranges: `waves` spans, several of them per
  // wavefront for long units.
  unsigned row_blocks = blocks;
  g.spans = 0;
  const int64_t spw = LUMEN_KV_CKPT_RANGE_SPANS_PER_WAVE;
  if (ranges && spw > 1 && g.row_bytes / lay->num_layers >= 4096 &&
      waves >= 2 * spw) {
    g.spans = waves;
    const int64_t phys = (waves + spw - 1) / spw;
    row_blocks = unsigned((phys + kWavesPerBlock - 1) / kWavesPerBlock);
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  const uint8_t *in = static_cast<const uint8_t *>(src);
  uint8_t *out = static_cast<uint8_t *>(dst);
  const Timing tm = take_timing();  // a copy kernel is launched below
  clear_pending_error();
  const bool page_major = pack && !hnd && row_lo == 0 &&
                          row_hi == INT64_MAX && win_first == 0 &&
                          max_waves == 0 && use_page_major(H * d_bytes);
  if (ranges && page_major && num_reqs <= kRangesPageMaxReqs) {
    // LDS: the token and page prefixes, [R + 1] each, and the wavefronts'
    // totals of both.
    const size_t lds =
        sizeof(int64_t) * (2 * (size_t(num_reqs) + 1) + 2 * kWavesPerBlock);
    LUMEN_LAUNCH(tm, (pack_pages_kernel<RangePages>), dim3(blocks),
                 dim3(kBlockThreads), lds, s, in, out, bt, ranges->start,
                 ranges->end, ranges->req_row_base, nullptr, nullptr,
                 ranges->row_base, err, g);
  } else if (ranges) {
    // LDS: prefix[R + 1] and the wavefronts' totals.
    const size_t lds = sizeof(int64_t) * (size_t(num_reqs) + 1 + kWavesPerBlock);
    launch_rows<RangeWalk>(pack, hnd, row_blocks, lds, s, tm, in, out, bt,
                           ranges->start, ranges->end, ranges->req_row_base,
                           nullptr, ranges->row_base, err, g);
  } else if (page_major) {
    hipLaunchKernelGGL(item_scan_kernel, dim3(1), dim3(kPlanThreads), 0, s,
                       v.hdr, v.prefix, v.start, v.items, num_reqs,
                       lay->block_size);
    LUMEN_LAUNCH(tm, (pack_pages_kernel<WsPages>), dim3(blocks),
                 dim3(kBlockThreads), 0, s, in, out, bt, v.hdr, v.prefix,
                 v.first_row, v.start, v.items, 0, err, g);
  } else {
    launch_rows<WsWalk>(pack, hnd, row_blocks, 0, s, tm, in, out, bt, v.hdr,
                        v.prefix, v.first_row, v.start, 0, err, g);
  }
  return hipGetLastError() == hipSuccess ? LUMEN_OK : LUMEN_ERR_HIP;
}

// Grows the device's pipeline event pool to n events; pipe_mu held.
int pipe_events(DeviceInfo *dev, size_t n) {
  while (dev->pipe_events.size() < n) {
    hipEvent_t ev = nullptr;
    if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess)
      return LUMEN_ERR_HIP;
    dev->pipe_events.push_back(ev);
  }
  return LUMEN_OK;
}

// The entry of staging ring `staging`, created (or the oldest entry
// recycled) on first use; pipe_mu held.
int ring_entry(DeviceInfo *dev, const void *staging, DeviceInfo::Ring **out) {
  for (auto &r : dev->rings)
    if (r.staging == staging) {
      *out = &r;
      return LUMEN_OK;
    }
  DeviceInfo::Ring *r = nullptr;
  if (dev->rings.size() < kMaxRings) {
    dev->rings.reserve(kMaxRings);  // entries never move
    hipEvent_t ev = nullptr;
    if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess)
      return LUMEN_ERR_HIP;
    dev->rings.push_back(DeviceInfo::Ring{});
    r = &dev->rings.back();
    r->idle = ev;
  } else {
    r = &dev->rings[dev->ring_next];
    dev->ring_next = (dev->ring_next + 1) % kMaxRings;
  }
  r->staging = staging;
  r->recorded = false;
  *out = r;
  return LUMEN_OK;
}

// Start of a staging pipeline on `first` (the stream that writes the ring
// first): outside graph capture, wait until the previous pipeline call on
// the same ring has finished with it.  Sets *ring to the entry to record at
// the end, or to null while `first` is being captured (a captured graph
// cannot wait on work outside it; its launches are ordered by the stream
// they are launched on).
int ring_acquire(DeviceInfo *dev, const void *staging, hipStream_t first,
                 DeviceInfo::Ring **ring) {
  *ring = nullptr;
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(first, &cap) != hipSuccess) return LUMEN_ERR_HIP;
  if (cap != hipStreamCaptureStatusNone) return LUMEN_OK;
  DeviceInfo::Ring *r = nullptr;
  const int st = ring_entry(dev, staging, &r);
  if (st != LUMEN_OK) return st;
  if (r->recorded && hipStreamWaitEvent(first, r->idle, 0) != hipSuccess)
    return LUMEN_ERR_HIP;
  *ring = r;
  return LUMEN_OK;
}

// End of a staging pipeline: `last` is the stream whose work finishes the
// ring's use (the copies of pack_to_host, the unpacks of unpack_from_host).
int ring_release(DeviceInfo::Ring *ring, hipStream_t last) {
  if (!ring) return LUMEN_OK;
  if (hipEventRecord(ring->idle, last) != hipSuccess) return LUMEN_ERR_HIP;
  ring->recorded = true;
  return LUMEN_OK;
}

// Host-side checks shared by the two staging pipelines.
int check_pipeline(const lumen_kv_layout *lay, int32_t num_reqs,
                   const void *ws, int64_t total_rows, const void *staging,
                   int64_t slot_rows, int32_t slots, const void *host) {
  int st = check_layout(lay);
  if (st != LUMEN_OK) return st;
  if (num_reqs < 0 || total_rows < 0 || !ws) return LUMEN_ERR_INVALID_ARG;
  if (slots < 1 || slots > kMaxSlots || slot_rows < 1)
    return LUMEN_ERR_INVALID_ARG;
  if (total_rows > 0 && (!staging || !host)) return LUMEN_ERR_INVALID_ARG;
  if (!aligned16(ws) || !aligned16(staging)) return LUMEN_ERR_MISALIGNED;
  return LUMEN_OK;
}

// Shared body of the two direct host copies: the checkpoint side is pinned
// host memory, reached through its device address.
int direct_copy(bool pack, const lumen_kv_layout *layout, const void *cache,
                const void *h_ckpt, const int32_t *d_block_tables,
                int32_t bt_cols, int32_t num_reqs, void *d_workspace,
                int64_t row_begin, int64_t row_end, int64_t ckpt_first_row,
                int64_t ckpt_rows, int32_t workgroups, lumen_stream_t stream) {
  if (workgroups < 0 || workgroups > kMaxDirectWorkgroups)
    return LUMEN_ERR_INVALID_ARG;
  int st = check_layout(layout);
  if (st != LUMEN_OK) return st;
  if (num_reqs < 0 || bt_cols < 0 || ckpt_rows < 0 || !d_workspace)
    return LUMEN_ERR_INVALID_ARG;
  if (row_begin < 0 || row_end < row_begin || ckpt_first_row < 0)
    return LUMEN_ERR_INVALID_ARG;
  if (num_reqs == 0 || row_end == row_begin) return LUMEN_OK;
  void *dev_ptr = nullptr;
  if (ckpt_rows > 0) {
    // Memory the device cannot reach (pageable, or another process's) is
    // refused here, before anything is enqueued: the runtime must know the
    // pointer as pinned host memory and give its device address.
    if (!h_ckpt) return LUMEN_ERR_INVALID_ARG;
    hipPointerAttribute_t attr{};
    if (hipPointerGetAttributes(&attr, h_ckpt) != hipSuccess ||
        attr.type != hipMemoryTypeHost) {
      (void)hipGetLastError();  // the failed query is not a sticky error
      return LUMEN_ERR_INVALID_ARG;
    }
    if (hipHostGetDevicePointer(&dev_ptr, const_cast<void *>(h_ckpt), 0) !=
            hipSuccess ||
        !dev_ptr) {
      (void)hipGetLastError();
      return LUMEN_ERR_INVALID_ARG;
    }
  }
  const int64_t waves =
      int64_t(workgroups > 0 ? workgroups : kDirectWorkgroups) *
      kWavesPerBlock;
  return pack ? launch_copy(true, layout, cache, dev_ptr, d_block_tables,
                            bt_cols, num_reqs, d_workspace, row_begin,
                            row_end, ckpt_first_row, ckpt_rows, stream, waves)
              : launch_copy(false, layout, dev_ptr, const_cast<void *>(cache),
                            d_block_tables, bt_cols, num_reqs, d_workspace,
                            row_begin, row_end, ckpt_first_row, ckpt_rows,
                            stream, waves);
}

// Plan and copy in one launch over the ranges (the _ranges entry points).
int ranges_copy(bool pack, const lumen_kv_layout *lay, void *cache,
                const int32_t *bt, int32_t bt_cols, const int32_t *d_start,
                const int32_t *d_end, int32_t num_reqs, int64_t row_base,
                const int64_t *d_req_row_base, void *ckpt, int64_t ckpt_rows,
                int32_t *d_status, lumen_stream_t stream) {
  int st = check_layout(lay);
  if (st != LUMEN_OK) return st;
  if (num_reqs < 0 || bt_cols < 0 || ckpt_rows < 0 || !d_status)
    return LUMEN_ERR_INVALID_ARG;
  if (num_reqs > kRangesMaxReqs) return LUMEN_ERR_TOO_MANY;
  if (reinterpret_cast<uintptr_t>(d_status) & 3) return LUMEN_ERR_MISALIGNED;
  if (num_reqs > 0 && (!d_start || !d_end)) return LUMEN_ERR_INVALID_ARG;
  const Ranges ranges{d_start, d_end, d_req_row_base, row_base};
  return launch_copy(pack, lay, pack ? cache : ckpt, pack ? ckpt : cache, bt,
                     bt_cols, num_reqs, nullptr, 0, INT64_MAX, 0, ckpt_rows,
                     stream, 0, d_status, &ranges);
}
}  // namespace

extern "C" {

size_t lumen_kv_ckpt_plan_workspace_bytes(int32_t num_reqs) {
  return num_reqs < 0 ? 0 : ws_bytes(num_reqs);
}

int lumen_kv_ckpt_plan(const int32_t *d_start, const int32_t *d_end,
                       int32_t num_reqs, int64_t row_base,
                       const int64_t *d_req_row_base, void *d_workspace,
                       lumen_stream_t stream) {
  if (num_reqs < 0 || !d_workspace) return LUMEN_ERR_INVALID_ARG;
  if (num_reqs > 0 && (!d_start || !d_end)) return LUMEN_ERR_INVALID_ARG;
  if (!aligned16(d_workspace)) return LUMEN_ERR_MISALIGNED;
  DeviceInfo *dev = nullptr;
  int st = current_device(&dev);
  if (st != LUMEN_OK) return st;
  WsView v = ws_view(d_workspace, num_reqs);
  clear_pending_error();
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), 0,
                     static_cast<hipStream_t>(stream), d_start, d_end,
                     num_reqs, row_base, d_req_row_base, v.hdr, v.prefix,
                     v.first_row, v.start, &v.hdr->err);
  return hipGetLastError() == hipSuccess ? LUMEN_OK : LUMEN_ERR_HIP;
}

int lumen_kv_ckpt_pack(const lumen_kv_layout *layout, const void *d_cache,
                       const int32_t *d_block_tables, int32_t bt_cols,
                       int32_t num_reqs, void *d_workspace, void *d_ckpt,
                       int64_t ckpt_rows, lumen_stream_t stream) {
  return launch_copy(true, layout, d_cache, d_ckpt, d_block_tables, bt_cols,
                     num_reqs, d_workspace, 0, INT64_MAX, 0, ckpt_rows,
                     stream);
}

int lumen_kv_ckpt_pack_noalloc(const lumen_kv_layout *layout,
                               const void *d_cache,
                               const int32_t *d_block_tables, int32_t bt_cols,
                               const int32_t *d_start, const int32_t *d_end,
                               int32_t num_reqs, int64_t row_base,
                               const int64_t *d_req_row_base, void *d_ckpt,
                               int64_t ckpt_rows, int32_t *d_status,
                               lumen_stream_t stream) {
  // Every host check comes before the first launch, so that an argument
  // error enqueues nothing.
  int st = check_layout(layout);
  if (st != LUMEN_OK) return st;
  if (num_reqs < 0 || bt_cols < 0 || ckpt_rows < 0 || !d_status)
    return LUMEN_ERR_INVALID_ARG;
  if (num_reqs > kNoAllocMaxReqs) return LUMEN_ERR_TOO_MANY;
  if (reinterpret_cast<uintptr_t>(d_status) & 3) return LUMEN_ERR_MISALIGNED;
  if (num_reqs > 0) {
    if (!d_start || !d_end) return LUMEN_ERR_INVALID_ARG;
    st = check_copy_buffers(layout, d_cache, d_ckpt, d_block_tables, bt_cols,
                            ckpt_rows);
    if (st != LUMEN_OK) return st;
  }
  DeviceInfo *dev = nullptr;
  st = current_device(&dev);
  if (st != LUMEN_OK) return st;
  if (!dev->scratch) return LUMEN_ERR_HIP;
  // The plan overwrites everything the pack reads from the scratch (its
  // header and per-request arrays) and the status word, so nothing left by
  // an earlier call is seen.
  WsView v = ws_view(dev->scratch, num_reqs);
  clear_pending_error();
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), 0,
                     static_cast<hipStream_t>(stream), d_start, d_end,
                     num_reqs, row_base, d_req_row_base, v.hdr, v.prefix,
                     v.first_row, v.start, d_status);
  if (hipGetLastError() != hipSuccess) return LUMEN_ERR_HIP;
  return launch_copy(true, layout, d_cache, d_ckpt, d_block_tables, bt_cols,
                     num_reqs, dev->scratch, 0, INT64_MAX, 0, ckpt_rows,
                     stream, 0, d_status);
}

int lumen_kv_ckpt_unpack(const lumen_kv_layout *layout, void *d_cache,
                         const int32_t *d_block_tables, int32_t bt_cols,
                         int32_t num_reqs, void *d_workspace,
                         const void *d_ckpt, int64_t ckpt_rows,
                         lumen_stream_t stream) {
  return launch_copy(false, layout, d_ckpt, d_cache, d_block_tables, bt_cols,
                     num_reqs, d_workspace, 0, INT64_MAX, 0, ckpt_rows,
                     stream);
}

int lumen_kv_ckpt_pack_ranges(const lumen_kv_layout *layout,
                              const void *d_cache,
                              const int32_t *d_block_tables, int32_t bt_cols,
                              const int32_t *d_start, const int32_t *d_end,
                              int32_t num_reqs, int64_t row_base,
                              const int64_t *d_req_row_base, void *d_ckpt,
                              int64_t ckpt_rows, int32_t *d_status,
                              lumen_stream_t stream) {
  return ranges_copy(true, layout, const_cast<void *>(d_cache),
                     d_block_tables, bt_cols, d_start, d_end, num_reqs,
                     row_base, d_req_row_base, d_ckpt, ckpt_rows, d_status,
                     stream);
}

int lumen_kv_ckpt_unpack_ranges(const lumen_kv_layout *layout,
                                void *d_cache,
                                const int32_t *d_block_tables,
                                int32_t bt_cols, const int32_t *d_start,
                                const int32_t *d_end, int32_t num_reqs,
                                int64_t row_base,
                                const int64_t *d_req_row_base,
                                const void *d_ckpt, int64_t ckpt_rows,
                                int32_t *d_status, lumen_stream_t stream) {
  return ranges_copy(false, layout, d_cache, d_block_tables, bt_cols,
                     d_start, d_end, num_reqs, row_base, d_req_row_base,
                     const_cast<void *>(d_ckpt), ckpt_rows, d_status, stream);
}

int lumen_kv_ckpt_pack_rows(const lumen_kv_layout *layout, const void *d_cache,
                            const int32_t *d_block_tables, int32_t bt_cols,
                            int32_t num_reqs, void *d_workspace,
                            int64_t row_begin, int64_t row_end, void *d_ckpt,
                            int64_t ckpt_first_row, int64_t ckpt_rows,
                            lumen_stream_t stream) {
  return launch_copy(true, layout, d_cache, d_ckpt, d_block_tables, bt_cols,
                     num_reqs, d_workspace, row_begin, row_end,
                     ckpt_first_row, ckpt_rows, stream);
}

int lumen_kv_ckpt_unpack_rows(const lumen_kv_layout *layout, void *d_cache,
                              const int32_t *d_block_tables, int32_t bt_cols,
                              int32_t num_reqs, void *d_workspace,
                              int64_t row_begin, int64_t row_end,
                              const void *d_ckpt, int64_t ckpt_first_row,
                              int64_t ckpt_rows, lumen_stream_t stream) {
  return launch_copy(false, layout, d_ckpt, d_cache, d_block_tables, bt_cols,
                     num_reqs, d_workspace, row_begin, row_end,
                     ckpt_first_row, ckpt_rows, stream);
}

size_t lumen_kv_ckpt_marks_bytes(int64_t num_blocks) {
  if (num_blocks < 0) return 0;
  return size_t((num_blocks + 127) / 128) * 16;
}

int lumen_kv_ckpt_validate_targets(const lumen_kv_layout *layout,
                                   const int32_t *d_block_tables,
                                   int32_t bt_cols, int32_t num_reqs,
                                   void *d_workspace, void *d_marks,
                                   size_t marks_bytes, lumen_stream_t stream) {
  int st = check_layout(layout);
  if (st != LUMEN_OK) return st;
  if (num_reqs < 0 || bt_cols < 0 || !d_workspace) return LUMEN_ERR_INVALID_ARG;
  if (!aligned16(d_workspace) || !aligned16(d_marks)) return LUMEN_ERR_MISALIGNED;
  if (num_reqs == 0) return LUMEN_OK;
  const size_t need = lumen_kv_ckpt_marks_bytes(layout->num_blocks);
  if (marks_bytes < need || (!d_marks && need > 0) ||
      (!d_block_tables && bt_cols > 0))
    return LUMEN_ERR_INVALID_ARG;
  DeviceInfo *dev = nullptr;
  st = current_device(&dev);
  if (st != LUMEN_OK) return st;
  WsView v = ws_view(d_workspace, num_reqs);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t n16 = int64_t(need / 16);
  clear_pending_error();
  if (n16 > 0) {
    const int64_t cap = int64_t(dev->cus) * 4;
    int64_t blocks = (n16 + kBlockThreads - 1) / kBlockThreads;
    if (blocks > cap) blocks = cap;
    hipLaunchKernelGGL(clear_marks_kernel, dim3(unsigned(blocks)),
                       dim3(kBlockThreads), 0, s,
                       static_cast<uint4 *>(d_marks), n16);
  }
  const int32_t blocks = num_reqs < 65536 ? num_reqs : 65536;
  hipLaunchKernelGGL(validate_kernel, dim3(unsigned(blocks)),
                     dim3(kBlockThreads), 0, s, d_block_tables, v.hdr,
                     v.prefix, v.start, static_cast<uint32_t *>(d_marks),
                     &v.hdr->err, num_reqs, bt_cols, layout->block_size,
                     layout->num_blocks);
  return hipGetLastError() == hipSuccess ? LUMEN_OK : LUMEN_ERR_HIP;
}

int lumen_kv_ckpt_pack_to_host(const lumen_kv_layout *layout,
                               const void *d_cache,
                               const int32_t *d_block_tables, int32_t bt_cols,
                               int32_t num_reqs, void *d_workspace,
                               int64_t total_rows, void *d_staging,
                               int64_t slot_rows, int32_t slots, void *h_ckpt,
                               lumen_stream_t pack_stream,
                               lumen_stream_t copy_stream) {
  int st = check_pipeline(layout, num_reqs, d_workspace, total_rows, d_staging,
                          slot_rows, slots, h_ckpt);
  if (st != LUMEN_OK || total_rows == 0 || num_reqs == 0) return st;
  DeviceInfo *dev = nullptr;
  st = current_device(&dev);
  if (st != LUMEN_OK) return st;
  const int64_t row_bytes = int64_t(layout->num_layers) * 2 *
                            layout->num_kv_heads * layout->head_dim *
                            layout->elem_bytes;
  hipStream_t ps = static_cast<hipStream_t>(pack_stream);
  hipStream_t cs = static_cast<hipStream_t>(copy_stream);
  std::lock_guard<std::mutex> lock(dev->pipe_mu);
  st = pipe_events(dev, 2 * size_t(slots));
  if (st != LUMEN_OK) return st;
  hipEvent_t *packed = dev->pipe_events.data();
  hipEvent_t *copied = packed + slots;
  DeviceInfo::Ring *ring = nullptr;
  st = ring_acquire(dev, d_staging, ps, &ring);
  if (st != LUMEN_OK) return st;
  for (int64_t c = 0, lo = 0; lo < total_rows; ++c, lo += slot_rows) {
    const int64_t hi = lo + slot_rows < total_rows ? lo + slot_rows : total_rows;
    const int32_t j = int32_t(c % slots);
    uint8_t *slot = static_cast<uint8_t *>(d_staging) + j * slot_rows * row_bytes;
    // A slot is packed again only after its previous rows reached the host.
    if (c >= slots && hipStreamWaitEvent(ps, copied[j], 0) != hipSuccess)
      return LUMEN_ERR_HIP;
    st = launch_copy(true, layout, d_cache, slot, d_block_tables, bt_cols,
                     num_reqs, d_workspace, lo, hi, lo, slot_rows, ps);
    if (st != LUMEN_OK) return st;
    if (hipEventRecord(packed[j], ps) != hipSuccess ||
        hipStreamWaitEvent(cs, packed[j], 0) != hipSuccess ||
        hipMemcpyAsync(static_cast<uint8_t *>(h_ckpt) + lo * row_bytes, slot,
                       size_t((hi - lo) * row_bytes), hipMemcpyDeviceToHost,
                       cs) != hipSuccess ||
        hipEventRecord(copied[j], cs) != hipSuccess)
      return LUMEN_ERR_HIP;
  }
  return ring_release(ring, cs);
}

int lumen_kv_ckpt_unpack_from_host(const lumen_kv_layout *layout,
                                   void *d_cache,
                                   const int32_t *d_block_tables,
                                   int32_t bt_cols, int32_t num_reqs,
                                   void *d_workspace, int64_t total_rows,
                                   const void *h_ckpt, void *d_staging,
                                   int64_t slot_rows, int32_t slots,
                                   lumen_stream_t copy_stream,
                                   lumen_stream_t unpack_stream) {
  int st = check_pipeline(layout, num_reqs, d_workspace, total_rows, d_staging,
                          slot_rows, slots, h_ckpt);
  if (st != LUMEN_OK || total_rows == 0 || num_reqs == 0) return st;
  DeviceInfo *dev = nullptr;
  st = current_device(&dev);
  if (st != LUMEN_OK) return st;
  const int64_t row_bytes = int64_t(layout->num_layers) * 2 *
                            layout->num_kv_heads * layout->head_dim *
                            layout->elem_bytes;
  hipStream_t cs = static_cast<hipStream_t>(copy_stream);
  hipStream_t us = static_cast<hipStream_t>(unpack_stream);
  std::lock_guard<std::mutex> lock(dev->pipe_mu);
  st = pipe_events(dev, 2 * size_t(slots));
  if (st != LUMEN_OK) return st;
  hipEvent_t *staged = dev->pipe_events.data();
  hipEvent_t *drained = staged + slots;
  DeviceInfo::Ring *ring = nullptr;
  st = ring_acquire(dev, d_staging, cs, &ring);
  if (st != LUMEN_OK) return st;
  for (int64_t c = 0, lo = 0; lo < total_rows; ++c, lo += slot_rows) {
    const int64_t hi = lo + slot_rows < total_rows ? lo + slot_rows : total_rows;
    const int32_t j = int32_t(c % slots);
    uint8_t *slot = static_cast<uint8_t *>(d_staging) + j * slot_rows * row_bytes;
    // A slot is refilled only after the unpack of its previous rows.
    if (c >= slots && hipStreamWaitEvent(cs, drained[j], 0) != hipSuccess)
      return LUMEN_ERR_HIP;
    if (hipMemcpyAsync(slot, static_cast<const uint8_t *>(h_ckpt) + lo * row_bytes,
                       size_t((hi - lo) * row_bytes), hipMemcpyHostToDevice,
                       cs) != hipSuccess ||
        hipEventRecord(staged[j], cs) != hipSuccess ||
        hipStreamWaitEvent(us, staged[j], 0) != hipSuccess)
      return LUMEN_ERR_HIP;
    st = launch_copy(false, layout, slot, d_cache, d_block_tables, bt_cols,
                     num_reqs, d_workspace, lo, hi, lo, slot_rows, us);
    if (st != LUMEN_OK) return st;
    if (hipEventRecord(drained[j], us) != hipSuccess) return LUMEN_ERR_HIP;
  }
  return ring_release(ring, us);
}

int lumen_kv_ckpt_pack_to_host_direct(
    const lumen_kv_layout *layout, const void *d_cache,
    const int32_t *d_block_tables, int32_t bt_cols, int32_t num_reqs,
    void *d_workspace, int64_t row_begin, int64_t row_end, void *h_ckpt,
    int64_t ckpt_first_row, int64_t ckpt_rows, int32_t workgroups,
    lumen_stream_t stream) {
  return direct_copy(true, layout, d_cache, h_ckpt, d_block_tables, bt_cols,
                     num_reqs, d_workspace, row_begin, row_end,
                     ckpt_first_row, ckpt_rows, workgroups, stream);
}

int lumen_kv_ckpt_unpack_from_host_direct(
    const lumen_kv_layout *layout, void *d_cache,
    const int32_t *d_block_tables, int32_t bt_cols, int32_t num_reqs,
    void *d_workspace, int64_t row_begin, int64_t row_end,
    const void *h_ckpt, int64_t ckpt_first_row, int64_t ckpt_rows,
    int32_t workgroups, lumen_stream_t stream) {
  return direct_copy(false, layout, d_cache, h_ckpt, d_block_tables, bt_cols,
                     num_reqs, d_workspace, row_begin, row_end,
                     ckpt_first_row, ckpt_rows, workgroups, stream);
}

int lumen_kv_draft_align(const int32_t *d_draft, int32_t draft_cols,
                         const int32_t *d_draft_len,
                         const int32_t *d_committed, int32_t committed_cols,
                         const int32_t *d_committed_len, int32_t *d_kv_len,
                         int32_t *d_block_tables, int32_t bt_cols,
                         int32_t block_size, int32_t num_reqs,
                         int32_t *d_replay, int32_t *d_freed,
                         int64_t freed_cap, int64_t *d_freed_count,
                         void *d_workspace, lumen_stream_t stream) {
  if (num_reqs < 0 || draft_cols < 0 || committed_cols < 0 || bt_cols < 0 ||
      block_size < 1 || freed_cap < 0 || !d_workspace || !d_freed_count)
    return LUMEN_ERR_INVALID_ARG;
  if (!aligned16(d_workspace)) return LUMEN_ERR_MISALIGNED;
  if (num_reqs > 0 &&
      (!d_draft_len || !d_committed_len || !d_kv_len || !d_replay ||
       (!d_draft && draft_cols > 0) || (!d_committed && committed_cols > 0) ||
       (!d_block_tables && bt_cols > 0)))
    return LUMEN_ERR_INVALID_ARG;
  if (!d_freed && freed_cap > 0) return LUMEN_ERR_INVALID_ARG;
  DeviceInfo *dev = nullptr;
  int st = current_device(&dev);
  if (st != LUMEN_OK) return st;
  WsView v = ws_view(d_workspace, num_reqs);
  hipStream_t s = static_cast<hipStream_t>(stream);
  clear_pending_error();
  if (num_reqs > 0) {
    int64_t blocks = (int64_t(num_reqs) + kWavesPerBlock - 1) / kWavesPerBlock;
    const int64_t cap = int64_t(dev->cus) * 8;
    if (blocks > cap) blocks = cap;
    hipLaunchKernelGGL(draft_match_kernel, dim3(unsigned(blocks)),
                       dim3(kBlockThreads), 0, s, d_draft, draft_cols,
                       d_draft_len, d_committed, committed_cols,
                       d_committed_len, d_kv_len, d_block_tables, bt_cols,
                       block_size, num_reqs, d_replay, v.prefix, v.first_row);
  }
  hipLaunchKernelGGL(draft_free_kernel, dim3(1), dim3(kPlanThreads), 0, s,
                     d_block_tables, bt_cols, num_reqs, v.prefix, v.first_row,
                     d_freed, freed_cap, d_freed_count, v.hdr);
  return hipGetLastError() == hipSuccess ? LUMEN_OK : LUMEN_ERR_HIP;
}

int lumen_kv_ckpt_status(void *d_workspace, lumen_stream_t stream) {
  if (!d_workspace) return LUMEN_ERR_INVALID_ARG;
  if (!aligned16(d_workspace)) return LUMEN_ERR_MISALIGNED;
  hipStream_t s = static_cast<hipStream_t>(stream);
  WsHeader *hdr = static_cast<WsHeader *>(d_workspace);
  int32_t code = 0;
  static const int32_t zero = 0;
  if (hipMemcpyAsync(&code, &hdr->err, sizeof(code), hipMemcpyDeviceToHost,
                     s) != hipSuccess)
    return LUMEN_ERR_HIP;
  if (hipMemcpyAsync(&hdr->err, &zero, sizeof(zero), hipMemcpyHostToDevice,
                     s) != hipSuccess)
    return LUMEN_ERR_HIP;
  if (hipStreamSynchronize(s) != hipSuccess) return LUMEN_ERR_HIP;
  return code;
}

int lumen_kv_ckpt_time_next_copy(void *start_event, void *stop_event) {
  next_timing.start = static_cast<hipEvent_t>(start_event);
  next_timing.stop = static_cast<hipEvent_t>(stop_event);
  next_timing.armed = start_event || stop_event;
  return LUMEN_OK;
}

const char *lumen_kv_ckpt_strerror(int code) {
  switch (code) {
    case LUMEN_OK: return "ok";
    case LUMEN_ERR_INVALID_ARG: return "invalid argument";
    case LUMEN_ERR_UNSUPPORTED: return "unsupported layout";
    case LUMEN_ERR_MISALIGNED: return "buffer not 16-byte aligned";
    case LUMEN_ERR_HIP: return "HIP runtime error";
    case LUMEN_ERR_RANGE: return "token range outside the request or its block table";
    case LUMEN_ERR_BLOCK_ID: return "block table entry outside the pool";
    case LUMEN_ERR_CAPACITY:
      return "checkpoint row outside the checkpoint buffer, or host memory "
             "exhausted";
    case LUMEN_ERR_DUP_BLOCK: return "block named by two pages of an unpack";
    case LUMEN_ERR_TOO_MANY:
      return "more requests or token rows than the call takes in one launch";
    default: return "unknown status";
  }
}

int lumen_kv_ckpt_offload(const void *d_src, void *h_dst, size_t bytes,
                          lumen_stream_t producer, lumen_stream_t side) {
  if (bytes == 0) return LUMEN_OK;
  if (!d_src || !h_dst) return LUMEN_ERR_INVALID_ARG;
  DeviceInfo *dev = nullptr;
  int st = current_device(&dev);
  if (st != LUMEN_OK) return st;
  hipStream_t p = static_cast<hipStream_t>(producer);
  hipStream_t q = static_cast<hipStream_t>(side);
  {
    // A wait captures the event's latest record at the time of the call, so
    // one event per device serves every call.
    std::lock_guard<std::mutex> lock(dev->event_mu);
    if (hipEventRecord(dev->order_event, p) != hipSuccess ||
        hipStreamWaitEvent(q, dev->order_event, 0) != hipSuccess)
      return LUMEN_ERR_HIP;
  }
  if (hipMemcpyAsync(h_dst, d_src, bytes, hipMemcpyDeviceToHost, q) != hipSuccess)
    return LUMEN_ERR_HIP;
  return LUMEN_OK;
}

int lumen_kv_ckpt_stage_in(const void *h_src, void *d_dst, size_t bytes,
                           lumen_stream_t side, lumen_stream_t consumer) {
  if (bytes == 0) return LUMEN_OK;
  if (!h_src || !d_dst) return LUMEN_ERR_INVALID_ARG;
  DeviceInfo *dev = nullptr;
  int st = current_device(&dev);
  if (st != LUMEN_OK) return st;
  hipStream_t q = static_cast<hipStream_t>(side);
  hipStream_t c = static_cast<hipStream_t>(consumer);
  if (hipMemcpyAsync(d_dst, h_src, bytes, hipMemcpyHostToDevice, q) != hipSuccess)
    return LUMEN_ERR_HIP;
  std::lock_guard<std::mutex> lock(dev->event_mu);
  if (hipEventRecord(dev->order_event, q) != hipSuccess ||
      hipStreamWaitEvent(c, dev->order_event, 0) != hipSuccess)
    return LUMEN_ERR_HIP;
  return LUMEN_OK;
}

}  // extern "C"
