/*
 * lumen_kv_ckpt: paged KV-cache checkpoint and restore data movement on
 * MI355X (gfx950).
 *
 * LUMEN keeps a checkpoint of every in-flight request's KV cache so that a
 * request interrupted by a worker failure resumes from its checkpointed
 * prefix instead of re-running prefill (Sec. 4.2, load-aware KV
 * checkpointing; Sec. 4.3, KV-reuse recovery).  This library moves the bytes
 * of that scheme on one GPU:
 *
 *   plan    device prefix sum that assigns checkpoint rows to each request's
 *           token range [start, end)  (the newly written tokens, Sec. 4.2)
 *   pack    gather of those tokens out of the paged cache through each
 *           request's block table into contiguous token-major rows
 *           (the copy of new KV pages out of GPU memory, Sec. 4.2 step 3)
 *   unpack  scatter of checkpoint rows into the blocks a new block table
 *           names (loading the checkpointed pages back into GPU memory,
 *           Sec. 4.3)
 *   pack_ranges / unpack_ranges
 *           plan and pack (unpack) in one launch, straight from the token
 *           ranges, with no workspace: the copy plans its rows itself
 *   pack_noalloc
 *           plan and pack with the library's own device scratch, for
 *           callers that cannot allocate
 *   offload / stage_in
 *           device->pinned-host and pinned-host->device copies of packed
 *           rows on a side stream, ordered after (before) the main stream's
 *           work (the pinned CPU buffer of Sec. 4.2)
 *   pack_rows / unpack_rows
 *           a row range of a plan through a window of the checkpoint
 *   pack_to_host / unpack_from_host
 *           chunked pipelines through a small device staging ring: pack
 *           overlapped with the copy to host memory, and the copy from host
 *           memory overlapped with the unpack
 *   pack_to_host_direct / unpack_from_host_direct
 *           the gather writing, or the scatter reading, pinned host memory
 *           itself on a small grid: no staging ring and no copy engine
 *   time_next_copy
 *           the next copy kernel's own start and end, on two HIP events
 *   validate_targets
 *           validate mode of a restore (duplicate target blocks)
 *   draft_align
 *           draft-state alignment of speculation-assisted recovery: truncate
 *           the draft KV at the first token mismatch (Sec. 4.4)
 *
 * Layouts.  The cache is one allocation of elements of elem_bytes bytes
 * (2 for bf16/fp16, 1 for an 8-bit cache, 4 for fp32; always moved as raw
 * bits), layer-major, K before V:
 *   LUMEN_CACHE_NHD  [L][2][num_blocks][block_size][H][D]
 *   LUMEN_CACHE_HND  [L][2][num_blocks][H][block_size][D]
 * A block (page) holds block_size consecutive token positions of one request
 * (Sec. 2.1).  Block table row r, of bt_cols int32 entries, maps request r's
 * page j (tokens [j*block_size, (j+1)*block_size)) to a physical block.
 * A checkpoint row holds one token, all layers, K and V, token-major:
 *   row [L][2][H][D]   (row_bytes = L*2*H*D*elem_bytes)
 * so the rows of successive increments append to a request's checkpoint and
 * any prefix of rows is a token prefix (the longest checkpointed prefix that
 * recovery restores, Sec. 4.3).
 *
 * Ownership and ordering.  Every buffer is allocated and owned by the
 * caller; the library allocates no device memory.  All calls are
 * asynchronous and stream-ordered on the hipStream_t passed as `stream`
 * (NULL is the null stream), except lumen_kv_ckpt_status, which
 * synchronises that stream.  A workspace must not be shared by calls that
 * are in flight at the same time.
 *
 * Errors.  Argument errors the host can see are returned synchronously
 * (negative codes) and nothing is enqueued.  Errors that depend on device
 * data (ranges, block ids, capacity) are recorded in the workspace's error
 * word: the offending token rows are skipped, all other rows are still
 * copied, and the word keeps the most negative code seen.  (The one
 * exception is a copy past LUMEN_KV_CKPT_MAX_UNITS, which copies nothing.)  lumen_kv_ckpt_plan
 * starts a new error epoch (it overwrites the word with its own result);
 * lumen_kv_ckpt_status reads and clears it.  The calls without a workspace
 * (_ranges, _noalloc) record the same codes in a caller-owned status word
 * instead, as their comments say.
 */
#ifndef LUMEN_KV_CKPT_H
#define LUMEN_KV_CKPT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LUMEN_OK 0
#define LUMEN_ERR_INVALID_ARG (-1) /* null pointer, negative size, bad dims */
#define LUMEN_ERR_UNSUPPORTED (-2) /* elem_bytes not 1/2/4, unknown order,
                                      D*elem_bytes not a multiple of 16, a row
                                      of 2^31 or more 16-byte vectors, or
                                      H*D*elem_bytes or block_size*D*elem_bytes
                                      of 2^31 bytes or more */
#define LUMEN_ERR_MISALIGNED (-3)  /* cache/ckpt/workspace not 16-byte aligned */
#define LUMEN_ERR_HIP (-4)         /* a HIP runtime call failed */
#define LUMEN_ERR_RANGE (-5)       /* start < 0, end < start, or a page past bt_cols */
#define LUMEN_ERR_BLOCK_ID (-6)    /* block table entry outside [0, num_blocks) */
#define LUMEN_ERR_CAPACITY (-7)    /* checkpoint row outside [0, ckpt_rows); host libraries: out of host memory */
#define LUMEN_ERR_DUP_BLOCK (-8)   /* validate mode: a block named by two
                                      pages that an unpack would write */
#define LUMEN_ERR_TOO_MANY (-9)    /* more requests than the call takes:
                                      LUMEN_KV_CKPT_NOALLOC_MAX_REQS for
                                      lumen_kv_ckpt_pack_noalloc,
                                      LUMEN_KV_CKPT_RANGES_MAX_REQS for the
                                      _ranges calls; recorded by a copy
                                      whose ranges hold more than
                                      LUMEN_KV_CKPT_MAX_UNITS units */

/* Most requests lumen_kv_ckpt_pack_noalloc takes in one call. */
#ifndef LUMEN_KV_CKPT_NOALLOC_MAX_REQS
#define LUMEN_KV_CKPT_NOALLOC_MAX_REQS 16384
#endif

/* Most requests lumen_kv_ckpt_pack_ranges / _unpack_ranges take in one
 * call: every workgroup of their launch scans all the ranges into LDS. */
#define LUMEN_KV_CKPT_RANGES_MAX_REQS 4096

/* Most (token row, layer) units one copy launch walks.  A copy whose
 * ranges hold more (their token rows times num_layers; for the calls that
 * take a row window, the rows inside the window) records LUMEN_ERR_TOO_MANY
 * and copies nothing.  No checkpoint in device memory comes near it: 2^40
 * units of the smallest unit (32 bytes) are 32 TiB.  It keeps a malformed
 * call, such as ends of INT32_MAX on thousands of requests, from holding
 * the GPU for minutes over rows that are all invalid, and keeps the
 * launch's 64-bit index arithmetic in range. */
#define LUMEN_KV_CKPT_MAX_UNITS ((int64_t)1 << 40)

#define LUMEN_CACHE_NHD 0
#define LUMEN_CACHE_HND 1

/* A hipStream_t, passed as an opaque pointer so that this header does not
 * depend on the HIP headers. */
typedef void *lumen_stream_t;

typedef struct lumen_kv_layout {
    int32_t num_layers;   /* L */
    int32_t num_kv_heads; /* H: KV heads held by this GPU */
    int32_t head_dim;     /* D; D*elem_bytes must be a multiple of 16 */
    int32_t block_size;   /* tokens per block (page) */
    int64_t num_blocks;   /* blocks in the pool */
    int32_t elem_bytes;   /* 1, 2 or 4 (fp8 / bf16 or fp16 / fp32; raw bits) */
    int32_t cache_order;  /* LUMEN_CACHE_NHD or LUMEN_CACHE_HND */
} lumen_kv_layout;

/* Bytes of device workspace a plan over num_reqs requests needs (header,
 * per-request row offsets and starts).  Returns 0 if num_reqs < 0. */
size_t lumen_kv_ckpt_plan_workspace_bytes(int32_t num_reqs);

/* Row plan for one set of token ranges (Sec. 4.2: only tokens written since
 * the last checkpoint are sent).  Device inputs d_start[num_reqs],
 * d_end[num_reqs] (int32).  Request r contributes n_r = end-start rows.
 * Rows are packed (d_req_row_base == NULL): request r's first row is
 * row_base + sum_{r'<r} n_r', in request order; or per-request
 * (d_req_row_base = device int64[num_reqs]): token t of request r goes to
 * row d_req_row_base[r] + t, so each request appends to its own reserved
 * checkpoint region.  A request with start < 0 or end < start contributes
 * no rows and records LUMEN_ERR_RANGE.  One plan serves any number of pack
 * and unpack calls over the same ranges.  d_workspace: device memory of
 * lumen_kv_ckpt_plan_workspace_bytes(num_reqs) bytes, 16-byte aligned. */
int lumen_kv_ckpt_plan(const int32_t *d_start, const int32_t *d_end,
                       int32_t num_reqs, int64_t row_base,
                       const int64_t *d_req_row_base, void *d_workspace,
                       lumen_stream_t stream);

/* Checkpoint gather (Sec. 4.2, copy of new KV pages out of GPU memory): for
 * every request r of the plan and token t in [start_r, end_r), copies the
 * token's K and V of every layer from block d_block_tables[r*bt_cols +
 * t/block_size], slot t % block_size, of d_cache into checkpoint row
 * row(r, t) of d_ckpt, which has room for ckpt_rows rows.  Per token row,
 * checked in this order: page t/block_size < bt_cols (RANGE); block id in
 * [0, num_blocks) (BLOCK_ID); row in [0, ckpt_rows) (CAPACITY).  num_reqs
 * must equal the plan's.  d_cache and d_ckpt 16-byte aligned; a buffer may
 * be NULL only if it is empty (num_blocks, ckpt_rows or bt_cols is 0).
 *
 * Grid size.  The plan's row count lives in device memory, so the launch is
 * sized without it: 384 wavefronts per CU, or 768 when a (row, layer) unit
 * is shorter than 4 KiB (LUMEN_KV_CKPT_WAVES_PER_CU in the environment
 * overrides both), but never more than one per (row, layer) unit that
 * ckpt_rows (or the row range of the _rows calls) could hold, nor more than
 * one per 4 KiB of it when that still leaves 16 per CU.  A checkpoint
 * buffer or window sized to the plan's rows keeps small steps free of idle
 * wavefronts: the pack of an 8-request Llama-3-8B-shaped decode step (65
 * rows) takes 8.4 us into a buffer of its rows and 20-31 us into a
 * multi-step arena, whose size sets the grid.
 *
 * Walk.  A pack of a token-major cache whose token runs (H*D*elem_bytes
 * bytes per layer and K/V) are at most 512 bytes is done page by page: whole
 * page runs are read, and each token's piece is written to its row.  The
 * environment variable LUMEN_KV_CKPT_PAGE_MAJOR=0 or 1 forces this off or
 * on.  The result and the status are the same either way. */
int lumen_kv_ckpt_pack(const lumen_kv_layout *layout, const void *d_cache,
                       const int32_t *d_block_tables, int32_t bt_cols,
                       int32_t num_reqs, void *d_workspace, void *d_ckpt,
                       int64_t ckpt_rows, lumen_stream_t stream);

/* Plan and pack in one call that allocates nothing, for callers that cannot
 * allocate device memory or be handed a workspace: code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation.  The same
 * as lumen_kv_ckpt_plan(d_start, d_end, num_reqs, row_base, d_req_row_base,
 * ws, stream) followed by lumen_kv_ckpt_pack(layout, d_cache,
 * d_block_tables, bt_cols, num_reqs, ws, d_ckpt, ckpt_rows, stream), with
 * the workspace ws replaced by a device array the library holds (one per
 * GPU, about 460 KB, kept until the process ends) and the status written to
 * d_status (caller-owned device int32, 4-byte aligned): the most negative
 * code the plan and the pack recorded, 0 if none, once the stream has
 * passed the call.  The caller still owns every input and output.
 * Calls no allocating routine.  num_reqs above
 * LUMEN_KV_CKPT_NOALLOC_MAX_REQS returns LUMEN_ERR_TOO_MANY and enqueues
 * nothing.  Every call on a GPU shares that GPU's array: calls that overlap
 * on one GPU (two streams, or two host threads, with no ordering between
 * them) race and give undefined results; calls ordered on one stream are
 * safe, since each call's plan rewrites what its pack reads. */
int lumen_kv_ckpt_pack_noalloc(const lumen_kv_layout *layout,
                               const void *d_cache,
                               const int32_t *d_block_tables, int32_t bt_cols,
                               const int32_t *d_start, const int32_t *d_end,
                               int32_t num_reqs, int64_t row_base,
                               const int64_t *d_req_row_base, void *d_ckpt,
                               int64_t ckpt_rows, int32_t *d_status,
                               lumen_stream_t stream);

/* Restore scatter (Sec. 4.3, loading checkpointed pages into GPU memory):
 * the inverse of lumen_kv_ckpt_pack under d_block_tables (usually freshly
 * allocated, fragmented blocks).  Writes only the slots of the planned
 * tokens; every other byte of d_cache is left untouched.  Two planned tokens
 * mapping to the same (block, slot) race; the allocator must not do that
 * (lumen_kv_ckpt_validate_targets checks for it). */
int lumen_kv_ckpt_unpack(const lumen_kv_layout *layout, void *d_cache,
                         const int32_t *d_block_tables, int32_t bt_cols,
                         int32_t num_reqs, void *d_workspace,
                         const void *d_ckpt, int64_t ckpt_rows,
                         lumen_stream_t stream);

/* Plan and copy in one launch (Sec. 4.2's incremental checkpoint of the
 * tokens written since the last one, and Sec. 4.3's restore): the same
 * rows, bytes and device-detected errors as lumen_kv_ckpt_plan(d_start,
 * d_end, num_reqs, row_base, d_req_row_base, ws, stream) followed by
 * lumen_kv_ckpt_pack (or _unpack) over ws, but with no workspace and no
 * plan kernel: each workgroup of the copy scans the ranges (device int32
 * [num_reqs] each) into 8 * (num_reqs + 5) bytes of its LDS, which saves
 * the plan's launch and the wait for it on every call.  The walk is
 * lumen_kv_ckpt_pack's: page by page for a pack of a token-major cache
 * with token runs of at most 512 bytes (for up to 2,048 requests; the
 * page-major walk keeps token and page prefixes, 16 * (num_reqs + 5) bytes
 * of LDS), token by token otherwise.  The grid is sized as for
 * lumen_kv_ckpt_pack; where a (token, layer) unit of the token-major walk
 * is 4 KiB or more, it has half as many wavefronts, each copying two spans
 * of it, so that one scan serves both.
 *
 * Status.  d_status is a caller-owned device int32, 4-byte aligned.  A call
 * only lowers it (atomic minimum) to the most negative code it records and
 * never sets it back: write LUMEN_OK to it before the first call; it then
 * holds the most negative code of every call since, once the stream has
 * passed them, so a loop of steps can check it once.  An invalid range
 * (start < 0 or end < start) records LUMEN_ERR_RANGE and copies no rows for
 * that request, as the plan does.
 *
 * Host errors (nothing enqueued): those of the plan and the copy, NULL
 * d_status (INVALID_ARG), d_status not 4-byte aligned (MISALIGNED), and
 * num_reqs above LUMEN_KV_CKPT_RANGES_MAX_REQS (TOO_MANY).  num_reqs == 0
 * enqueues nothing and leaves d_status as it is. */
int lumen_kv_ckpt_pack_ranges(const lumen_kv_layout *layout,
                              const void *d_cache,
                              const int32_t *d_block_tables, int32_t bt_cols,
                              const int32_t *d_start, const int32_t *d_end,
                              int32_t num_reqs, int64_t row_base,
                              const int64_t *d_req_row_base, void *d_ckpt,
                              int64_t ckpt_rows, int32_t *d_status,
                              lumen_stream_t stream);

/* The inverse of lumen_kv_ckpt_pack_ranges, as lumen_kv_ckpt_unpack is of
 * lumen_kv_ckpt_pack: checkpoint rows into the planned tokens' slots of
 * d_cache under d_block_tables; every other byte of d_cache is left
 * untouched.  Status, limits and errors as lumen_kv_ckpt_pack_ranges. */
int lumen_kv_ckpt_unpack_ranges(const lumen_kv_layout *layout,
                                void *d_cache,
                                const int32_t *d_block_tables,
                                int32_t bt_cols, const int32_t *d_start,
                                const int32_t *d_end, int32_t num_reqs,
                                int64_t row_base,
                                const int64_t *d_req_row_base,
                                const void *d_ckpt, int64_t ckpt_rows,
                                int32_t *d_status, lumen_stream_t stream);

/* Part of a pack, through a window of the checkpoint.  Copies only the
 * plan's packed rows [row_begin, row_end), clipped to the plan's total;
 * packed row i is the i-th planned token in request order, so a sequence
 * of calls over consecutive row ranges does the whole pack in pieces (the
 * chunks of Sec. 4.2's pipelined copy to pinned host memory).  d_ckpt
 * holds the checkpoint rows [ckpt_first_row, ckpt_first_row + ckpt_rows):
 * the token of checkpoint row c goes to buffer row c - ckpt_first_row, and
 * a row outside the window is a CAPACITY error.  With a packed-mode plan
 * from row_base 0, checkpoint row = packed row, so the window of rows
 * [row_begin, row_end) is exactly a buffer of row_end - row_begin rows.
 * row_begin <= row_end, both >= 0, ckpt_first_row >= 0 (INVALID_ARG).
 * lumen_kv_ckpt_pack is this call with rows [0, INT64_MAX) and window 0. */
int lumen_kv_ckpt_pack_rows(const lumen_kv_layout *layout, const void *d_cache,
                            const int32_t *d_block_tables, int32_t bt_cols,
                            int32_t num_reqs, void *d_workspace,
                            int64_t row_begin, int64_t row_end, void *d_ckpt,
                            int64_t ckpt_first_row, int64_t ckpt_rows,
                            lumen_stream_t stream);

/* Part of an unpack, through a window of the checkpoint: the inverse of
 * lumen_kv_ckpt_pack_rows, with the same row range and window rules. */
int lumen_kv_ckpt_unpack_rows(const lumen_kv_layout *layout, void *d_cache,
                              const int32_t *d_block_tables, int32_t bt_cols,
                              int32_t num_reqs, void *d_workspace,
                              int64_t row_begin, int64_t row_end,
                              const void *d_ckpt, int64_t ckpt_first_row,
                              int64_t ckpt_rows, lumen_stream_t stream);

/* Checkpoint straight to host memory (Sec. 4.2, steps 3 and 4 on one GPU:
 * the new tokens are copied out of GPU memory into a pinned CPU buffer by
 * background work while serving continues).  The plan's rows are packed in
 * chunks of slot_rows rows into a device staging ring of `slots` slots
 * (d_staging: slots * slot_rows rows, 16-byte aligned) on pack_stream, and
 * each chunk is copied to h_ckpt on copy_stream as soon as it is packed;
 * a slot is reused only after its previous copy has finished, so at most
 * `slots` chunks are in flight and the device needs no full-size
 * checkpoint buffer.  h_ckpt (host, pinned for overlap) receives packed rows
 * [0, total_rows) in order, row i at byte i * row_bytes.
 * The plan must be packed-mode from row_base 0 and enqueued before (on
 * pack_stream, or ordered before it); total_rows must equal its total (the
 * caller knows it: the sum of its ranges).  Both streams must differ from
 * the serving stream for the work to stay off it.  Returns after enqueuing;
 * the copies are complete once copy_stream has drained.  1 <= slots <= 64,
 * slot_rows >= 1 (INVALID_ARG).  Device errors go to the workspace word.
 *
 * Reuse of the staging ring.  The ring is busy until the last stream that
 * touches it (copy_stream here, unpack_stream in the restore) has passed
 * this call's work.  A later pipeline call (either direction) with the same
 * d_staging pointer on the same device waits for that on its own, outside
 * graph capture: its first stream to write the ring waits on an event the
 * earlier call recorded.  The library remembers the last 16 rings per
 * device.  The caller orders every other reuse: a ring reached through a
 * different pointer (an overlapping view), a 17th ring, or a call being
 * captured into a graph. */
int lumen_kv_ckpt_pack_to_host(const lumen_kv_layout *layout,
                               const void *d_cache,
                               const int32_t *d_block_tables, int32_t bt_cols,
                               int32_t num_reqs, void *d_workspace,
                               int64_t total_rows, void *d_staging,
                               int64_t slot_rows, int32_t slots, void *h_ckpt,
                               lumen_stream_t pack_stream,
                               lumen_stream_t copy_stream);

/* Restore straight from host memory (Sec. 4.3, loading the checkpointed
 * pages back into GPU memory): the inverse pipeline.  Chunks of slot_rows
 * rows of h_ckpt (packed rows in order, as lumen_kv_ckpt_pack_to_host
 * writes them) are copied into the staging ring on copy_stream, and each is
 * unpacked on unpack_stream as soon as it has arrived; a slot is refilled
 * only after its previous unpack.  Same plan, total_rows and slot rules as
 * lumen_kv_ckpt_pack_to_host, and the same reuse rule for the ring; the
 * restore is complete once unpack_stream has drained. */
int lumen_kv_ckpt_unpack_from_host(const lumen_kv_layout *layout,
                                   void *d_cache,
                                   const int32_t *d_block_tables,
                                   int32_t bt_cols, int32_t num_reqs,
                                   void *d_workspace, int64_t total_rows,
                                   const void *h_ckpt, void *d_staging,
                                   int64_t slot_rows, int32_t slots,
                                   lumen_stream_t copy_stream,
                                   lumen_stream_t unpack_stream);

/* Checkpoint rows straight into pinned host memory, with no device staging
 * (Sec. 4.2, steps 3 and 4 on one GPU): the gather kernel writes each row
 * to host memory across the host link itself.  The same operation as
 * lumen_kv_ckpt_pack_rows (same plan, row range and window rules; CAPACITY
 * for rows outside the window) with d_ckpt replaced by h_ckpt, host memory
 * of at least ckpt_rows rows that the device can address: memory from
 * hipHostMalloc (torch's pin_memory).  Other memory is refused with
 * INVALID_ARG before anything is enqueued.  The grid is `workgroups`
 * workgroups of 256 threads (0: 64, which reaches the link rate on MI355X;
 * at most 4096), so the copy holds a few CU slots rather than the chip
 * while it waits on the link.  The rows are in host memory once `stream`
 * has drained past the call.  One kernel, no events: the call can be
 * captured in a graph.  h_ckpt must stay allocated until then. */
int lumen_kv_ckpt_pack_to_host_direct(const lumen_kv_layout *layout,
                                      const void *d_cache,
                                      const int32_t *d_block_tables,
                                      int32_t bt_cols, int32_t num_reqs,
                                      void *d_workspace, int64_t row_begin,
                                      int64_t row_end, void *h_ckpt,
                                      int64_t ckpt_first_row,
                                      int64_t ckpt_rows, int32_t workgroups,
                                      lumen_stream_t stream);

/* Restore straight from pinned host memory (Sec. 4.3): the scatter kernel
 * reads each checkpoint row from host memory across the host link itself.
 * The inverse of lumen_kv_ckpt_pack_to_host_direct; the same operation as
 * lumen_kv_ckpt_unpack_rows with d_ckpt replaced by h_ckpt, and the same
 * host memory, grid and ordering rules.  h_ckpt must not be written by the
 * host until `stream` has drained past the call. */
int lumen_kv_ckpt_unpack_from_host_direct(const lumen_kv_layout *layout,
                                          void *d_cache,
                                          const int32_t *d_block_tables,
                                          int32_t bt_cols, int32_t num_reqs,
                                          void *d_workspace,
                                          int64_t row_begin, int64_t row_end,
                                          const void *h_ckpt,
                                          int64_t ckpt_first_row,
                                          int64_t ckpt_rows,
                                          int32_t workgroups,
                                          lumen_stream_t stream);

/* Bytes of the mark buffer lumen_kv_ckpt_validate_targets needs for a pool
 * of num_blocks blocks: one bit per block, rounded up to 16 bytes.  Returns
 * 0 if num_blocks < 0. */
size_t lumen_kv_ckpt_marks_bytes(int64_t num_blocks);

/* Validate mode of a restore.  Recovery loads pages into blocks that an
 * allocator hands out, one owner per block (Sec. 4.3), so a physical block
 * named by two pages that an unpack writes is a caller error; the unpack
 * itself does not look for it.  Run after lumen_kv_ckpt_plan and before the
 * unpack, with the same plan and table.  The pages an unpack writes are,
 * for every request with a non-empty planned range [start, end), pages
 * start/block_size through (end-1)/block_size.  Each is checked: page <
 * bt_cols (RANGE); block id in [0, num_blocks) (BLOCK_ID); no block named by
 * two such pages (DUP_BLOCK).  Results go to the workspace's error word like
 * the copies' (most negative code wins; read with lumen_kv_ckpt_status).
 * d_marks: caller-owned device scratch of marks_bytes >=
 * lumen_kv_ckpt_marks_bytes(num_blocks) bytes, 16-byte aligned, cleared by
 * this call (by a kernel, not a memset); it may be NULL only if num_blocks
 * is 0.  Calls sharing d_marks must not be in flight at the same time.
 * Nothing in the cache or the checkpoint is read or written. */
int lumen_kv_ckpt_validate_targets(const lumen_kv_layout *layout,
                                   const int32_t *d_block_tables,
                                   int32_t bt_cols, int32_t num_reqs,
                                   void *d_workspace, void *d_marks,
                                   size_t marks_bytes, lumen_stream_t stream);

/* Draft-state alignment (Sec. 4.4): after a progress update, the recovering
 * worker's draft KV stays valid only up to the first position where its
 * draft tokens and the authoritative committed tokens differ (compared by
 * position, not value).  For each request r:
 *   p = first i < min(draft_len, committed_len) with draft[i] !=
 *       committed[i], else that minimum;
 *   kv_len[r] <- valid = min(kv_len[r], p)          (in place);
 *   replay[r] <- committed_len[r] - valid  (committed tokens to run through
 *                                           the draft model again);
 *   pages ceil(valid/bs) .. ceil(old kv_len/bs) - 1 of its table are freed:
 *   their entries become -1 and their block ids (entries < 0 skipped) go
 *   to d_freed in request order, then page order.
 * *d_freed_count receives the number of freed blocks.  If it exceeds
 * freed_cap, only the first freed_cap are listed and cleared (the others
 * stay in their tables) and CAPACITY is recorded.  A request with negative
 * lengths, lengths past draft_cols / committed_cols, or kv_len past
 * bt_cols * block_size is left unchanged (replay 0) and RANGE is recorded.
 * Layouts: d_draft [R][draft_cols], d_committed [R][committed_cols],
 * d_block_tables [R][bt_cols] (int32, row-major); lengths [R] int32.
 * d_workspace: a workspace of lumen_kv_ckpt_plan_workspace_bytes(R) bytes;
 * the call starts a new error epoch there (read it with
 * lumen_kv_ckpt_status) and the workspace holds no copy plan afterwards. */
int lumen_kv_draft_align(const int32_t *d_draft, int32_t draft_cols,
                         const int32_t *d_draft_len,
                         const int32_t *d_committed, int32_t committed_cols,
                         const int32_t *d_committed_len, int32_t *d_kv_len,
                         int32_t *d_block_tables, int32_t bt_cols,
                         int32_t block_size, int32_t num_reqs,
                         int32_t *d_replay, int32_t *d_freed,
                         int64_t freed_cap, int64_t *d_freed_count,
                         void *d_workspace, lumen_stream_t stream);

/* Synchronises `stream`, then returns and clears the workspace's error word
 * (LUMEN_OK if no device-side error was recorded since the last plan). */
int lumen_kv_ckpt_status(void *d_workspace, lumen_stream_t stream);

/* Static string for a status code. */
const char *lumen_kv_ckpt_strerror(int code);

/* Times the next copy kernel this host thread launches, for callers that
 * want a kernel's own duration with no marker commands of theirs on the
 * stream around it (benchmarks, profilers).  start_event and stop_event
 * are hipEvent_t handles created with timing enabled (either may be NULL).
 * The next gather or scatter kernel of this thread (of a pack, unpack,
 * their _rows, _ranges, _noalloc and _direct forms, or the first chunk of
 * a pipeline) is launched through hipExtLaunchKernel with these events:
 * `start` takes the time that kernel starts and `stop` the time it ends,
 * so hipEventElapsedTime(start, stop) is its duration.  Plan and scan
 * kernels are not timed.  Calls that launch no copy kernel (empty or
 * refused ones) leave the pair armed; the launch that uses it clears it.
 * Passing two NULLs disarms it.  Returns LUMEN_OK. */
int lumen_kv_ckpt_time_next_copy(void *start_event, void *stop_event);

/* Device -> host copy of `bytes` from d_src to h_dst on stream `side`,
 * ordered after all work enqueued on `producer` so far, so the main stream
 * goes on without waiting (Sec. 4.2: the background copy of new pages to a
 * pinned CPU buffer).  h_dst should be pinned (hipHostMalloc) for the copy
 * to overlap. The caller synchronises `side` before reading h_dst. */
int lumen_kv_ckpt_offload(const void *d_src, void *h_dst, size_t bytes,
                          lumen_stream_t producer, lumen_stream_t side);

/* Host -> device copy of `bytes` from h_src to d_dst on stream `side`; work
 * enqueued on `consumer` afterwards waits for it (restore from a host
 * checkpoint store, Sec. 4.3). */
int lumen_kv_ckpt_stage_in(const void *h_src, void *d_dst, size_t bytes,
                           lumen_stream_t side, lumen_stream_t consumer);

#ifdef __cplusplus
}
#endif
#endif /* LUMEN_KV_CKPT_H */
