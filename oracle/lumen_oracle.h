/*
 * CPU oracle for the paged-KV checkpoint path.
 *
 * TEST INFRASTRUCTURE ONLY.  This is the plain, slow, obviously correct
 * statement of what checkpoint pack and restore unpack compute.  Only the
 * test suite, the smoke check and the benchmark's CPU-baseline leg may load
 * it; the GPU library never does, and the two share no code, headers or
 * tables.
 *
 * What is computed (LUMEN, Sec. 2.1 and Sec. 4.2-4.3):
 *  - The KV cache is paged: a page (block) holds the keys and values of a
 *    fixed number of consecutive token positions (Sec. 2.1).  Request r's
 *    block table maps its page j to a physical block of the pool.
 *  - After each prefill or decode batch only the tokens written since the
 *    last checkpoint are sent (Sec. 4.2, incremental checkpoint pipeline):
 *    the token range [start[r], end[r]) of each request.
 *  - On recovery the checkpointed prefix is loaded back into GPU memory, into
 *    whatever blocks the new block table names (Sec. 4.3, KV-reuse recovery).
 *
 * Layouts (an element is elem_bytes bytes -- 1 for an 8-bit cache, 2 for
 * bf16/fp16, 4 for fp32 -- moved as raw bits):
 *   token-major cache  [L][2][NB][block_size][H][D]
 *   head-major cache   [L][2][NB][H][block_size][D]
 *   checkpoint rows    [rows][L][2][H][D]      (index 0 of the "2" is K)
 *
 * Status codes share their numeric values with the GPU library's so that the
 * tests can compare them; the definitions are written out separately here.
 */
#ifndef LUMEN_ORACLE_H
#define LUMEN_ORACLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ORACLE_OK 0
#define ORACLE_ERR_INVALID_ARG (-1)
#define ORACLE_ERR_UNSUPPORTED (-2)
#define ORACLE_ERR_RANGE (-5)
#define ORACLE_ERR_BLOCK_ID (-6)
#define ORACLE_ERR_CAPACITY (-7)
#define ORACLE_ERR_DUP_BLOCK (-8)

typedef struct {
    int32_t num_layers;   /* L */
    int32_t num_kv_heads; /* H */
    int32_t head_dim;     /* D */
    int32_t block_size;   /* tokens per page */
    int64_t num_blocks;   /* NB, blocks in the pool */
    int32_t head_major;   /* 0: [L][2][NB][bs][H][D], 1: [L][2][NB][H][bs][D] */
    int32_t elem_bytes;   /* 1, 2 or 4 */
} oracle_cache_shape;

/* Row of each request's first checkpointed token.
 * Packed mode (req_row_base == NULL): requests are laid out one after the
 * other in request order starting at row_base.  Per-request mode: token t of
 * request r lives at row req_row_base[r] + t.
 * A request with start < 0 or end < start is a RANGE error and contributes no
 * rows.  Writes first_row[num_reqs] and *total_rows (rows of valid requests).
 * Returns ORACLE_OK or the most negative error code found. */
int oracle_plan(const int32_t *start, const int32_t *end, int32_t num_reqs,
                int64_t row_base, const int64_t *req_row_base,
                int64_t *first_row, int64_t *total_rows);

/* Gather: checkpoint[row(r,t)] <- cache tokens t in [start[r], end[r]).
 * Per token, checks in order: page index t / block_size < bt_cols (RANGE),
 * 0 <= block < num_blocks (BLOCK_ID), 0 <= row < ckpt_rows (CAPACITY).
 * The status is the most negative code over all requests and tokens; on any
 * error nothing is written. */
int oracle_pack(const oracle_cache_shape *shape, const void *cache,
                const int32_t *block_tables, int32_t bt_cols,
                const int32_t *start, const int32_t *end, int32_t num_reqs,
                int64_t row_base, const int64_t *req_row_base,
                void *ckpt, int64_t ckpt_rows);

/* Scatter: the inverse of oracle_pack under (possibly different) block
 * tables.  Only the slots of the named tokens are written. */
int oracle_unpack(const oracle_cache_shape *shape, void *cache,
                  const int32_t *block_tables, int32_t bt_cols,
                  const int32_t *start, const int32_t *end, int32_t num_reqs,
                  int64_t row_base, const int64_t *req_row_base,
                  const void *ckpt, int64_t ckpt_rows);

/* Validate mode of a restore.  Recovery loads pages into blocks that an
 * allocator hands out, one owner per block (Sec. 4.3), so a physical block
 * named by two written pages is a caller error.  The pages an unpack writes
 * are, for each request with a valid non-empty range, pages start/bs through
 * (end-1)/bs.  Each is checked: page < bt_cols (RANGE), block in the pool
 * (BLOCK_ID), and no block named by two such pages (DUP_BLOCK).  An invalid
 * range (start < 0 or end < start) is a RANGE error, as in oracle_plan.
 * Returns the most negative code found. */
int oracle_validate_targets(const oracle_cache_shape *shape,
                            const int32_t *block_tables, int32_t bt_cols,
                            const int32_t *start, const int32_t *end,
                            int32_t num_reqs);

#ifdef __cplusplus
}
#endif
#endif
