/*
 * CPU oracle for the paged-KV checkpoint path.  TEST INFRASTRUCTURE ONLY:
 * loaded by the tests, the smoke check and the benchmark's CPU-baseline leg,
 * never by the GPU library.  Plain loops over block tables, one element at a
 * time, in the order the definition reads.  See lumen_oracle.h for the
 * layouts and the passages each function follows.
 */
#include "lumen_oracle.h"

#include <stdlib.h>
#include <string.h>

/* Element offset of (layer l, k-or-v kv, block b, slot s, head h, dim d) in
 * the paged cache (Sec. 2.1: a page holds consecutive token positions). */
static int64_t cache_index(const oracle_cache_shape *sh, int64_t l, int64_t kv,
                           int64_t b, int64_t s, int64_t h, int64_t d)
{
    const int64_t NB = sh->num_blocks, bs = sh->block_size;
    const int64_t H = sh->num_kv_heads, D = sh->head_dim;
    if (sh->head_major)
        return ((((l * 2 + kv) * NB + b) * H + h) * bs + s) * D + d;
    return ((((l * 2 + kv) * NB + b) * bs + s) * H + h) * D + d;
}

/* Element offset of (row, layer l, kv, head h, dim d) in the checkpoint. */
static int64_t ckpt_index(const oracle_cache_shape *sh, int64_t row, int64_t l,
                          int64_t kv, int64_t h, int64_t d)
{
    const int64_t L = sh->num_layers, H = sh->num_kv_heads;
    const int64_t D = sh->head_dim;
    return (((row * L + l) * 2 + kv) * H + h) * D + d;
}

static int worse(int a, int b) { return a < b ? a : b; }

int oracle_plan(const int32_t *start, const int32_t *end, int32_t num_reqs,
                int64_t row_base, const int64_t *req_row_base,
                int64_t *first_row, int64_t *total_rows)
{
    if (num_reqs < 0)
        return ORACLE_ERR_INVALID_ARG;
    if (num_reqs > 0 && (!start || !end || !first_row))
        return ORACLE_ERR_INVALID_ARG;
    int status = ORACLE_OK;
    int64_t next = row_base, total = 0;
    for (int32_t r = 0; r < num_reqs; ++r) {
        int64_t n = (int64_t)end[r] - (int64_t)start[r];
        if (start[r] < 0 || n < 0) {
            status = worse(status, ORACLE_ERR_RANGE);
            n = 0;
        }
        if (req_row_base)
            first_row[r] = req_row_base[r] + start[r];
        else
            first_row[r] = next;
        next += n;
        total += n;
    }
    if (total_rows)
        *total_rows = total;
    return status;
}

static int check_shape(const oracle_cache_shape *sh)
{
    if (!sh)
        return ORACLE_ERR_INVALID_ARG;
    if (sh->num_layers <= 0 || sh->num_kv_heads <= 0 || sh->head_dim <= 0 ||
        sh->block_size <= 0 || sh->num_blocks < 0)
        return ORACLE_ERR_INVALID_ARG;
    if (sh->head_major != 0 && sh->head_major != 1)
        return ORACLE_ERR_UNSUPPORTED;
    if (sh->elem_bytes != 1 && sh->elem_bytes != 2 && sh->elem_bytes != 4)
        return ORACLE_ERR_UNSUPPORTED;
    return ORACLE_OK;
}

/* Validates every token of every request against the block tables and the
 * checkpoint capacity, in the order documented in the header. */
static int check_tokens(const oracle_cache_shape *sh, const int32_t *block_tables,
                        int32_t bt_cols, const int32_t *start,
                        const int32_t *end, int32_t num_reqs,
                        const int64_t *first_row, int64_t ckpt_rows)
{
    int status = ORACLE_OK;
    for (int32_t r = 0; r < num_reqs; ++r) {
        if (start[r] < 0 || end[r] < start[r])
            continue; /* already a RANGE error, contributes no tokens */
        for (int64_t t = start[r]; t < end[r]; ++t) {
            int64_t page = t / sh->block_size;
            if (page >= bt_cols) {
                status = worse(status, ORACLE_ERR_RANGE);
                continue;
            }
            int64_t b = block_tables[(int64_t)r * bt_cols + page];
            if (b < 0 || b >= sh->num_blocks) {
                status = worse(status, ORACLE_ERR_BLOCK_ID);
                continue;
            }
            int64_t row = first_row[r] + (t - start[r]);
            if (row < 0 || row >= ckpt_rows)
                status = worse(status, ORACLE_ERR_CAPACITY);
        }
    }
    return status;
}

/* Shared argument handling of pack and unpack: shape, pointers, plan. */
static int prepare(const oracle_cache_shape *sh, const void *cache,
                   const int32_t *block_tables, int32_t bt_cols,
                   const int32_t *start, const int32_t *end, int32_t num_reqs,
                   int64_t row_base, const int64_t *req_row_base,
                   const void *ckpt, int64_t ckpt_rows, int64_t *first_row)
{
    int st = check_shape(sh);
    if (st != ORACLE_OK)
        return st;
    if (num_reqs < 0 || bt_cols < 0 || ckpt_rows < 0)
        return ORACLE_ERR_INVALID_ARG;
    if (num_reqs > 0 && (!cache || !block_tables || !start || !end || !ckpt))
        return ORACLE_ERR_INVALID_ARG;
    st = oracle_plan(start, end, num_reqs, row_base, req_row_base, first_row,
                     0);
    st = worse(st, check_tokens(sh, block_tables, bt_cols, start, end,
                                num_reqs, first_row, ckpt_rows));
    return st;
}

/* Copies element `from` of `src` to element `to` of `dst`. */
static void copy_elem(void *dst, int64_t to, const void *src, int64_t from,
                      int32_t elem_bytes)
{
    memcpy((unsigned char *)dst + to * elem_bytes,
           (const unsigned char *)src + from * elem_bytes, (size_t)elem_bytes);
}

int oracle_pack(const oracle_cache_shape *sh, const void *cache,
                const int32_t *block_tables, int32_t bt_cols,
                const int32_t *start, const int32_t *end, int32_t num_reqs,
                int64_t row_base, const int64_t *req_row_base, void *ckpt,
                int64_t ckpt_rows)
{
    int64_t *first_row = malloc(sizeof(int64_t) * (num_reqs > 0 ? num_reqs : 1));
    if (!first_row)
        return ORACLE_ERR_INVALID_ARG;
    int st = prepare(sh, cache, block_tables, bt_cols, start, end, num_reqs,
                     row_base, req_row_base, ckpt, ckpt_rows, first_row);
    if (st != ORACLE_OK) {
        free(first_row);
        return st;
    }
    for (int32_t r = 0; r < num_reqs; ++r) {
        for (int64_t t = start[r]; t < end[r]; ++t) {
            int64_t b = block_tables[(int64_t)r * bt_cols + t / sh->block_size];
            int64_t slot = t % sh->block_size;
            int64_t row = first_row[r] + (t - start[r]);
            for (int64_t l = 0; l < sh->num_layers; ++l)
                for (int64_t kv = 0; kv < 2; ++kv)
                    for (int64_t h = 0; h < sh->num_kv_heads; ++h)
                        for (int64_t d = 0; d < sh->head_dim; ++d)
                            copy_elem(ckpt, ckpt_index(sh, row, l, kv, h, d),
                                      cache, cache_index(sh, l, kv, b, slot, h, d),
                                      sh->elem_bytes);
        }
    }
    free(first_row);
    return ORACLE_OK;
}

int oracle_unpack(const oracle_cache_shape *sh, void *cache,
                  const int32_t *block_tables, int32_t bt_cols,
                  const int32_t *start, const int32_t *end, int32_t num_reqs,
                  int64_t row_base, const int64_t *req_row_base,
                  const void *ckpt, int64_t ckpt_rows)
{
    int64_t *first_row = malloc(sizeof(int64_t) * (num_reqs > 0 ? num_reqs : 1));
    if (!first_row)
        return ORACLE_ERR_INVALID_ARG;
    int st = prepare(sh, cache, block_tables, bt_cols, start, end, num_reqs,
                     row_base, req_row_base, ckpt, ckpt_rows, first_row);
    if (st != ORACLE_OK) {
        free(first_row);
        return st;
    }
    for (int32_t r = 0; r < num_reqs; ++r) {
        for (int64_t t = start[r]; t < end[r]; ++t) {
            int64_t b = block_tables[(int64_t)r * bt_cols + t / sh->block_size];
            int64_t slot = t % sh->block_size;
            int64_t row = first_row[r] + (t - start[r]);
            for (int64_t l = 0; l < sh->num_layers; ++l)
                for (int64_t kv = 0; kv < 2; ++kv)
                    for (int64_t h = 0; h < sh->num_kv_heads; ++h)
                        for (int64_t d = 0; d < sh->head_dim; ++d)
                            copy_elem(cache, cache_index(sh, l, kv, b, slot, h, d),
                                      ckpt, ckpt_index(sh, row, l, kv, h, d),
                                      sh->elem_bytes);
        }
    }
    free(first_row);
    return ORACLE_OK;
}

int oracle_validate_targets(const oracle_cache_shape *sh,
                            const int32_t *block_tables, int32_t bt_cols,
                            const int32_t *start, const int32_t *end,
                            int32_t num_reqs)
{
    int status = check_shape(sh);
    if (status != ORACLE_OK)
        return status;
    if (num_reqs < 0 || bt_cols < 0)
        return ORACLE_ERR_INVALID_ARG;
    if (num_reqs > 0 && (!block_tables || !start || !end))
        return ORACLE_ERR_INVALID_ARG;
    /* times[b]: how many written pages name block b */
    int32_t *times = calloc((size_t)sh->num_blocks + 1, sizeof(int32_t));
    if (!times)
        return ORACLE_ERR_INVALID_ARG;
    for (int32_t r = 0; r < num_reqs; ++r) {
        if (start[r] < 0 || end[r] < start[r]) {
            status = worse(status, ORACLE_ERR_RANGE);
            continue;
        }
        if (end[r] == start[r])
            continue;
        int64_t first = start[r] / sh->block_size;
        int64_t last = (end[r] - 1) / sh->block_size;
        for (int64_t page = first; page <= last; ++page) {
            if (page >= bt_cols) {
                status = worse(status, ORACLE_ERR_RANGE);
                continue;
            }
            int64_t b = block_tables[(int64_t)r * bt_cols + page];
            if (b < 0 || b >= sh->num_blocks) {
                status = worse(status, ORACLE_ERR_BLOCK_ID);
                continue;
            }
            times[b] += 1;
        }
    }
    for (int64_t b = 0; b < sh->num_blocks; ++b)
        if (times[b] > 1)
            status = worse(status, ORACLE_ERR_DUP_BLOCK);
    free(times);
    return status;
}
