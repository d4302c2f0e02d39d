/*
 * Page tags and the longest checkpointed prefix (host side of LUMEN's
 * KV-reuse recovery).
 *
 *   Sec. 4.2, page tags: every transferred page carries a tag, a hash of
 *   the token IDs stored in the page paired with the page's end position
 *   (the request's token count after the page).  A tag derives from the
 *   token sequence alone, so any worker can regenerate it from the token
 *   history the gateway keeps.  Pages become visible in the checkpoint store
 *   only once completely received.
 *   Sec. 4.3, KV-reuse recovery: the holder regenerates the tags from the
 *   token history and finds the longest contiguous checkpointed prefix; the
 *   rest is recomputed by a partial prefill.
 *
 * Readings, where the paper names no function and says nothing of partial
 * pages:
 *   - hash: BLAKE2b with an 8-byte digest (RFC 7693, no key) over the page's
 *     token IDs as little-endian int32, taken as a little-endian uint64;
 *   - page i holds tokens [i*block_size, (i+1)*block_size) and only complete
 *     pages are tagged, so a reusable prefix is a whole number of pages.
 *
 * Host code only (no GPU needed); every function is thread-safe.  Status
 * codes are those of lumen_kv_ckpt.h.
 */
#ifndef LUMEN_PAGE_TAGS_H
#define LUMEN_PAGE_TAGS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lumen_page_tag {
    uint64_t hash; /* BLAKE2b-64 of the page's token IDs */
    int64_t end;   /* token count after the page: (page + 1) * block_size */
} lumen_page_tag;

/* Tags of the complete pages [page_begin, page_end) of a token history
 * tokens[0, num_tokens) (host memory), written to tags[0, page_end -
 * page_begin).  INVALID_ARG for block_size < 1, a negative count, or a page
 * range that is not within the complete pages (page_end * block_size >
 * num_tokens). */
int lumen_page_tags(const int32_t *tokens, int64_t num_tokens,
                    int32_t block_size, int64_t page_begin, int64_t page_end,
                    lumen_page_tag *tags);

/* A holder's checkpoint store as recovery reads it: per request, the tag of
 * every page that has been received completely.  Created empty; owned by
 * the caller; destroy releases everything.  NULL on bad block_size or out
 * of memory. */
typedef struct lumen_tag_store lumen_tag_store;
lumen_tag_store *lumen_tag_store_create(int32_t block_size);
void lumen_tag_store_destroy(lumen_tag_store *store);

/* Makes page `page` of `request` visible with `tag`.  Call it only once the
 * page's payload has been received completely: that is what makes pages
 * atomic (a transfer cut short leaves its page invisible).  Pages may be
 * published in any order; publishing a page again replaces its tag.
 * INVALID_ARG for a null store, page < 0, page > INT32_MAX, or tag.end !=
 * (page + 1) * block_size.  CAPACITY if host memory for the page cannot be
 * allocated; the store is then unchanged. */
int lumen_tag_store_publish(lumen_tag_store *store, int64_t request,
                            int64_t page, lumen_page_tag tag);

/* Computes the tags of pages [page_begin, page_end) from the token history
 * and publishes them (the receiver's call once those pages have arrived).
 * Same argument rules as lumen_page_tags, and pages past INT32_MAX are
 * INVALID_ARG; CAPACITY as for lumen_tag_store_publish (the pages before
 * the failing one stay published). */
int lumen_tag_store_publish_pages(lumen_tag_store *store, int64_t request,
                                  const int32_t *tokens, int64_t num_tokens,
                                  int64_t page_begin, int64_t page_end);

/* Drops every page of `request` (its checkpoint is released when the
 * request terminates).  OK also if the request has no pages. */
int lumen_tag_store_release(lumen_tag_store *store, int64_t request);

/* Longest contiguous checkpointed prefix of `request` for the token history
 * tokens[0, num_tokens): regenerates the tags of pages 0, 1, ... and counts
 * the leading pages that are visible with an equal tag.  Returns that count
 * times block_size (tokens to restore; the rest is recomputed), or a
 * negative status (INVALID_ARG). */
int64_t lumen_tag_store_longest_prefix(lumen_tag_store *store,
                                       int64_t request, const int32_t *tokens,
                                       int64_t num_tokens);

/* Pages currently visible for `request` (any order), or a negative status. */
int64_t lumen_tag_store_pages(lumen_tag_store *store, int64_t request);

#ifdef __cplusplus
}
#endif
#endif
