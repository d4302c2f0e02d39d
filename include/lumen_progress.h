/*
 * Checkpoint progress of a serving worker: which tokens of each request
 * still have to be sent (the ranges the row plan takes).
 *
 *   Sec. 4.2, incremental checkpoint pipeline: workers track checkpoint
 *   progress and, after each prefill or decode batch, send only the KV that
 *   is new since the last checkpoint.
 *
 * Per request the tracker keeps `sent`, the number of leading tokens
 * already handed to the checkpoint pipeline.  For a batch it returns the
 * ranges [sent, length) and advances `sent` to length.  A history that got
 * shorter (rejected speculative tokens rewrite the tail) lowers `sent` to
 * the new length, so the rewritten tokens are sent again with the next
 * batch; the holder's page tags tell stale pages apart at recovery.
 *
 * Host code only; one tracker is not thread-safe (callers serialise).
 * Status codes are those of lumen_kv_ckpt.h.
 */
#ifndef LUMEN_PROGRESS_H
#define LUMEN_PROGRESS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lumen_progress lumen_progress;

lumen_progress *lumen_progress_create(void);
void lumen_progress_destroy(lumen_progress *p);

/* For the n requests ids[i] whose KV now covers lengths[i] tokens, writes
 * start[i] = tokens already sent (0 for a request not seen before, at most
 * lengths[i]) and end[i] = lengths[i], then records end[i] as sent.  The
 * arrays are host memory, ready to be copied to the device for
 * lumen_kv_ckpt_plan.  INVALID_ARG for n < 0, a negative length, null
 * arrays with n > 0, or an id repeated in the batch; CAPACITY if host
 * memory for new requests cannot be allocated.  Nothing changes on either
 * error. */
int lumen_progress_ranges(lumen_progress *p, const int64_t *ids,
                          const int32_t *lengths, int32_t n, int32_t *start,
                          int32_t *end);

/* Tokens of `request` sent so far (0 if unknown), or INVALID_ARG. */
int64_t lumen_progress_sent(lumen_progress *p, int64_t request);

/* The request finished: forget it.  OK also for an unknown request. */
int lumen_progress_release(lumen_progress *p, int64_t request);

#ifdef __cplusplus
}
#endif
#endif
