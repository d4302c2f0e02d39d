/*
 * Checkpoint placement and recovery scheduling (the host-side driver of
 * LUMEN's load-aware checkpointing and locality-aware recovery).
 *
 *   Placement (Sec. 4.2, checkpoint placement, Eq. 1): every active
 *   request r gets one checkpoint holder,
 *       h(r) = argmin over w in F(r) of  q_w + lambda * p_w(r),
 *   where F(r) holds the workers whose free checkpoint budget can take r's
 *   reserved footprint (sized from the maximum context length), minus the
 *   worker serving r; q_w is w's queueing delay; p_w(r) is the mean
 *   reserved footprint of the checkpoints w would hold with r added,
 *   divided by a fixed host-to-GPU bandwidth.  The footprint is reserved on
 *   assignment and released when the request completes.
 *   Recovery (Sec. 4.3): interrupted requests go to their holders for KV
 *   reuse, or are recomputed on the least-loaded survivor when the holder
 *   failed too; then the average-based request-count rule sheds requests
 *   from the most congested worker to the least-loaded one, smallest
 *   checkpointed size first, recomputing loads after every move.  Several
 *   failures form one recovery event.
 *
 * Readings where the paper is silent: ties go to the lowest worker index;
 * F(r) empty leaves r without a checkpoint; a request moves only if the
 * target's load plus one stays below the source's (otherwise integer loads
 * can cycle); the movable requests of a worker are its newly assigned
 * interrupted requests, a recomputed one counting as checkpointed size 0;
 * interrupted requests are dispatched in increasing request id; once
 * recovered, a request's old checkpoint is released and the caller places
 * a new one; with no survivor at all a request is reported with worker -1
 * and stays interrupted, so the next recovery event reports it again.
 *
 * Host code only; one scheduler is not thread-safe (callers serialise).
 * Status codes are those of lumen_kv_ckpt.h.
 */
#ifndef LUMEN_SCHED_H
#define LUMEN_SCHED_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lumen_sched lumen_sched;

/* num_workers workers, worker w with a checkpoint budget of
 * budget_bytes[w] host bytes; h2d_bytes_per_s > 0 prices restore pressure;
 * lambda >= 0 weighs it against queueing delay.  NULL on bad arguments. */
lumen_sched *lumen_sched_create(int32_t num_workers,
                                const int64_t *budget_bytes,
                                double h2d_bytes_per_s, double lambda);
void lumen_sched_destroy(lumen_sched *s);

/* Observed state of a worker: queueing delay (seconds) and its queued and
 * running request counts. */
int lumen_sched_set_worker(lumen_sched *s, int32_t worker,
                           double queueing_delay, int64_t queued,
                           int64_t running);

/* Eq. 1 for a new request served by `serving`: *holder receives the chosen
 * worker (the footprint is reserved there), or -1 if no worker can take
 * it.  Returns OK, INVALID_ARG (unknown worker, a request already
 * placed, a negative footprint, null holder), or CAPACITY if host memory
 * for the request cannot be allocated (nothing changes then). */
int lumen_sched_place(lumen_sched *s, int64_t request, int32_t serving,
                      int64_t reserved_bytes, int32_t *holder);

/* Bytes of r's checkpoint received by its holder so far. */
int lumen_sched_set_persisted(lumen_sched *s, int64_t request,
                              int64_t bytes);

/* r completed: its reservation is released and it is forgotten. */
int lumen_sched_release(lumen_sched *s, int64_t request);

/* *holder receives r's current holder (-1: none).  INVALID_ARG for an
 * unknown request. */
int lumen_sched_holder(lumen_sched *s, int64_t request, int32_t *holder);

/* Reserved bytes on a worker, or INVALID_ARG. */
int64_t lumen_sched_reserved(lumen_sched *s, int32_t worker);

/* Recovery event for the workers failed[0, num_failed).  For each
 * interrupted request, in increasing id, writes its id, the worker that
 * resumes it and whether it reuses its checkpoint (1) or is recomputed
 * (0); *num_out receives the count.  Returns INVALID_ARG if max_out is too
 * small or a worker index is bad, CAPACITY if host memory for the
 * decision cannot be allocated; nothing changes on either error. */
int lumen_sched_recover(lumen_sched *s, const int32_t *failed,
                        int32_t num_failed, int64_t *out_request,
                        int32_t *out_worker, int8_t *out_reuse,
                        int64_t max_out, int64_t *num_out);

#ifdef __cplusplus
}
#endif
#endif
