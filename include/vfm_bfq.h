/* Batch-aware fair queueing (BFQ): forms the mixed-task batches that
 * vfm_plan / vfm_layer_forward run (paper Section 4.2, "Batch-aware Fair
 * Scheduling", Eq. 1-3 and the service-time correction after a batch).
 *
 * Host only, no device memory.  The scheduler state lives in a caller-owned
 * host buffer (vfm_bfq_state_size bytes, 8-byte aligned); the library keeps
 * no pointers and allocates nothing.  Calls on one state must not overlap;
 * distinct states are independent.  Status codes are the vfm_status values
 * of vfm.h; on any error nothing in the state changes.
 *
 * Tags.  Task i has weight w_i > 0.  A request gets, when enqueued, the start
 * tag S = max(F of the task's previous request, v) and the finish tag
 * F = S + T(1) / w_i, where v is the largest finish tag among the tasks'
 * most recently dispatched requests (0 before the first dispatch).
 *
 * Batches.  vfm_bfq_next_batch takes the queued requests in increasing start
 * tag (ties: lower task id, then earlier request of the task) and admits
 * them one at a time while the batch holds fewer than b_max requests and
 * now + T(b) (b = the batch size with the new request) is at most every
 * admitted request's deadline; the first request is always admitted, and
 * the scan stops at the first request that cannot be.  Afterwards every task
 * with requests in the batch has its tags recomputed with the per-request
 * service time l(b) = T(b) / b: its dispatched requests, then its queued
 * ones, each S = max(F of the task's previous request, v at its arrival),
 * F = S + l(b) / w_i.
 */
#ifndef VFM_BFQ_H
#define VFM_BFQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t n_tasks;           /* tasks (vFMs) sharing the backbone, >= 1 */
  int32_t b_max;             /* largest batch, >= 1 */
  int32_t max_queued;        /* queue capacity per task, >= 1 */
  const double* weight;      /* host [n_tasks], each > 0 (copied by vfm_bfq_init) */
  const double* batch_time;  /* host [b_max + 1]: T(b), the estimated service time of a batch of
                                b requests; T(0) is ignored; T(b) > 0 (copied by vfm_bfq_init) */
} vfm_bfq_config;

/* Bytes of state for this configuration.  VFM_ERR_ARG for null pointers,
 * VFM_ERR_SHAPE for sizes out of range. */
int vfm_bfq_state_size(const vfm_bfq_config* cfg, size_t* bytes);

/* Initialises the state (empty queues, all tags 0).  VFM_ERR_ARG for null
 * pointers or a buffer not 8-byte aligned, VFM_ERR_SHAPE for bytes below
 * vfm_bfq_state_size or a weight / batch time that is not > 0 (or not
 * finite). */
int vfm_bfq_init(const vfm_bfq_config* cfg, void* state, size_t bytes);

/* Queues request `request` of task `task`, arrived at `arrival`, due by
 * `deadline` (same time unit as T; +inf for none).  VFM_ERR_TASK for a task
 * out of range, VFM_ERR_SHAPE when the task's queue is full. */
int vfm_bfq_enqueue(void* state, int32_t task, int64_t request, double arrival, double deadline);

/* Forms the next batch at time `now` and removes it from the queues:
 * requests[k], tasks[k] for k < *n, in admission order (host arrays of
 * `capacity` entries; capacity >= b_max).  *n = 0 when nothing is queued.
 * VFM_ERR_SHAPE if capacity < b_max. */
int vfm_bfq_next_batch(void* state, double now, int64_t* requests, int32_t* tasks, int32_t capacity,
                       int32_t* n);

/* Token-based FMs (Section 4.2: token-level work charged in service-time
 * units): adds `service` (>= 0, the unit of T) of realised work to task
 * `task`, e.g. the decode tokens its running sequences produced in one
 * iteration times the per-token time.  The task's last dispatched request's
 * finish tag moves by service / w_task (a task with nothing dispatched yet
 * starts from 0), its queued requests' tags follow (each S = max(F of the
 * previous one, v at its arrival), F = S + its own service / w), and v is
 * recomputed.  VFM_ERR_TASK for a task out of range, VFM_ERR_SHAPE for a
 * negative or non-finite service. */
int vfm_bfq_charge(void* state, int32_t task, double service);

/* Requests of task `task` waiting in the state. */
int vfm_bfq_queued(const void* state, int32_t task, int32_t* n);

/* Start and finish tags of the k-th queued request of task `task` (k = 0 is
 * the next one to be dispatched), for inspection and tests.  VFM_ERR_SHAPE
 * if k is not below the task's queue length. */
int vfm_bfq_tags(const void* state, int32_t task, int32_t k, double* start, double* finish);

#ifdef __cplusplus
}
#endif

#endif /* VFM_BFQ_H */
