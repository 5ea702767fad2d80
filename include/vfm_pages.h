/* KV page allocator for continuous batching of token-based FMs (paper
 * Section 4.2: LLMs served with continuous batching and long-lived decode
 * iterations; Section 6: a vLLM-style runtime, whose KV cache is paged).
 *
 * Host only.  Hands out the page ids of one KV pool (vfm_kv_pages in vfm.h)
 * to sequences: a sequence grows page by page as its tokens do, and returns
 * all its pages when it finishes, so requests of any length share one pool
 * without fragmentation.  The state lives in a caller-owned host buffer
 * (vfm_pages_state_size bytes, 8-byte aligned); nothing is allocated and no
 * pointer is kept.  Calls on one state must not overlap.  Status codes are
 * the vfm_status values of vfm.h; on any error the state is unchanged.
 *
 * Order.  Free pages form a stack; a fresh pool hands out 0, 1, 2, ... and
 * a released sequence's pages are handed out again before older free ones
 * (most recently released first), which keeps the working set of the pool
 * small.
 */
#ifndef VFM_PAGES_H
#define VFM_PAGES_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t n_pages;     /* pages in the pool, >= 1 */
  int32_t page_size;   /* tokens per page, >= 1 */
  int32_t max_seqs;    /* sequence slots 0 .. max_seqs - 1 */
  int32_t max_pages;   /* pages one sequence may hold */
} vfm_pages_config;

/* Bytes of state.  VFM_ERR_ARG for null pointers, VFM_ERR_SHAPE for sizes
 * out of range (each field >= 1, at most 2^30 pages, 2^24 sequences). */
int vfm_pages_state_size(const vfm_pages_config* cfg, size_t* bytes);

/* Every page free, every sequence empty.  VFM_ERR_SHAPE if bytes is below
 * vfm_pages_state_size. */
int vfm_pages_init(const vfm_pages_config* cfg, void* state, size_t bytes);

/* Grows sequence `seq` to hold n_tokens tokens: ceil(n_tokens / page_size)
 * pages (a no-op if it holds that many).  VFM_ERR_TASK for a slot out of
 * range; VFM_ERR_SHAPE if that exceeds max_pages or the free pages. */
int vfm_pages_reserve(void* state, int32_t seq, int64_t n_tokens);

/* Returns all pages of `seq` to the pool (the sequence becomes empty). */
int vfm_pages_release(void* state, int32_t seq);

/* Page-table rows for a batch: row r (max_cols entries) of `table` gets the
 * pages of sequence seqs[r] in token order, then -1.  VFM_ERR_TASK for a
 * sequence slot out of range, VFM_ERR_SHAPE if a sequence holds more than
 * max_cols pages (nothing is written then). */
int vfm_pages_table(const void* state, const int32_t* seqs, int32_t n, int32_t* table, int32_t max_cols);

/* Pages held by `seq` (*held) and free in the pool (*free_pages). */
int vfm_pages_count(const void* state, int32_t seq, int32_t* held, int32_t* free_pages);

#ifdef __cplusplus
}
#endif

#endif /* VFM_PAGES_H */
