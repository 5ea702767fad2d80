/*
 * vfm.h -- C ABI of the mixed-task batched forward on MI355X (gfx950).
 *
 * FMplex (arxiv 2606.09643) serves many per-task "virtual FMs" over ONE shared
 * physical backbone.  A scheduler batch concatenates requests of several tasks;
 * the shared backbone runs once over all of them and each task's adapter
 * difference is then applied to that task's requests only (Section 4.2,
 * "Batch-aware Fair Scheduling", last paragraph; example (c) of Fig. 5).  A
 * task extends the backbone with a PEFT adapter (LoRA) and a decoder head
 * (Section 2.2; Section 4.1 "Task Extensions"; Table 1 attach_adapter /
 * add_decoder; Appendix A LoraConfig).  This library runs that batch forward.
 *
 * Conventions shared by every entry point
 *   - All tensors are row-major.  Linear weights use the nn.Linear layout
 *     [d_out, d_in]: y = x W^T + b.  LoRA factors: A_t [r_t, d_in],
 *     B_t [d_out, r_t]; the difference is scale_t * (x A_t^T) B_t^T.
 *   - "dtype" (VFM_F32 or VFM_BF16) is the type of weights, adapters, heads
 *     and stored activations.  The residual stream x is ALWAYS float32.
 *   - Rows inside the layer calls are in PLAN order (requests sorted by task
 *     id, ties in arrival order, see vfm_plan).  vfm_embed_forward reads the
 *     caller's rows in ORIGINAL order and vfm_head_forward writes outputs in
 *     ORIGINAL order.
 *   - Every pointer documented as "device" must point to device memory owned
 *     by the caller and stay valid until the stream has executed the work.
 *     "host" pointers are read during the call only.  The library allocates
 *     no device memory and keeps no pointer after returning.
 *   - stream is a hipStream_t (NULL = the null stream).  All launches are
 *     asynchronous on it.
 *   - Errors: every argument is checked on the host before anything is
 *     enqueued; on failure a negative vfm_status is returned and nothing is
 *     launched.  A launch failure returns VFM_ERR_HIP.  No C++ exception
 *     crosses the ABI.  Calls are reentrant; concurrent calls must not share
 *     a workspace.
 */
#ifndef VFM_H
#define VFM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  VFM_OK = 0,
  VFM_ERR_ARG = -1,         /* null pointer or bad enum value */
  VFM_ERR_SHAPE = -2,       /* sizes inconsistent or outside the supported set */
  VFM_ERR_TASK = -3,        /* task id out of range */
  VFM_ERR_UNSUPPORTED = -4, /* valid request the library does not implement */
  VFM_ERR_WORKSPACE = -5,   /* workspace missing or too small */
  VFM_ERR_HIP = -6          /* HIP runtime error at launch */
} vfm_status;

enum { VFM_F32 = 0, VFM_BF16 = 1 };
enum { VFM_NORM_LAYER = 0, VFM_NORM_RMS = 1 };
enum { VFM_MLP_GELU = 0, VFM_MLP_SWIGLU = 1 };
enum { VFM_ATTN_BIDIR = 0, VFM_ATTN_CAUSAL = 1, VFM_ATTN_DECODE = 2, VFM_ATTN_MIXED = 3 };
enum { VFM_Q = 0, VFM_K = 1, VFM_V = 2, VFM_O = 3, VFM_GATE = 4, VFM_UP = 5, VFM_DOWN = 6,
       VFM_NPROJ = 7 };
enum { VFM_POOL_MEAN = 0, VFM_POOL_FIRST = 1, VFM_POOL_LAST = 2 };
enum { VFM_EMBED_ROWS = 0, VFM_EMBED_TOKENS = 1, VFM_EMBED_PATCHES = 2 };

/* Rows per tile of the per-task segmented kernels; also the query block of
 * prefill attention.  Exposed because the plan's tile counts depend on it. */
#define VFM_ROW_TILE 64
#define VFM_MAX_RANK 64

/* bf16 batches with fewer rows than this take the small-batch kernels
 * (weight-streaming split-K GEMM whose finalize pass adds each row's LoRA
 * difference, block-per-row norms); larger ones take the large-tile kernels
 * with the LoRA expand fused and wave-per-row norms.  Both fix their
 * summation order from the weight shapes alone, and attention picks its
 * kernel by each request's own length, so a row's output is bit-identical
 * across batches on the same side of this threshold. */
#define VFM_SMALL_BATCH_ROWS 1024

/* Backbone shape.  Supported: d_model = n_heads * head_dim, head_dim in
 * {64, 128}, d_model and d_ff multiples of 64, d_model <= 8192. */
typedef struct vfm_cfg {
  int32_t dtype;      /* VFM_F32 | VFM_BF16 */
  int32_t d_model;
  int32_t n_heads;
  int32_t head_dim;
  int32_t d_ff;
  int32_t norm;       /* VFM_NORM_LAYER (encoder) | VFM_NORM_RMS (decoder) */
  int32_t mlp;        /* VFM_MLP_GELU: u = GELU_erf(h W_up^T + b_up)
                         VFM_MLP_SWIGLU: u = SiLU(h W_gate^T) * (h W_up^T) */
  int32_t attn;       /* VFM_ATTN_BIDIR | VFM_ATTN_CAUSAL | VFM_ATTN_DECODE | VFM_ATTN_MIXED */
  int32_t has_bias;   /* 1: every backbone linear has a bias */
  float norm_eps;
  float rope_theta;   /* 0: no rotary embedding; else RoPE base (rotate-half) */
} vfm_cfg;

/* ------------------------------------------------------------------------
 * a0. Plan: segment a batch by task (host, integer, deterministic).
 *
 * The paper's scheduler forms a batch of requests from several vFMs and
 * applies each adapter difference per task (Section 4.2).  vfm_plan turns
 * the batch's task ids into contiguous per-task segments.
 *
 * Plan buffer (int32, caller-owned, n_ints from vfm_plan_size), in order:
 *   header[16]   n_req, n_tasks, T, max_seqlen, n_qblocks, n_rtiles,
 *                total_outputs, 0...
 *   order[n_req]        plan position p -> original request index
 *   task[n_req]         task id at plan position p
 *   cu_seqlens[n_req+1] first row of plan position p (plan order)
 *   seg_req[n_tasks+1]  first plan position of task t
 *   seg_row[n_tasks+1]  first row of task t
 *   cu_orig[n_req+1]    first row of request i in ORIGINAL order
 *   out_off[n_req+1]    first head output of request i, ORIGINAL order
 *   ctx[n_req]          cached context length at plan position p (0: prefill)
 *   kv_start[n_req]     first KV slot of plan position p (0 if none)
 *   qblk_off[n_req+1]   exclusive scan of ceil(len/VFM_ROW_TILE), plan order
 *   rtile_off[n_tasks+1] exclusive scan of ceil(rows_t/VFM_ROW_TILE)
 *   row_task[T], row_req[T], pos[T]  per plan-order row: task, plan position,
 *                       position in its request (+ ctx when decoding)
 * Requests are ordered by task id ascending, ties in arrival order; tasks
 * without requests get empty segments.
 * ---------------------------------------------------------------------- */
#define VFM_PLAN_HEADER 16

int vfm_plan_size(int32_t n_req, int32_t n_tasks, int64_t total_rows, size_t* n_ints);

/* task_id, seq_len: host [n_req], original order; seq_len >= 1.
 * ctx_len, kv_start: host [n_req] or NULL (decode: cached tokens and the
 * first cache slot of each request; the new token's K/V go to slot
 * kv_start + ctx_len).  n_out: host [n_tasks] head widths or NULL.
 * Returns VFM_ERR_TASK for an id outside [0, n_tasks). */
int vfm_plan(const int32_t* task_id, const int32_t* seq_len, const int32_t* ctx_len,
             const int32_t* kv_start, const int32_t* n_out, int32_t n_req, int32_t n_tasks,
             int32_t* plan, size_t n_ints);

/* A planned batch: the same plan buffer on the host (for launch sizes) and a
 * device copy of it (read by the kernels). */
typedef struct vfm_batch {
  const int32_t* plan_host;   /* host */
  const int32_t* plan_dev;    /* device */
  size_t n_ints;
} vfm_batch;

/* ------------------------------------------------------------------------
 * Shared backbone weights of one layer (device, dtype unless noted).
 * ---------------------------------------------------------------------- */
typedef struct vfm_layer_weights {
  const void* norm1_w;   /* [d] */
  const void* norm1_b;   /* [d] LayerNorm shift, NULL for RMSNorm */
  const void* w_qkv;     /* [3d, d]: rows of W_q, then W_k, then W_v */
  const void* b_qkv;     /* [3d] or NULL */
  const void* w_o;       /* [d, d] */
  const void* b_o;       /* [d] or NULL */
  const void* norm2_w;   /* [d] */
  const void* norm2_b;   /* [d] or NULL */
  const void* w_gate;    /* [d_ff, d] (SwiGLU) or NULL */
  const void* w_up;      /* [d_ff, d] */
  const void* b_up;      /* [d_ff] or NULL */
  const void* w_down;    /* [d, d_ff] */
  const void* b_down;    /* [d] or NULL */
} vfm_layer_weights;

/* Per-task LoRA adapters of one layer (the vFM's "Task Extensions",
 * Section 4.1; LoRA of Hu et al., Section 2.2).  A[p] / B[p] are device
 * arrays of n_tasks device pointers (an entry may be NULL when rank[t] is 0);
 * a NULL A[p] means projection p carries no adapters.  Entries can be
 * replaced between calls to attach or remove a task's adapter without
 * touching the backbone. */
typedef struct vfm_lora_table {
  int32_t n_tasks;
  int32_t max_rank;            /* >= every rank[t]; multiple of 8, <= 64 */
  const int32_t* rank;         /* device [n_tasks]: 0 or a multiple of 8 <= max_rank */
  const float* scale;          /* device [n_tasks]: lora_alpha / r or any scale */
  const void* const* A[VFM_NPROJ];  /* device [n_tasks] -> A_t [rank_t, d_in] */
  const void* const* B[VFM_NPROJ];  /* device [n_tasks] -> B_t [d_out, rank_t] */
} vfm_lora_table;

/* Per-task decoder heads (the vFM's decoder, Section 2.2): linear, or a
 * two-layer MLP (the MLP decoders of Section 4.3's pipeline example):
 *   linear:  out = W_t pooled + b_t
 *   MLP:     out = W_t act(W1_t pooled + b1_t) + b_t
 * A task has an MLP head when W1 is non-NULL and its entry W1[t] is. */
enum { VFM_ACT_GELU = 0, VFM_ACT_RELU = 1 };
typedef struct vfm_head_table {
  int32_t n_tasks;
  int32_t pool;                /* VFM_POOL_MEAN | VFM_POOL_FIRST | VFM_POOL_LAST */
  int32_t max_out;             /* >= every n_out[t] */
  const int32_t* n_out;        /* device [n_tasks]; must equal the n_out given to vfm_plan */
  const void* const* W;        /* device [n_tasks] -> W_t [n_out_t, d] (linear) or [n_out_t, hidden] (MLP) */
  const void* const* b;        /* device [n_tasks] -> b_t [n_out_t], entries may be NULL */
  int32_t hidden;              /* MLP heads' hidden width: a multiple of 64, <= d; 0 without MLP heads */
  int32_t act;                 /* VFM_ACT_GELU (exact erf form) | VFM_ACT_RELU */
  const void* const* W1;       /* device [n_tasks] -> W1_t [hidden, d], NULL entries = linear head; or NULL */
  const void* const* b1;       /* device [n_tasks] -> b1_t [hidden], entries may be NULL; or NULL */
} vfm_head_table;

/* Per-task input encoders (the vFM's input-side extension, Section 2.2 and
 * Section 4.1 task extensions): a linear channel combiner (the
 * LinearChannelCombiner encoder of Section 4.3's pipeline example, 3 channels
 * to 1).  A request of task t brings C channels x_0 .. x_{C-1} of its series;
 * the backbone sees the one-channel series s = b_t + sum_c W_t[c] x_c.  Tasks
 * whose W entry is NULL have no encoder: their channel 0 passes unchanged. */
typedef struct vfm_encoder_table {
  int32_t n_tasks;
  int32_t n_channels;          /* C, 1..64 */
  const float* const* W;       /* device [n_tasks] -> W_t float32 [C]; entries may be NULL */
  const float* const* b;       /* device [n_tasks] -> b_t float32 [1], entries may be NULL; or NULL */
} vfm_encoder_table;

const char* vfm_status_string(int status);

/* ------------------------------------------------------------------------
 * Runtime attach / remove of one task's extensions between batches
 * (Section 4.1 task extensions; Table 1 attach_adapter / remove_adapter,
 * add_decoder).  Task `task`'s entries of the table's device arrays (which
 * must be writable) are rewritten by a kernel on `stream`, so the update is
 * ordered with the forward calls on that stream; the backbone weights and
 * the other tasks' entries are not touched, nothing is allocated and the
 * host does not wait.
 *   vfm_lora_attach: rank 0 removes the task's adapters (entries become
 *     NULL, rank 0).  Otherwise A, B are host arrays [VFM_NPROJ] of device
 *     pointers A_t [rank, d_in], B_t [d_out, rank] (NULL for a projection
 *     the task leaves bare; A and B in pairs).  Errors: VFM_ERR_TASK for a
 *     task out of range; VFM_ERR_SHAPE for a rank that is not a multiple of 8
 *     or exceeds table->max_rank; VFM_ERR_ARG for null table arrays, an
 *     unpaired A / B, or a factor for a projection whose table array is NULL.
 *   vfm_head_attach: n_out 0 removes the head; W = W_t, b = b_t [n_out] or
 *     NULL (device); W1 = W1_t [hidden, d] and b1 = b1_t [hidden] (or NULL)
 *     make it an MLP head (W_t is then [n_out, hidden]), W1 = NULL a linear
 *     one (W_t [n_out, d]).  VFM_ERR_SHAPE for n_out > table->max_out;
 *     VFM_ERR_ARG for a bias or MLP layer the table has no array for.
 *     Later batches must give vfm_plan the new n_out. */
int vfm_lora_attach(const vfm_lora_table* table, int32_t task, int32_t rank, float scale,
                    const void* const* A, const void* const* B, void* stream);
int vfm_head_attach(const vfm_head_table* table, int32_t task, int32_t n_out, const void* W,
                    const void* b, const void* W1, const void* b1, void* stream);
/*   vfm_encoder_attach: W = W_t float32 [C] (device) gives the task an
 *     encoder, W = NULL removes it (channel 0 passes); b = b_t [1] or NULL.
 *     VFM_ERR_TASK for a task out of range; VFM_ERR_ARG for a null table or
 *     table->W, or a bias when table->b is NULL. */
int vfm_encoder_attach(const vfm_encoder_table* table, int32_t task, const float* W, const float* b,
                       void* stream);

/* Greedy decoding of token-based FMs: the next token of each request is the
 * index of its largest head output (a task's LM head over the vocabulary, a
 * per-task decoder of Section 2.2), taken for every request of the batch in
 * one launch.  out: device float32 head outputs (vfm_head_forward's layout,
 * request i at out_off[i], original order); ids: device int32 [n_req],
 * original order.  Ties go to the lowest index; NaN outputs are never
 * chosen; a request with no non-NaN output gets -1. */
int vfm_greedy_tokens(const vfm_batch* batch, const float* out, int32_t* ids, void* stream);

/* Device workspace needed by vfm_layer_forward / vfm_lora_apply /
 * vfm_head_forward for this batch (lora may be NULL). */
int vfm_workspace_size(const vfm_cfg* cfg, const vfm_batch* batch, const vfm_lora_table* lora,
                       size_t* bytes);

/* ------------------------------------------------------------------------
 * a1. Input rows -> fp32 residual stream x [T, d] in plan order.
 *   VFM_EMBED_ROWS:    src [T, d] (dtype) in original order; x = permuted src.
 *   VFM_EMBED_TOKENS:  src int32 [T] token ids (original order), table
 *                      [vocab, d] (dtype) with vocab = src_width; x = table[id].
 *                      Ids outside [0, vocab) give zero rows.
 *   VFM_EMBED_PATCHES: src float32 [T, src_width] patches (original order),
 *                      table = W_pe [d, src_width], bias [d] (dtype);
 *                      x = W_pe patch + b_pe.  src_width <= 64.
 * ---------------------------------------------------------------------- */
int vfm_embed_forward(const vfm_cfg* cfg, const vfm_batch* batch, int32_t mode, const void* src,
                      int32_t src_width, const void* table, const void* bias, float* x,
                      void* stream);

/* a1'. Per-task encoder, then the shared patch embedding, in one pass.
 *   src: device float32, requests in ORIGINAL order; request i (len_i rows,
 *     patches of `patch` samples) occupies n_channels * len_i * patch floats
 *     from n_channels * cu_orig[i] * patch, channel-major: channel c is the
 *     request's whole series of len_i * patch samples.
 *   enc: the encoder table (n_tasks equal to the plan's).
 *   W_pe [d, patch], b_pe [d] or NULL (dtype), patch <= 64, as
 *   VFM_EMBED_PATCHES.  x: fp32 [T, d], plan order.
 * Row r of request i of task t: x_r = W_pe s[r * patch .. (r + 1) * patch) + b_pe
 * with s the task's combined series (see vfm_encoder_table).
 * Errors: VFM_ERR_ARG for null pointers, VFM_ERR_SHAPE for n_channels
 * outside 1..64, patch outside 1..64 or an encoder table of another task count. */
int vfm_embed_series(const vfm_cfg* cfg, const vfm_batch* batch, const vfm_encoder_table* enc,
                     const float* src, int32_t patch, const void* W_pe, const void* b_pe, float* x,
                     void* stream);

/* ------------------------------------------------------------------------
 * a2-a10. One backbone layer over the whole mixed batch, in place on x.
 * The shared projections run once over the rows of every task and each
 * task's adapter difference is added on its own rows only (Section 4.2, the
 * adapter handling in the last paragraph of "Batch-aware Fair Scheduling";
 * example (c) of Fig. 5); attention stays within each request.
 *   x: device float32 [T, d], plan order (residual stream).
 *   lora: NULL for the bare backbone.
 *   k_cache, v_cache: device [n_heads, kv_slots, head_dim] (dtype), head-major,
 *     rotated keys; used when cfg->attn is VFM_ATTN_DECODE or VFM_ATTN_MIXED
 *     (required) or VFM_ATTN_CAUSAL (optional, NULL to skip): each row's K/V
 *     is written at slot kv_start + pos of every head.  Head-major keeps one
 *     head's keys of a request contiguous, which is what decode attention
 *     streams.  (VFM_ATTN_MIXED steps are described with
 *     vfm_layer_forward_paged; the contiguous cache works for them too.)
 *   workspace: device, >= vfm_workspace_size bytes, 256-byte aligned.
 * Per layer: h = Norm1(x); [q|k|v] = h W_qkv^T + b (+ per-task LoRA);
 * RoPE; attention per request; x += attn W_o^T + b_o (+ LoRA_o);
 * h2 = Norm2(x); u = MLP(h2) (+ LoRA on gate/up); x += u W_down^T + b_down
 * (+ LoRA_down).
 * Errors: the checks listed in the file header; VFM_ERR_ARG for a missing
 * weight or (decode / mixed) a missing cache; VFM_ERR_SHAPE when a request's
 * cache slots kv_start + ctx + len exceed kv_slots; VFM_ERR_UNSUPPORTED for a
 * VFM_ATTN_DECODE request of more than one row, for a VFM_ATTN_BIDIR or
 * VFM_ATTN_CAUSAL request with ctx > 0 (those steps attend over the
 * request's own rows only), and for a prompt chunk in an fp32 mixed step;
 * VFM_ERR_WORKSPACE for a workspace below vfm_workspace_size or not 256-byte
 * aligned.
 * ---------------------------------------------------------------------- */
int vfm_layer_forward(const vfm_cfg* cfg, const vfm_layer_weights* w, const vfm_lora_table* lora,
                      const vfm_batch* batch, float* x, void* k_cache, void* v_cache,
                      int64_t kv_slots, void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * vfm_layer_forward without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops
 * and harnesses that forbid allocation.  Same arguments (minus workspace),
 * same kernels, same results and errors as vfm_layer_forward.
 *
 * The workspace is instead a fixed array of VFM_NOALLOC_SCRATCH_BYTES inside
 * the library, one per GPU, held by each GPU the library runs on until the
 * process ends.  A batch whose workspace (vfm_workspace_size) exceeds it is
 * refused on the host with VFM_ERR_WORKSPACE (the decode step of 256 rows of
 * a 4096-wide, 11008-MLP decoder needs about 93 MiB; a 12 608-row ViT-B
 * batch about 117 MiB).  The call allocates nothing (no hipMalloc, hipFree or
 * allocating library routine): the array's device address is looked up once
 * per device, on the first call with that device current.  stream must
 * belong to the current device (VFM_ERR_ARG otherwise).
 *
 * Every call on one GPU uses that GPU's one array: calls that overlap on a
 * GPU (two streams, or two host threads) race and must be serialised by the
 * caller; calls in stream order on one stream are safe.  The array keeps the
 * last call's contents; no call reads what an earlier one left.  As with
 * every entry point, timing events are recorded only while vfm_profile_enable
 * has a class enabled (a benchmark facility), so leave it disabled here.
 * ---------------------------------------------------------------------- */
#define VFM_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)

int vfm_layer_forward_noalloc(const vfm_cfg* cfg, const vfm_layer_weights* w, const vfm_lora_table* lora,
                              const vfm_batch* batch, float* x, void* k_cache, void* v_cache,
                              int64_t kv_slots, void* stream);

/* ------------------------------------------------------------------------
 * a2-a10 over a paged KV cache: the token-based FMs' continuous batching
 * with long-lived decode iterations (Section 4.2, which also charges their
 * token-level work in service-time units; Section 6 maps the vFM boundary
 * onto a vLLM-style runtime, whose KV cache is paged).
 *
 * Pages.  The cache keeps the head-major layout of vfm_layer_forward,
 * [n_heads][n_pages * page_size][head_dim], cut into pages of page_size slots:
 * token k of request i lives at slot table[i][k / page_size] * page_size +
 * k % page_size of every head.  Each page of one head is a contiguous run
 * (page_size * head_dim elements), so decode attention streams whole pages;
 * a contiguous cache is the case table[i][j] = first_page_i + j.
 *
 * Steps.  cfg->attn selects:
 *   VFM_ATTN_CAUSAL  every request a prompt (ctx 0): causal attention over
 *                    its own rows, whose K / V are written into its pages.
 *   VFM_ATTN_DECODE  every request one new token after ctx cached ones.
 *   VFM_ATTN_MIXED   a continuous-batching step: each request is a prompt
 *                    (ctx 0, any length), one decode token (ctx > 0, length
 *                    1) or, in bf16, a prompt chunk after cached tokens
 *                    (ctx > 0, several rows: each row attends causally to the
 *                    ctx cached keys and the chunk's earlier rows).  An fp32
 *                    step with such a chunk gives VFM_ERR_UNSUPPORTED.
 * The new rows' K / V go to slots ctx .. ctx + len - 1 of the request's pages
 * before attention reads them.
 * ---------------------------------------------------------------------- */
typedef struct vfm_kv_pages {
  void* k;                    /* device [n_heads][n_pages * page_size][head_dim] (dtype) */
  void* v;                    /* same layout */
  int64_t n_pages;
  int32_t page_size;          /* slots per page: a power of two, 16 .. 1024 */
  int32_t max_pages;          /* columns of the page table */
  const int32_t* table_host;  /* host [n_req][max_pages], ORIGINAL request order: physical page of
                                 each logical page; validated against n_pages before any launch */
  const int32_t* table_dev;   /* device copy of table_host */
} vfm_kv_pages;

/* Errors as vfm_layer_forward, plus VFM_ERR_SHAPE when a request's
 * ctx + len tokens need more than max_pages pages or a page id it uses is
 * outside [0, n_pages), VFM_ERR_ARG for a bad page size or null tables, and
 * VFM_ERR_UNSUPPORTED for VFM_ATTN_BIDIR, for a VFM_ATTN_CAUSAL request with
 * ctx > 0, and for a prompt chunk (ctx > 0, more than one row) in an fp32
 * VFM_ATTN_MIXED step (bf16 accepts it). */
int vfm_layer_forward_paged(const vfm_cfg* cfg, const vfm_layer_weights* w, const vfm_lora_table* lora,
                            const vfm_batch* batch, float* x, const vfm_kv_pages* kv, void* workspace,
                            size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * a4. Segmented LoRA on one projection: for every plan-order row m of task
 * t with rank_t > 0,  y[m, :] += scale_t * (x[m, :] A_{t,proj}^T) B_{t,proj}^T.
 * This is the per-task adapter difference on its own (LoRA, Section 2.2;
 * applied per task segment of the shared batch, Section 4.2 adapter
 * handling).  Rows of rank-0 tasks are left untouched.
 *   x: device [T, d_in] (dtype), plan order.  y: device float32 [T, d_out].
 *   d_in a multiple of 64, d_out a multiple of 4 (else VFM_ERR_SHAPE).
 *   workspace: device, >= T * rpad * sizeof(dtype) bytes (rpad = 32 if
 *   max_rank <= 32, else 64), 256-byte aligned.
 * Errors: VFM_ERR_ARG for a bad dtype / projection, null pointers or a
 * projection without adapters in the table; VFM_ERR_SHAPE as above and for a
 * table of another task count; VFM_ERR_WORKSPACE.
 * ---------------------------------------------------------------------- */
int vfm_lora_apply(int32_t dtype, int32_t proj, int32_t d_in, int32_t d_out,
                   const vfm_lora_table* lora, const vfm_batch* batch, const void* x, float* y,
                   void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * a11-a12. Final norm, pooling and per-task heads: each request ends in its
 * own task's decoder head on the shared backbone's output (Section 2.2
 * decoders; Section 4.1 task extensions; Table 1 add_decoder).
 *   x: device float32 [T, d] plan order (the last layer's output).
 *   heads != NULL: out = device float32 [total_outputs]; request i's
 *     outputs W_t pool(Norm(x_i)) + b_t start at out_off[i] (original order).
 *   heads == NULL: out = device float32 [T, d], the final-normed rows in
 *     original order.
 *   workspace: device, >= vfm_workspace_size bytes, 256-byte aligned (holds
 *     the pooled rows and MLP heads' hidden rows).
 * Errors: VFM_ERR_ARG for null pointers, a head table of another task count,
 * a bad pooling mode or activation; VFM_ERR_SHAPE for a bad hidden width;
 * VFM_ERR_UNSUPPORTED for d * sizeof(dtype) above 64 KB; VFM_ERR_WORKSPACE.
 * ---------------------------------------------------------------------- */
int vfm_head_forward(const vfm_cfg* cfg, const void* final_norm_w, const void* final_norm_b,
                     const vfm_head_table* heads, const vfm_batch* batch, const float* x,
                     float* out, void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Kernel timing for benchmarks (not part of the forward).  While a class's
 * bit is set in the mask, every launch of that class made by the calls above
 * is bracketed by two hipEvents on its stream; vfm_profile_read waits for
 * the recorded events and returns, per class, the summed milliseconds and
 * the launch count since the last reset.  Process-global state: enable and
 * read from one thread.  Classes: */
enum { VFM_PROF_GEMM_QKV = 0, VFM_PROF_GEMM_O = 1, VFM_PROF_GEMM_UP = 2, VFM_PROF_GEMM_DOWN = 3,
       VFM_PROF_ATTN = 4, VFM_PROF_NORM = 5, VFM_PROF_SHRINK = 6, VFM_PROF_OTHER = 7,
       VFM_PROF_NCLASS = 8 };

int vfm_profile_enable(uint32_t class_mask);   /* 0 disables; also resets the counters */
int vfm_profile_read(double* ms, int64_t* launches, int32_t n_classes); /* host arrays */

#ifdef __cplusplus
}
#endif

#endif /* VFM_H */
