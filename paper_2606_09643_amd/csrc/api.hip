// C ABI entry points: argument validation, workspace carving and the launch
// sequence of one backbone layer over a mixed-task batch.
#include <algorithm>
#include <initializer_list>
#include <mutex>

#include "vfm_internal.h"

namespace {

constexpr size_t ALIGN = 256;
inline size_t align_up(size_t v) { return (v + ALIGN - 1) / ALIGN * ALIGN; }

inline size_t elem_size(int dtype) { return dtype == VFM_BF16 ? 2 : 4; }

int check_cfg(const vfm_cfg* c) {
  if (!c) return VFM_ERR_ARG;
  if (c->dtype != VFM_F32 && c->dtype != VFM_BF16) return VFM_ERR_ARG;
  if (c->norm != VFM_NORM_LAYER && c->norm != VFM_NORM_RMS) return VFM_ERR_ARG;
  if (c->mlp != VFM_MLP_GELU && c->mlp != VFM_MLP_SWIGLU) return VFM_ERR_ARG;
  if (c->attn < VFM_ATTN_BIDIR || c->attn > VFM_ATTN_MIXED) return VFM_ERR_ARG;
  if (c->head_dim != 64 && c->head_dim != 128) return VFM_ERR_UNSUPPORTED;
  if (c->n_heads < 1 || (int64_t)c->n_heads * c->head_dim != c->d_model) return VFM_ERR_SHAPE;
  if (c->d_model % 64 || c->d_model > 8192 || c->d_ff < 64 || c->d_ff % 64) return VFM_ERR_SHAPE;
  if (c->mlp == VFM_MLP_SWIGLU && c->has_bias) return VFM_ERR_UNSUPPORTED;
  if (!(c->norm_eps >= 0.f) || !(c->rope_theta >= 0.f)) return VFM_ERR_ARG;
  return VFM_OK;
}

int check_batch(const vfm_batch* b, Plan* out) {
  if (!b || !b->plan_host || !b->plan_dev) return VFM_ERR_ARG;
  if (b->n_ints < VFM_PLAN_HEADER) return VFM_ERR_SHAPE;
  const int32_t* h = b->plan_host;
  if (h[0] < 1 || h[1] < 1 || h[2] < h[0]) return VFM_ERR_SHAPE;
  if ((size_t)plan_offsets(h[0], h[1], h[2]).total > b->n_ints) return VFM_ERR_SHAPE;
  *out = make_plan(h, b->plan_dev);
  return VFM_OK;
}

// host-side view of the plan arrays (for validation of cache bounds)
inline const int32_t* host_arr(const vfm_batch* b, int64_t off) { return b->plan_host + off; }

int check_lora(const vfm_lora_table* l, const Plan& pl) {
  if (!l) return VFM_OK;
  if (l->n_tasks != pl.n_tasks) return VFM_ERR_SHAPE;
  if (l->max_rank < 0 || l->max_rank > VFM_MAX_RANK || l->max_rank % 8) return VFM_ERR_SHAPE;
  if (!l->rank || !l->scale) return VFM_ERR_ARG;
  for (int p = 0; p < VFM_NPROJ; ++p)
    if ((l->A[p] == nullptr) != (l->B[p] == nullptr)) return VFM_ERR_ARG;
  return VFM_OK;
}

inline int rpad_of(const vfm_lora_table* l) {
  if (!l || l->max_rank == 0) return 0;
  return l->max_rank <= 32 ? 32 : 64;
}

// Small bf16 batches take the split-K GEMM + separate shrink + finalize path.
inline bool use_skinny(const vfm_cfg& c, const Plan& pl) {
  return c.dtype == VFM_BF16 && pl.T < VFM_SMALL_BATCH_ROWS;
}

// Largest number of keys one request attends to (ctx + its rows), from the
// host copy of the plan.
int max_keys_of(const vfm_batch* b, const Plan& pl) {
  const PlanOffsets po = plan_offsets(pl.n_req, pl.n_tasks, pl.T);
  const int32_t* ctx = b->plan_host + po.ctx;
  const int32_t* cu = b->plan_host + po.cu_seqlens;
  int mk = 0;
  for (int p = 0; p < pl.n_req; ++p) mk = std::max(mk, ctx[p] + cu[p + 1] - cu[p]);
  return mk;
}

struct LayerWs {
  size_t h, big, attn, u, z, p, aws, total;
  int kchunks;
};

LayerWs layer_ws(const vfm_cfg& c, const Plan& pl, const vfm_lora_table* l, int max_keys) {
  const size_t es = elem_size(c.dtype);
  const size_t T = (size_t)pl.T;
  const int d = c.d_model, f = c.d_ff, rpad = rpad_of(l);
  LayerWs w;
  size_t off = 0;
  w.h = off;    off += align_up(T * d * es);
  w.big = off;  off += align_up(T * std::max<size_t>(3 * (size_t)d, f) * es);
  w.attn = off; off += align_up(T * d * es);
  w.u = off;    off += align_up(T * 8 * rpad * es);
  w.aws = off; off += align_up(attention_workspace(c, pl, max_keys));
  w.z = w.p = off;
  w.kchunks = 0;
  if (use_skinny(c, pl)) {
    // fp32 split partials of the largest projection group
    auto zbytes = [&](int N, int K) { return (size_t)skinny_splits(N, K) * T * N * 4; };
    const int n_up = c.mlp == VFM_MLP_SWIGLU ? 2 * f : f;
    const size_t zmax = std::max(std::max(zbytes(3 * d, d), zbytes(d, d)),
                                 std::max(zbytes(n_up, d), zbytes(d, f)));
    w.z = off; off += align_up(zmax);
    if (rpad > 0) {
      w.kchunks = std::max(shrink_chunks(d), shrink_chunks(f));
      w.p = off; off += align_up((size_t)w.kchunks * T * 8 * rpad * 4);
    }
  }
  w.total = off;
  return w;
}

// pooled rows, then room for the MLP heads' hidden rows (hidden <= d)
size_t head_ws(const vfm_cfg& c, const Plan& pl) {
  return 2 * align_up((size_t)pl.n_req * c.d_model * elem_size(c.dtype));
}

inline int hip_status(hipError_t e) { return e == hipSuccess ? VFM_OK : VFM_ERR_HIP; }

#define VFM_TRY(expr)              \
  do {                             \
    int _st = (expr);              \
    if (_st != VFM_OK) return _st; \
  } while (0)
#define VFM_HIP(expr)                               \
  do {                                              \
    hipError_t _e = (expr);                         \
    if (_e != hipSuccess) return VFM_ERR_HIP;       \
  } while (0)
// a launch bracketed by the optional timing hooks
#define VFM_TIMED(cls, expr)                        \
  do {                                              \
    const int _pi = prof_begin((cls), s);           \
    hipError_t _e = (expr);                         \
    prof_end(_pi, s);                               \
    if (_e != hipSuccess) return VFM_ERR_HIP;       \
  } while (0)

}  // namespace

extern "C" const char* vfm_status_string(int status) {
  switch (status) {
    case VFM_OK: return "ok";
    case VFM_ERR_ARG: return "invalid argument (null pointer or bad enum)";
    case VFM_ERR_SHAPE: return "inconsistent or unsupported sizes";
    case VFM_ERR_TASK: return "task id out of range";
    case VFM_ERR_UNSUPPORTED: return "configuration not supported by the library";
    case VFM_ERR_WORKSPACE: return "workspace missing or too small";
    case VFM_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

extern "C" int vfm_workspace_size(const vfm_cfg* cfg, const vfm_batch* batch,
                                  const vfm_lora_table* lora, size_t* bytes) {
  if (!bytes) return VFM_ERR_ARG;
  VFM_TRY(check_cfg(cfg));
  Plan pl;
  VFM_TRY(check_batch(batch, &pl));
  VFM_TRY(check_lora(lora, pl));
  size_t need = layer_ws(*cfg, pl, lora, max_keys_of(batch, pl)).total;
  need = std::max(need, head_ws(*cfg, pl));
  *bytes = need;
  return VFM_OK;
}

extern "C" int vfm_embed_forward(const vfm_cfg* cfg, const vfm_batch* batch, int32_t mode,
                                 const void* src, int32_t src_width, const void* table,
                                 const void* bias, float* x, void* stream) {
  VFM_TRY(check_cfg(cfg));
  Plan pl;
  VFM_TRY(check_batch(batch, &pl));
  if (!src || !x) return VFM_ERR_ARG;
  if (mode == VFM_EMBED_TOKENS) {
    if (!table) return VFM_ERR_ARG;
    if (src_width < 1) return VFM_ERR_SHAPE;
  } else if (mode == VFM_EMBED_PATCHES) {
    if (!table) return VFM_ERR_ARG;
    if (src_width < 1 || src_width > 64) return VFM_ERR_SHAPE;
  } else if (mode != VFM_EMBED_ROWS) {
    return VFM_ERR_ARG;
  }
  return hip_status(launch_embed(cfg->dtype, pl, mode, src, src_width, table, bias, cfg->d_model, x,
                                 (hipStream_t)stream));
}

namespace {

// Checks shared by the two layer entry points (everything but the cache).
int check_layer(const vfm_cfg* cfg, const vfm_layer_weights* w, const vfm_lora_table* lora,
                const vfm_batch* batch, const float* x, bool have_cache, Plan* pl) {
  VFM_TRY(check_cfg(cfg));
  VFM_TRY(check_batch(batch, pl));
  VFM_TRY(check_lora(lora, *pl));
  if (!w || !x) return VFM_ERR_ARG;
  if (!w->norm1_w || !w->norm2_w || !w->w_qkv || !w->w_o || !w->w_up || !w->w_down)
    return VFM_ERR_ARG;
  if (cfg->mlp == VFM_MLP_SWIGLU && !w->w_gate) return VFM_ERR_ARG;
  if (cfg->attn == VFM_ATTN_DECODE || cfg->attn == VFM_ATTN_MIXED) {
    if (!have_cache) return VFM_ERR_ARG;
  }
  if (cfg->attn == VFM_ATTN_DECODE && pl->max_seqlen != 1) return VFM_ERR_UNSUPPORTED;
  const PlanOffsets po = plan_offsets(pl->n_req, pl->n_tasks, pl->T);
  if (cfg->attn == VFM_ATTN_BIDIR || cfg->attn == VFM_ATTN_CAUSAL) {
    // these steps attend over a request's own rows only: cached tokens
    // before them would be ignored, so a request with ctx > 0 is refused
    const int32_t* ctx = host_arr(batch, po.ctx);
    for (int p = 0; p < pl->n_req; ++p)
      if (ctx[p] > 0) return VFM_ERR_UNSUPPORTED;
  }
  if (cfg->attn == VFM_ATTN_MIXED && cfg->dtype != VFM_BF16) {   // prompt chunks after cached tokens: bf16
    const int32_t* ctx = host_arr(batch, po.ctx);
    const int32_t* cu = host_arr(batch, po.cu_seqlens);
    for (int p = 0; p < pl->n_req; ++p)
      if (ctx[p] > 0 && cu[p + 1] - cu[p] != 1) return VFM_ERR_UNSUPPORTED;
  }
  return VFM_OK;
}

int layer_impl(const vfm_cfg& c, const vfm_layer_weights* w, const vfm_lora_table* lora,
               const vfm_batch* batch, const Plan& pl, float* x, void* k_cache, void* v_cache,
               int64_t kv_slots, const KvPages& kp, void* workspace, size_t ws_bytes, void* stream);

}  // namespace

namespace {

// Checks of the contiguous-cache layer call: check_layer plus the cache's
// bounds (host copy of the plan).
int check_layer_contiguous(const vfm_cfg* cfg, const vfm_layer_weights* w, const vfm_lora_table* lora,
                           const vfm_batch* batch, const float* x, const void* k_cache,
                           const void* v_cache, int64_t kv_slots, Plan* pl) {
  if ((k_cache != nullptr) != (v_cache != nullptr)) return VFM_ERR_ARG;
  VFM_TRY(check_layer(cfg, w, lora, batch, x, k_cache != nullptr, pl));
  if (k_cache) {
    const PlanOffsets po = plan_offsets(pl->n_req, pl->n_tasks, pl->T);
    const int32_t* ctx = host_arr(batch, po.ctx);
    const int32_t* kvs = host_arr(batch, po.kv_start);
    const int32_t* cu = host_arr(batch, po.cu_seqlens);
    for (int p = 0; p < pl->n_req; ++p) {
      const int64_t end = (int64_t)kvs[p] + ctx[p] + (cu[p + 1] - cu[p]);
      if (end > kv_slots) return VFM_ERR_SHAPE;
    }
  }
  return VFM_OK;
}

}  // namespace

extern "C" int vfm_layer_forward(const vfm_cfg* cfg, const vfm_layer_weights* w,
                                 const vfm_lora_table* lora, const vfm_batch* batch, float* x,
                                 void* k_cache, void* v_cache, int64_t kv_slots, void* workspace,
                                 size_t ws_bytes, void* stream) {
  Plan pl;
  VFM_TRY(check_layer_contiguous(cfg, w, lora, batch, x, k_cache, v_cache, kv_slots, &pl));
  return layer_impl(*cfg, w, lora, batch, pl, x, k_cache, v_cache, kv_slots, KvPages{nullptr, 0, 0},
                    workspace, ws_bytes, stream);
}

// ---- the allocation-free layer call ----------------------------------------
namespace {

// Workspace of vfm_layer_forward_noalloc.  Every GPU the library runs on
// holds its own copy of this array, at its own address, until the process
// ends.  In host code `scratch` names a host-side stand-in, not the device
// memory: host code uses only the device address hipGetSymbolAddress returns
// for the current device (kept per device below), never the name itself.
static __device__ __align__(256) unsigned char scratch[VFM_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// Device address of the current device's scratch array, looked up once per
// device (with that device current) on its first call.  The stream must
// belong to the current device, since the address is that device's.
int scratch_of_current_device(hipStream_t s, void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return VFM_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return VFM_ERR_UNSUPPORTED;
  if (s != nullptr) {
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice(s, &sdev) != hipSuccess) return VFM_ERR_HIP;
    if (sdev != dev) return VFM_ERR_ARG;
  }
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_dev[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return VFM_ERR_HIP;
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return VFM_OK;
}

}  // namespace

extern "C" int vfm_layer_forward_noalloc(const vfm_cfg* cfg, const vfm_layer_weights* w,
                                         const vfm_lora_table* lora, const vfm_batch* batch, float* x,
                                         void* k_cache, void* v_cache, int64_t kv_slots, void* stream) {
  Plan pl;
  VFM_TRY(check_layer_contiguous(cfg, w, lora, batch, x, k_cache, v_cache, kv_slots, &pl));
  // the batch's workspace must fit the fixed scratch array (checked on the
  // host, before the device is touched)
  if (layer_ws(*cfg, pl, lora, max_keys_of(batch, pl)).total > VFM_NOALLOC_SCRATCH_BYTES)
    return VFM_ERR_WORKSPACE;
  void* ws = nullptr;
  VFM_TRY(scratch_of_current_device((hipStream_t)stream, &ws));
  // nothing in the scratch array needs to start at zero: every kernel writes
  // the workspace regions it reads in the same call (stale bytes of an
  // earlier call are never read)
  return layer_impl(*cfg, w, lora, batch, pl, x, k_cache, v_cache, kv_slots, KvPages{nullptr, 0, 0}, ws,
                    VFM_NOALLOC_SCRATCH_BYTES, stream);
}

extern "C" int vfm_layer_forward_paged(const vfm_cfg* cfg, const vfm_layer_weights* w,
                                       const vfm_lora_table* lora, const vfm_batch* batch, float* x,
                                       const vfm_kv_pages* kv, void* workspace, size_t ws_bytes,
                                       void* stream) {
  if (!kv || !kv->k || !kv->v || !kv->table_host || !kv->table_dev) return VFM_ERR_ARG;
  const int ps = kv->page_size;
  if (ps < 16 || ps > 1024 || (ps & (ps - 1))) return VFM_ERR_ARG;
  if (kv->n_pages < 1 || kv->max_pages < 1 || kv->n_pages > ((int64_t)1 << 40) / ps) return VFM_ERR_SHAPE;
  Plan pl;
  VFM_TRY(check_layer(cfg, w, lora, batch, x, true, &pl));
  if (cfg->attn == VFM_ATTN_BIDIR) return VFM_ERR_UNSUPPORTED;
  // every page a request uses (ctx + len tokens) exists
  const PlanOffsets po = plan_offsets(pl.n_req, pl.n_tasks, pl.T);
  const int32_t* ctx = host_arr(batch, po.ctx);
  const int32_t* cu = host_arr(batch, po.cu_seqlens);
  const int32_t* order = host_arr(batch, po.order);
  for (int p = 0; p < pl.n_req; ++p) {
    const int64_t need = ((int64_t)ctx[p] + (cu[p + 1] - cu[p]) + ps - 1) / ps;
    if (need > kv->max_pages) return VFM_ERR_SHAPE;
    const int32_t* row = kv->table_host + (int64_t)order[p] * kv->max_pages;
    for (int64_t j = 0; j < need; ++j)
      if (row[j] < 0 || row[j] >= kv->n_pages) return VFM_ERR_SHAPE;
  }
  int lp = 0;
  while ((1 << lp) < ps) ++lp;
  return layer_impl(*cfg, w, lora, batch, pl, x, kv->k, kv->v, kv->n_pages * ps,
                    KvPages{kv->table_dev, kv->max_pages, lp}, workspace, ws_bytes, stream);
}

namespace {

int layer_impl(const vfm_cfg& c, const vfm_layer_weights* w, const vfm_lora_table* lora,
               const vfm_batch* batch, const Plan& pl, float* x, void* k_cache, void* v_cache,
               int64_t kv_slots, const KvPages& kp, void* workspace, size_t ws_bytes, void* stream) {
  const int d = c.d_model, f = c.d_ff, T = pl.T;
  const int max_keys = max_keys_of(batch, pl);
  const LayerWs ws = layer_ws(c, pl, lora, max_keys);
  if (!workspace || ws_bytes < ws.total || ((uintptr_t)workspace % ALIGN)) return VFM_ERR_WORKSPACE;

  hipStream_t s = (hipStream_t)stream;
  char* base = (char*)workspace;
  void* h = base + ws.h;
  void* qkv = base + ws.big;
  void* act = base + ws.big;  // the MLP activation reuses the qkv region
  void* attn = base + ws.attn;
  void* U = base + ws.u;
  float* Z = (float*)(base + ws.z);
  float* P = (float*)(base + ws.p);
  const int rpad = rpad_of(lora);
  const int ldu = 8 * rpad;  // 7 projections + one spare slot
  const bool use_lora = lora && rpad > 0;

  const bool skinny = use_skinny(c, pl);

  auto has = [&](int p) { return use_lora && lora->A[p] != nullptr; };
  // One projection group: X [T, K] times the stacked weights (W, then W2
  // for SwiGLU), the per-task LoRA of `projs` (column slots of slot_width),
  // and the epilogue.
  // norm_into: for a residual projection, the pre-norm that follows it (its
  // output buffer); the small-batch path then fuses the two, and the caller
  // skips its own norm launch when `fused_norm` comes back true
  bool fused_norm = false;
  // set for the QKV projection of a small batch: the finalize applies RoPE
  // (and the cache write) itself
  FinRope fin_rope = {};
  // set for the QKV projection of a large bf16 batch: the GEMM applies RoPE
  GemmRope gemm_rope = {};
  auto project = [&](int cls, const void* X, int K, const void* W, const void* W2,
                     const void* bias, int N, int epi, void* out, int ldo,
                     std::initializer_list<int> projs, int slot_width, const void* norm_g = nullptr,
                     const void* norm_b = nullptr, void* norm_into = nullptr) -> int {
    fused_norm = false;
    bool any = false;
    for (int p : projs) any = any || has(p);
    if (!skinny) {
      if (any) {
        ShrinkArgs a = {};
        a.X = X; a.ldx = K; a.K = K; a.U = U; a.ldu = ldu; a.rpad = rpad;
        a.rank = lora->rank; a.scale = lora->scale;
        a.nsub = std::min(std::max(1, (lora->max_rank + 15) / 16), rpad / 16);
        for (int p : projs) {
          if (!has(p)) continue;
          a.A[a.n_proj] = lora->A[p];
          a.ucol[a.n_proj] = p * rpad;
          a.n_proj++;
        }
        VFM_TIMED(VFM_PROF_SHRINK, launch_lora_shrink(c.dtype, pl, a, s));
      }
      GemmArgs g = {};
      g.X = X; g.ldx = K; g.W = W; g.W2 = W2; g.bias = bias;
      g.M = T; g.N = N; g.K = K; g.epi = epi; g.out = out; g.ldo = ldo;
      g.rope = gemm_rope;
      if (any) {
        GemmLora& L = g.lora;
        int i = 0;
        for (int p : projs) {
          if (has(p)) L.B[i] = lora->B[p];
          L.ucol[i] = p * rpad;
          ++i;
        }
        L.enabled = 1;
        L.U = U; L.ldu = ldu; L.slot_width = slot_width;
        L.rank = lora->rank; L.row_task = pl.row_task; L.seg_row = pl.seg_row;
        L.max_rank = lora->max_rank;
      }
      VFM_TIMED(cls, launch_gemm(c.dtype, g, s));
      return VFM_OK;
    }
    // small batch: split-K shrink, split-K GEMM into partial slices, then
    // the streaming sum, which also reduces the shrink partials and adds
    // each row's LoRA difference
    const bool sw = epi == EPI_SWIGLU;
    const int nz = sw ? 2 * N : N;
    SkinnyArgs k = {};
    k.X = X; k.ldx = K; k.W = W; k.W2 = W2; k.n_half = N;
    k.M = T; k.N = nz; k.K = K; k.Z = Z;
    k.nsplit = skinny_splits(nz, K);
    FinalizeArgs fa = {};
    fa.Z = Z; fa.nslices = k.nsplit; fa.M = T; fa.N = N; fa.epi = epi; fa.bias = bias;
    fa.out = out; fa.ldo = ldo;
    fa.rope = fin_rope;
    if (any) {
      // the split shrink writes fp32 partials; the finalize pass sums them
      // into each row's U and adds U B_t^T to the row's columns
      ShrinkSplitArgs a = {};
      a.X = X; a.ldx = K; a.K = K; a.P = P; a.ldp = ldu; a.rpad = rpad;
      a.kchunks = shrink_chunks(K); a.rank = lora->rank;
      a.nsub = std::min(std::max(1, (lora->max_rank + 15) / 16), rpad / 16);
      for (int p : projs) {
        if (!has(p)) continue;
        a.A[a.n_proj] = lora->A[p];
        a.ucol[a.n_proj] = p * rpad;
        a.n_proj++;
      }
      VFM_TIMED(VFM_PROF_SHRINK, launch_shrink_split(pl, a, s));
      FinLora& fl = fa.lora;
      fl.enabled = 1;
      fl.P = P; fl.ldp = ldu; fl.cstride = (int64_t)T * ldu; fl.kchunks = a.kchunks;
      int i = 0;
      for (int p : projs) {
        fl.ucol[i] = p * rpad;
        fl.B[i] = has(p) ? lora->B[p] : nullptr;
        ++i;
      }
      fl.n_slots = i; fl.rpad = rpad;
      fl.slot_width = sw ? N : slot_width;
      fl.scale = lora->scale; fl.rank = lora->rank; fl.max_rank = lora->max_rank;
      fl.row_task = pl.row_task;
    }
    const int pi = prof_begin(cls, s);
    hipError_t e = launch_gemm_skinny(k, s);
    const bool fuse = norm_into != nullptr && epi == EPI_RESID && c.dtype == VFM_BF16 && ldo == N && N <= 8192;
    if (e == hipSuccess)
      e = fuse ? launch_finalize_norm(c.dtype, fa, norm_g, norm_b, c.norm, c.norm_eps, norm_into, s)
               : launch_finalize(fa, s);
    prof_end(pi, s);
    fused_norm = fuse && e == hipSuccess;
    return hip_status(e);
  };

  // a2: pre-norm 1
  VFM_TIMED(VFM_PROF_NORM, launch_norm(c.dtype, x, T, d, w->norm1_w, w->norm1_b, c.norm, c.norm_eps, h, s));
  // a5 (small bf16 batches): the QKV finalize also applies the rotary
  // embedding of q and k and, with a KV cache, writes each row's rotated k
  // and its v to its slot
  // (large bf16 batches): the QKV GEMM's store pass rotates q and k, and the
  // cache write is the attention launcher's plain copy
  const bool cache_write = k_cache != nullptr && c.attn != VFM_ATTN_BIDIR;
  const bool rope_fusable = c.dtype == VFM_BF16 && c.rope_theta > 0.f &&
                            (c.head_dim == 64 || c.head_dim == 128) && d % 256 == 0;
  const bool rope_in_finalize = skinny && rope_fusable;
  const bool rope_in_gemm = !skinny && rope_fusable && T >= 1024 &&
                            (int64_t)T * d < ((int64_t)1 << 31) && (int64_t)3 * d * d < ((int64_t)1 << 31);
  const bool rope_writes_kv = c.rope_theta > 0.f && cache_write && !rope_in_gemm;
  if (rope_in_gemm) {
    gemm_rope.on = 1; gemm_rope.d = d; gemm_rope.head_dim = c.head_dim;
    gemm_rope.log2_theta = log2f(c.rope_theta); gemm_rope.pos = pl.pos;
  }
  if (rope_in_finalize) {
    fin_rope.on = 1; fin_rope.d = d; fin_rope.head_dim = c.head_dim; fin_rope.log2_theta = log2f(c.rope_theta);
    fin_rope.pl = pl; fin_rope.kp = kp; fin_rope.kv_slots = kv_slots;
    fin_rope.kc = rope_writes_kv ? (bf16*)k_cache : nullptr;
    fin_rope.vc = rope_writes_kv ? (bf16*)v_cache : nullptr;
  }
  // a3 + a4: shared QKV projection with the per-task LoRA of q, k, v
  VFM_TRY(project(VFM_PROF_GEMM_QKV, h, d, w->w_qkv, nullptr, w->b_qkv, 3 * d, EPI_STORE, qkv,
                  3 * d, {VFM_Q, VFM_K, VFM_V}, d));
  fin_rope = FinRope{};
  gemm_rope = GemmRope{};
  // a5: rotary embedding of q and k
  // (with a KV cache the same pass writes each row's rotated k and its v)
  if (c.rope_theta > 0.f && !rope_in_finalize && !rope_in_gemm)
    VFM_TIMED(VFM_PROF_OTHER, launch_rope(c.dtype, pl, qkv, d, c.n_heads, c.head_dim, c.rope_theta,
                                          rope_writes_kv ? k_cache : nullptr, rope_writes_kv ? v_cache : nullptr,
                                          kv_slots, kp, s));
  // a6: attention per request (and the KV-cache write)
  // (timed per kernel inside the launcher)
  bool chunked = false;                      // a prompt chunk after cached tokens
  if (c.attn == VFM_ATTN_MIXED) {
    const PlanOffsets po = plan_offsets(pl.n_req, pl.n_tasks, pl.T);
    const int32_t* ctx = host_arr(batch, po.ctx);
    const int32_t* cu = host_arr(batch, po.cu_seqlens);
    for (int p = 0; p < pl.n_req && !chunked; ++p) chunked = ctx[p] > 0 && cu[p + 1] - cu[p] > 1;
  }
  VFM_HIP(launch_attention(c.dtype, pl, c, qkv, attn, k_cache, v_cache, kv_slots, kp, rope_writes_kv, chunked,
                           base + ws.aws, ws.z - ws.aws, max_keys, s));
  // a7: output projection + LoRA_o + residual
  VFM_TRY(project(VFM_PROF_GEMM_O, attn, d, w->w_o, nullptr, w->b_o, d, EPI_RESID, x, d, {VFM_O}, d,
                  w->norm2_w, w->norm2_b, h));
  // a8: pre-norm 2 (already done with the residual finalize on small batches)
  if (!fused_norm)
    VFM_TIMED(VFM_PROF_NORM, launch_norm(c.dtype, x, T, d, w->norm2_w, w->norm2_b, c.norm, c.norm_eps, h, s));
  // a9: MLP up (+ gate) with LoRA and the activation fused
  if (c.mlp == VFM_MLP_SWIGLU)
    VFM_TRY(project(VFM_PROF_GEMM_UP, h, d, w->w_gate, w->w_up, nullptr, f, EPI_SWIGLU, act, f,
                    {VFM_GATE, VFM_UP}, f));
  else
    VFM_TRY(project(VFM_PROF_GEMM_UP, h, d, w->w_up, nullptr, w->b_up, f, EPI_GELU, act, f,
                    {VFM_UP}, f));
  // a10: down projection + LoRA_down + residual
  VFM_TRY(project(VFM_PROF_GEMM_DOWN, act, f, w->w_down, nullptr, w->b_down, d, EPI_RESID, x, d,
                  {VFM_DOWN}, d));
  return VFM_OK;
}

}  // namespace

extern "C" int vfm_lora_apply(int32_t dtype, int32_t proj, int32_t d_in, int32_t d_out,
                              const vfm_lora_table* lora, const vfm_batch* batch, const void* x,
                              float* y, void* workspace, size_t ws_bytes, void* stream) {
  if (dtype != VFM_F32 && dtype != VFM_BF16) return VFM_ERR_ARG;
  if (proj < 0 || proj >= VFM_NPROJ) return VFM_ERR_ARG;
  if (!lora || !x || !y) return VFM_ERR_ARG;
  Plan pl;
  VFM_TRY(check_batch(batch, &pl));
  VFM_TRY(check_lora(lora, pl));
  if (!lora->A[proj]) return VFM_ERR_ARG;
  if (d_in < 64 || d_in % 64 || d_out < 4 || d_out % 4) return VFM_ERR_SHAPE;
  const int rpad = rpad_of(lora);
  if (rpad == 0) return VFM_OK;
  const size_t need = align_up((size_t)pl.T * rpad * elem_size(dtype));
  if (!workspace || ws_bytes < need || ((uintptr_t)workspace % ALIGN)) return VFM_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  ShrinkArgs a = {};
  a.X = x; a.ldx = d_in; a.K = d_in; a.U = workspace; a.ldu = rpad; a.rpad = rpad;
  a.rank = lora->rank; a.scale = lora->scale;
  a.nsub = std::min(std::max(1, (lora->max_rank + 15) / 16), rpad / 16);
  a.A[0] = lora->A[proj]; a.ucol[0] = 0; a.n_proj = 1;
  VFM_HIP(launch_lora_shrink(dtype, pl, a, s));
  ExpandArgs e = {};
  e.U = workspace; e.ldu = rpad; e.ucol = 0; e.B = lora->B[proj]; e.N = d_out;
  e.Y = y; e.ldy = d_out; e.rank = lora->rank; e.max_rank = lora->max_rank;
  VFM_HIP(launch_lora_expand(dtype, pl, e, s));
  return VFM_OK;
}

extern "C" int vfm_head_forward(const vfm_cfg* cfg, const void* final_norm_w,
                                const void* final_norm_b, const vfm_head_table* heads,
                                const vfm_batch* batch, const float* x, float* out,
                                void* workspace, size_t ws_bytes, void* stream) {
  VFM_TRY(check_cfg(cfg));
  Plan pl;
  VFM_TRY(check_batch(batch, &pl));
  if (!final_norm_w || !x || !out) return VFM_ERR_ARG;
  hipStream_t s = (hipStream_t)stream;
  const vfm_cfg& c = *cfg;
  if (!heads) {
    return hip_status(launch_norm_pool(c.dtype, pl, x, c.d_model, final_norm_w, final_norm_b,
                                       c.norm, c.norm_eps, -1, nullptr, out, s));
  }
  if (heads->n_tasks != pl.n_tasks || !heads->n_out || !heads->W) return VFM_ERR_ARG;
  if (heads->pool < VFM_POOL_MEAN || heads->pool > VFM_POOL_LAST) return VFM_ERR_ARG;
  if (heads->max_out < 0) return VFM_ERR_SHAPE;
  if (heads->W1) {
    if (heads->hidden < 64 || heads->hidden % 64 || heads->hidden > c.d_model) return VFM_ERR_SHAPE;
    if (heads->act != VFM_ACT_GELU && heads->act != VFM_ACT_RELU) return VFM_ERR_ARG;
  }
  if ((size_t)c.d_model * elem_size(c.dtype) > 64 * 1024) return VFM_ERR_UNSUPPORTED;
  const size_t need = head_ws(c, pl);
  if (!workspace || ws_bytes < need || ((uintptr_t)workspace % ALIGN)) return VFM_ERR_WORKSPACE;
  VFM_HIP(launch_norm_pool(c.dtype, pl, x, c.d_model, final_norm_w, final_norm_b, c.norm,
                           c.norm_eps, heads->pool, workspace, nullptr, s));
  VFM_HIP(launch_heads(c.dtype, pl, workspace, c.d_model, *heads, out, s));
  return VFM_OK;
}

extern "C" int vfm_greedy_tokens(const vfm_batch* batch, const float* out, int32_t* ids, void* stream) {
  Plan pl;
  VFM_TRY(check_batch(batch, &pl));
  if (!out || !ids) return VFM_ERR_ARG;
  return hip_status(launch_greedy(pl, out, ids, (hipStream_t)stream));
}
