// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "vfm.h"

typedef __bf16 bf16;
typedef bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

#define VFM_WAVE 64

// Offsets of the plan arrays inside the int32 plan buffer (layout documented
// in vfm.h).  Shared by host and device code.
struct PlanOffsets {
  int64_t order, task, cu_seqlens, seg_req, seg_row, cu_orig, out_off, ctx, kv_start, qblk_off,
      rtile_off, row_task, row_req, pos, total;
};

__host__ __device__ inline PlanOffsets plan_offsets(int64_t n_req, int64_t n_tasks, int64_t T) {
  PlanOffsets o;
  int64_t p = VFM_PLAN_HEADER;
  o.order = p;      p += n_req;
  o.task = p;       p += n_req;
  o.cu_seqlens = p; p += n_req + 1;
  o.seg_req = p;    p += n_tasks + 1;
  o.seg_row = p;    p += n_tasks + 1;
  o.cu_orig = p;    p += n_req + 1;
  o.out_off = p;    p += n_req + 1;
  o.ctx = p;        p += n_req;
  o.kv_start = p;   p += n_req;
  o.qblk_off = p;   p += n_req + 1;
  o.rtile_off = p;  p += n_tasks + 1;
  o.row_task = p;   p += T;
  o.row_req = p;    p += T;
  o.pos = p;        p += T;
  o.total = p;
  return o;
}

// Device-side view of a plan.
struct Plan {
  const int32_t *order, *task, *cu_seqlens, *seg_req, *seg_row, *cu_orig, *out_off, *ctx,
      *kv_start, *qblk_off, *rtile_off, *row_task, *row_req, *pos;
  int32_t n_req, n_tasks, T, max_seqlen, n_qblocks, n_rtiles, total_outputs;
  // launch facts from the host copy: the longest request of at most
  // VFM_SHORT_ATTN_ROWS rows (0 if none) and the number of longer ones
  int32_t max_short, n_long;
};

// Prompt attention with head dim 64 takes the whole-request kernel for
// requests of at most this many rows and the flash kernel for longer ones
// (head dim 128: the flash kernel for every prompt; its whole-request variant
// needs 128 KB of LDS and measured slower), by each request's own length, so
// a request's result does not depend on the rest of the batch.
constexpr int VFM_SHORT_ATTN_ROWS = 256;

inline Plan make_plan(const int32_t* host, const int32_t* dev) {
  Plan p;
  p.n_req = host[0];
  p.n_tasks = host[1];
  p.T = host[2];
  p.max_seqlen = host[3];
  p.n_qblocks = host[4];
  p.n_rtiles = host[5];
  p.total_outputs = host[6];
  PlanOffsets o = plan_offsets(p.n_req, p.n_tasks, p.T);
  p.order = dev + o.order;
  p.task = dev + o.task;
  p.cu_seqlens = dev + o.cu_seqlens;
  p.seg_req = dev + o.seg_req;
  p.seg_row = dev + o.seg_row;
  p.cu_orig = dev + o.cu_orig;
  p.out_off = dev + o.out_off;
  p.ctx = dev + o.ctx;
  p.kv_start = dev + o.kv_start;
  p.qblk_off = dev + o.qblk_off;
  p.rtile_off = dev + o.rtile_off;
  p.row_task = dev + o.row_task;
  p.row_req = dev + o.row_req;
  p.pos = dev + o.pos;
  p.max_short = 0;
  p.n_long = 0;
  const int32_t* cu = host + o.cu_seqlens;
  for (int i = 0; i < p.n_req; ++i) {
    const int len = cu[i + 1] - cu[i];
    if (len > VFM_SHORT_ATTN_ROWS) ++p.n_long;
    else if (len > p.max_short) p.max_short = len;
  }
  return p;
}

// Largest i in [0, n) with arr[i] <= v, for a non-decreasing arr (arr[0] <= v).
__device__ inline int upper_index(const int32_t* arr, int n, int v) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (arr[mid] <= v) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// The task owning segmented row tile `tile` (rtile_off[t] <= tile <
// rtile_off[t + 1]; tasks without rows own no tile), found by the whole
// block in one round of parallel loads instead of a chain of dependent ones.
// Every thread of the block must call it: it ends with a barrier.
__device__ inline int block_tile_task(const Plan& pl, int tile, int* slot) {
  if (threadIdx.x == 0) *slot = 0;
  __syncthreads();
  for (int i = threadIdx.x; i < pl.n_tasks; i += blockDim.x)
    if (pl.rtile_off[i] <= tile && tile < pl.rtile_off[i + 1]) *slot = i;
  __syncthreads();
  return *slot;
}

__device__ __forceinline__ void add4(float4& a, const float4& b) {
  a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w;
}

// 16-byte load with the nontemporal hint (data read once)
__device__ __forceinline__ float4 load4_nt(const float* p) {
  typedef float f4v __attribute__((ext_vector_type(4)));
  const f4v v = __builtin_nontemporal_load(reinterpret_cast<const f4v*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}

// Sum of ns fp32 partial slices (stride zs floats) at z, 4 columns, in a
// fixed order: slice j goes to lane j mod 4 of four running sums, which are
// then added pairwise.  Each partial is read once: nontemporal loads.
__device__ __forceinline__ float4 sum_slices(const float* z, int64_t zs, int ns) {
  float4 s4[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) s4[j] = make_float4(0.f, 0.f, 0.f, 0.f);
  int sp = 0;
  for (; sp + 4 <= ns; sp += 4) {
    float4 v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = load4_nt(z + (sp + j) * zs);
#pragma unroll
    for (int j = 0; j < 4; ++j) add4(s4[j], v[j]);
  }
#pragma unroll
  for (int j = 0; j < 3; ++j)  // the last ns mod 4 slices
    if (sp + j < ns) add4(s4[j], load4_nt(z + (sp + j) * zs));
  add4(s4[0], s4[1]);
  add4(s4[2], s4[3]);
  add4(s4[0], s4[2]);
  return s4[0];
}

__device__ inline float to_f32(float v) { return v; }
__device__ inline float to_f32(bf16 v) { return (float)v; }
template <typename T> __device__ inline T from_f32(float v);
template <> __device__ inline float from_f32<float>(float v) { return v; }
template <> __device__ inline bf16 from_f32<bf16>(float v) { return (bf16)v; }

// GELU for bf16 outputs, x Phi(x) with no transcendental instruction:
// Phi(x) - 1/2 = x Q(x^2) on |x| <= 4, x clamped to +-4 outside (where Phi
// is within 3.2e-5 of 0 or 1).  Q has 8 terms, a weighted least-squares fit
// with Lawson reweighting to the normal CDF (gelu_fit.py in the package
// reproduces the coefficients); |error in Phi| <= 2.2e-5, so the GELU error
// is at most 1e-4 for |x| <= 4 and 5.4e-5 |x| beyond, far below the 2^-9
// relative rounding of the bf16 result.  11 VALU operations.
__device__ inline float gelu_fast(float v) {
  const float t = __builtin_amdgcn_fmed3f(v, -4.f, 4.f);
  const float u = t * t;
  float p = -1.58078362e-09f;
  p = fmaf(p, u, 1.21710954e-07f);
  p = fmaf(p, u, -4.1008625e-06f);
  p = fmaf(p, u, 8.06673488e-05f);
  p = fmaf(p, u, -0.00104820414f);
  p = fmaf(p, u, 0.00966487359f);
  p = fmaf(p, u, -0.0661753789f);
  p = fmaf(p, u, 0.39884752f);
  return v * fmaf(p, t, 0.5f);
}

// SiLU for bf16 outputs, v sigmoid(v) = v / (1 + 2^(-v log2 e)), from the
// hardware base-2 exponential and reciprocal (each within about 1 ulp, far
// below the 2^-9 relative rounding of the bf16 result): 5 VALU operations
// against ~23 for the library exponential and an IEEE divide.  For very
// negative v the power overflows to +inf, the reciprocal gives 0 and the
// result a signed zero, as the exact form does.
__device__ __forceinline__ float silu_fast(float v) {
  return v * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(v * -1.44269504088896341f));
}

// Benchmark timing hooks (profile.hip): bracket one launch of class `cls`.
int prof_begin(int cls, hipStream_t s);
void prof_end(int idx, hipStream_t s);

// ---- launchers implemented in the kernel translation units ---------------
// All return hipSuccess or the launch error.  Shapes are validated by the API
// layer before any of these is called.

// LayerNorm / RMSNorm of fp32 rows into dtype rows.
hipError_t launch_norm(int dtype, const float* x, int T, int d, const void* g, const void* b,
                       int kind, float eps, void* out, hipStream_t s);

// Segmented LoRA shrink: U[m, ucol[p] + j] = scale_t * sum_k X[m,k] A_{t,p}[j,k]
// for j < rank_t, zero for rank_t <= j < rpad; p over n_proj projections.
// nsub: 16-column sub-tiles worth computing, ceil(max_rank / 16) <= rpad / 16
// (columns past them are written as zeros).
struct ShrinkArgs {
  const void* X; int ldx; int K;
  const void* const* A[3]; int ucol[3]; int n_proj;
  void* U; int ldu; int rpad; int nsub;
  const int32_t* rank; const float* scale;
};
hipError_t launch_lora_shrink(int dtype, const Plan& pl, const ShrinkArgs& a, hipStream_t s);

// Segmented LoRA expand into fp32: Y[m, n] += sum_j U[m, ucol + j] B_t[n, j].
struct ExpandArgs {
  const void* U; int ldu; int ucol;
  const void* const* B; int N;
  float* Y; int ldy;
  const int32_t* rank; int max_rank;
};
hipError_t launch_lora_expand(int dtype, const Plan& pl, const ExpandArgs& a, hipStream_t s);

// Shared GEMM  C[m, n] = sum_k X[m, k] W[n, k]  with a fused epilogue.
enum GemmEpi {
  EPI_STORE = 0,      // out(dtype)[m, n] = acc + bias
  EPI_GELU = 1,       // out(dtype)[m, n] = GELU(acc + bias)
  EPI_RESID = 2,      // x(fp32)[m, n] += acc + bias
  EPI_SWIGLU = 3      // out(dtype)[m, j] = SiLU(gate) * up; W = gate rows, W2 = up rows
};
struct GemmLora {
  // Optional per-task LoRA expand fused into the GEMM, up to 3 column slots
  // (q/k/v of a stacked projection, or gate/up of SwiGLU).  Column n belongs
  // to slot n / slot_width (SwiGLU: gate = slot 0, up = slot 1).
  int enabled;
  const void* U; int ldu; int ucol[3];
  const void* const* B[3];
  int slot_width;
  const int32_t* rank; const int32_t* row_task; const int32_t* seg_row;
  int max_rank;
};
// Rotary embedding applied by the QKV GEMM of a large bf16 batch (EPI_STORE):
// rotate-half of the q and k columns (the first 2d) per head of head_dim
// columns at each row's position pos[m], in the epilogue's store pass on the
// staged bf16 sums (rounded again after the rotation, as a separate pass
// over q and k would).  Needs head_dim 64 or 128 and d a multiple of 256;
// the launcher then picks tiles whose width is a multiple of head_dim.
struct GemmRope {
  int on; int d; int head_dim; float log2_theta;
  const int32_t* pos;
};
struct GemmArgs {
  const void* X; int ldx;
  const void* W; const void* W2;   // W2: SwiGLU up weights
  const void* bias;                // [N] dtype or NULL
  int M, N, K;                     // N = output columns (SwiGLU: d_ff)
  int epi;
  void* out; int ldo;              // EPI_STORE/GELU/SWIGLU (dtype) or EPI_RESID (fp32)
  GemmLora lora;
  GemmRope rope;
  int m_lo, m_hi;                  // rows one large-tile launch covers (set by launch_gemm)
};
hipError_t launch_gemm(int dtype, const GemmArgs& a, hipStream_t s);

// ---- small-batch (decode) projections, bf16 only -------------------------
// Split-K shared GEMM into fp32 partials: Z[s, m, n] = sum over the s-th
// K range of X[m, k] W[n, k]; rows n >= n_half of the stacked weight come
// from W2 (SwiGLU: gate columns then up columns).
struct SkinnyArgs {
  const void* X; int ldx;
  const void* W; const void* W2; int n_half;
  int M, N, K;
  int nsplit;
  float* Z;
};
hipError_t launch_gemm_skinny(const SkinnyArgs& a, hipStream_t s);
int skinny_splits(int N, int K);

// Split-K segmented LoRA shrink into fp32 partials:
// P[c, m, ucol[p] + j] = sum over K chunk c of X[m, k] A_{t,p}[j, k] for
// j < rpad (zero past rank_t); kchunks chunks of kchunk columns.
// nsub: 16-column sub-tiles worth computing, ceil(max_rank / 16) <= rpad / 16
// (the finalize reads no partial column past a task's rank).
struct ShrinkSplitArgs {
  const void* X; int ldx; int K;
  const void* const* A[3]; int ucol[3]; int n_proj;
  float* P; int ldp; int rpad; int nsub; int kchunk; int kchunks;
  const int32_t* rank;
};
hipError_t launch_shrink_split(const Plan& pl, const ShrinkSplitArgs& a, hipStream_t s);
int shrink_chunks(int K);

// Where the K / V of token k of plan position p live in a head-major cache:
// slot kv_start[p] + k, or with a page table (original request order,
// max_pages columns) slot table[order[p]][k >> log2_page] pages in.
struct KvPages {
  const int32_t* table;       // device; NULL: contiguous (kv_start)
  int max_pages, log2_page;
};
__device__ inline int64_t kv_slot(const Plan& pl, const KvPages& kp, int p, int k) {
  if (!kp.table) return (int64_t)pl.kv_start[p] + k;
  const int pg = kp.table[(int64_t)pl.order[p] * kp.max_pages + (k >> kp.log2_page)];
  return ((int64_t)pg << kp.log2_page) + (k & ((1 << kp.log2_page) - 1));
}

// Per-task LoRA of a small-batch projection group, applied by the finalize
// pass: for row m of task t, U = bf16(s_t * sum_c P[c, m, ucol[i] + j]) (the
// split shrink's partials, four running sums by chunk index mod 4, added
// pairwise) and
// column n of slot i gains sum_{j < r_t} U[i][j] B_{t,i}[n', j], n' = the
// column within its slot (SwiGLU: gate columns slot 0, up columns slot 1).
struct FinLora {
  int enabled;
  const float* P; int ldp; int64_t cstride; int kchunks;   // P[c, m, col] at c * cstride + m * ldp + col
  int ucol[3]; int n_slots; int rpad;
  const void* const* B[3]; int slot_width;
  const float* scale; const int32_t* rank; int max_rank;
  const int32_t* row_task;
};

// Rotary embedding of the q and k columns, applied by the finalize of a
// small batch's QKV projection (EPI_STORE, bf16): rotate-half per head of
// head_dim columns at each row's position (pl.pos), before the bf16 rounding;
// with kc / vc non-null the row's rotated k and its v also go to its cache
// slot (kv_slot), as launch_rope does.  Needs head_dim 64 or 128 and d a
// multiple of 256 (a wave's 256 columns then lie in one part of the row).
struct FinRope {
  int on; int d; int head_dim; float log2_theta;
  Plan pl; bf16* kc; bf16* vc; int64_t kv_slots; KvPages kp;
};

// Sum of nslices partial slices Z[s] ([M, N], SwiGLU [M, 2N]: gate then up
// columns) in a fixed order, plus bias, plus the fused LoRA difference, and
// the epilogue of GemmEpi.
struct FinalizeArgs {
  const float* Z; int nslices; int M; int N; int epi;   // epi: GemmEpi
  const void* bias;
  void* out; int ldo;
  FinLora lora;
  FinRope rope;
};
hipError_t launch_finalize(const FinalizeArgs& a, hipStream_t s);

// The fused LoRA of the finalize pass for row m.  Every thread of the block
// calls fin_lora_u: it fills Us[i * rpad + j] = bf16(scale_t * sum over the
// K chunks c of P[c, m, ucol[i] + j]) for the slots with adapters and j < r
// (r = the row's task rank, returned) and ends with a barrier.  All threads
// share the sums: thread q takes element (i, j) = q % (n_slots * r) and
// chunk group q / (n_slots * r) of G = blockDim / (n_slots * r) groups
// (chunks g, g + G, ... added in increasing order, 8 loads in flight), and
// the G group sums are added in group order through red[blockDim].  The
// order follows from the row's rank and the weight's K split alone, never
// from the batch.
__device__ __forceinline__ int fin_lora_u(const FinLora& L, int m, float* Us, float* red) {
  const int t = L.row_task[m];
  const int r = min(L.rank[t], L.max_rank) & ~7;
  const float sc = L.scale[t];
  const int ne = L.n_slots * r;                 // <= 3 * VFM_MAX_RANK = 192 < 256 threads
  if (ne == 0) return r;                        // block-uniform: no slot reads Us
  const int G = blockDim.x / ne;
  const int q = threadIdx.x, g = q / ne, e = q - g * ne;
  float s = 0.f;
  if (g < G) {
    const int i = e / r, j = e - i * r;
    if (L.B[i] != nullptr) {
      const float* p = L.P + (int64_t)m * L.ldp + L.ucol[i] + j;
      for (int c0 = g; c0 < L.kchunks; c0 += 8 * G) {
        float v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const int c = c0 + k * G;
          v[k] = c < L.kchunks ? p[(int64_t)c * L.cstride] : 0.f;
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) s += v[k];
      }
    }
  }
  red[q] = s;
  __syncthreads();
  if (q < ne) {
    float u = 0.f;
    for (int k = 0; k < G; ++k) u += red[k * ne + q];
    const int i = q / r, j = q - i * r;
    Us[i * L.rpad + j] = (float)(bf16)(u * sc);
  }
  __syncthreads();
  return r;
}

// The row's task's B pointers of every slot, read at the start of the
// finalize (t is the block's own), so that after the U rebuild the B rows
// are requested at once instead of after one more dependent load.
struct FinB { const bf16* p0; const bf16* p1; const bf16* p2; };
__device__ __forceinline__ FinB fin_lora_bptrs(const FinLora& L, int t) {
  FinB b;
  b.p0 = L.B[0] != nullptr ? (const bf16*)L.B[0][t] : nullptr;
  b.p1 = L.B[1] != nullptr ? (const bf16*)L.B[1][t] : nullptr;
  b.p2 = L.B[2] != nullptr ? (const bf16*)L.B[2][t] : nullptr;
  return b;
}

// LoRA difference of 4 consecutive columns of slot i of row m (task t, rank
// r): rows brow .. brow + 3 of B_{t,i}, a fixed-order fp32 sum over the rank.
__device__ __forceinline__ float4 fin_lora_delta(const FinLora& L, const FinB& bp, int r, int i, int brow,
                                                 const float* Us) {
  float4 d = make_float4(0.f, 0.f, 0.f, 0.f);
  const bf16* B0 = i == 0 ? bp.p0 : i == 1 ? bp.p1 : bp.p2;
  if (r <= 0 || B0 == nullptr) return d;
  // B_t comes from a device pointer table: read it as global memory, not
  // through generic (flat) addressing
  typedef const bf16x8 __attribute__((address_space(1))) gbf16x8;
  const bf16* Bt = B0 + (int64_t)brow * r;
  const float* u = Us + i * L.rpad;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int j0 = 0; j0 < r; j0 += 8) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const bf16x8 bv = *(gbf16x8*)(Bt + (int64_t)c * r + j0);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[c] = fmaf(u[j0 + e], (float)bv[e], acc[c]);
    }
  }
  d.x = acc[0]; d.y = acc[1]; d.z = acc[2]; d.w = acc[3];
  return d;
}

// Residual finalize fused with the next pre-norm (small batches): per row,
// x += sum of the slices + bias (exactly as launch_finalize with EPI_RESID),
// then h = Norm(x) as launch_norm.
hipError_t launch_finalize_norm(int dtype, const FinalizeArgs& a, const void* g, const void* b, int kind,
                                float eps, void* h, hipStream_t s);

// In-place rotary embedding of the q and k parts of qkv [T, 3d]; with
// k_cache / v_cache (head-major [n_heads, kv_slots, head_dim]) non-null, each
// row's rotated k and its v are also written to its slot (kv_slot of pos).
hipError_t launch_rope(int dtype, const Plan& pl, void* qkv, int d, int n_heads, int head_dim,
                       float theta, void* k_cache, void* v_cache, int64_t kv_slots, const KvPages& kp,
                       hipStream_t s);

// Attention per request over qkv [T, 3d] (plan order) into out [T, d].
// Decode and mixed steps need attention_workspace() bytes of ws; max_keys =
// the largest ctx + length over the batch's requests.  kv_written: the rows'
// K / V are already in the cache (written by the RoPE pass), so no cache
// write here.  Mixed steps: prompts (ctx 0) attend causally over their own
// rows, single-row requests with ctx > 0 over their cached keys, and (bf16,
// `chunked` set) prompt chunks with ctx > 0 over the cached keys and their
// own rows, all read from the cache.
hipError_t launch_attention(int dtype, const Plan& pl, const vfm_cfg& c, const void* qkv,
                            void* out, void* k_cache, void* v_cache, int64_t kv_slots, const KvPages& kp,
                            bool kv_written, bool chunked, void* ws, size_t ws_bytes, int max_keys,
                            hipStream_t s);
size_t attention_workspace(const vfm_cfg& c, const Plan& pl, int max_keys);

// Input rows into the fp32 residual stream (plan order).
hipError_t launch_embed(int dtype, const Plan& pl, int mode, const void* src, int width,
                        const void* table, const void* bias, int d, float* x, hipStream_t s);

// Final norm + pooling into pooled [n_req, d] (dtype, plan order), or the
// final-normed rows [T, d] fp32 in original order when pool < 0.
hipError_t launch_norm_pool(int dtype, const Plan& pl, const float* x, int d, const void* g,
                            const void* b, int kind, float eps, int pool, void* pooled,
                            float* rows_out, hipStream_t s);

// Per-task heads on pooled rows: out[out_off[i] + j] = pooled[p] . W_t[j] + b_t[j].
hipError_t launch_heads(int dtype, const Plan& pl, const void* pooled, int d,
                        const vfm_head_table& h, float* out, hipStream_t s);

// Greedy next token per request: ids[i] = argmax of out[out_off[i] ..
// out_off[i + 1]) (original order), ties to the lowest index, NaN never
// chosen, -1 when nothing can be.
hipError_t launch_greedy(const Plan& pl, const float* out, int32_t* ids, hipStream_t s);
