// Row-wise kernels: LayerNorm / RMSNorm (a2, a8), input embedding and
// permutation into plan order (a1), final norm + pooling (a11).
//
// All of these are HBM-bound streaming passes over [T, d] rows.  One wave64
// owns one row: each lane holds d/256 float4 chunks in registers, the mean and
// variance are wave-level butterfly reductions, and every global access is a
// coalesced 16-byte (fp32) or 8-byte (bf16x4) vector access.
#include "vfm_internal.h"

namespace {

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

template <typename T> __device__ inline float4 load4(const T* p);
template <> __device__ inline float4 load4<float>(const float* p) {
  return *reinterpret_cast<const float4*>(p);
}
template <> __device__ inline float4 load4<bf16>(const bf16* p) {
  bf16x4 v = *reinterpret_cast<const bf16x4*>(p);
  return make_float4((float)v[0], (float)v[1], (float)v[2], (float)v[3]);
}
template <typename T> __device__ inline void store4(T* p, float4 v);
template <> __device__ inline void store4<float>(float* p, float4 v) {
  *reinterpret_cast<float4*>(p) = v;
}
template <> __device__ inline void store4<bf16>(bf16* p, float4 v) {
  bf16x4 o;
  o[0] = (bf16)v.x; o[1] = (bf16)v.y; o[2] = (bf16)v.z; o[3] = (bf16)v.w;
  *reinterpret_cast<bf16x4*>(p) = o;
}

// Normalise one fp32 row held by one wave; MAXI = max float4 chunks per lane.
// For narrow rows (MAXI <= 8) the gain / shift loads are issued with the
// row's loads, so their latency overlaps the row's instead of following the
// two reductions; wide rows load them last (registers).
template <typename TW, int MAXI>
__device__ inline void norm_row_regs(const float* xr, int d, const TW* g, const TW* b, int kind,
                                     float eps, float4 (&v)[MAXI]) {
  const int lane = threadIdx.x & 63;
  const int nch = d >> 2;
  constexpr bool EARLY = MAXI <= 8;
  float4 gg[EARLY ? MAXI : 1], bb[EARLY ? MAXI : 1];
#pragma unroll
  for (int i = 0; i < MAXI; ++i) {
    const int c = lane + 64 * i;
    if (c < nch) {
      v[i] = *reinterpret_cast<const float4*>(xr + 4 * c);
      if (EARLY) {
        gg[EARLY ? i : 0] = load4<TW>(g + 4 * c);
        bb[EARLY ? i : 0] = b ? load4<TW>(b + 4 * c) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
  }
  float sum = 0.f;
#pragma unroll
  for (int i = 0; i < MAXI; ++i)
    if (lane + 64 * i < nch) sum += (v[i].x + v[i].y) + (v[i].z + v[i].w);
  float mean = 0.f;
  if (kind == VFM_NORM_LAYER) mean = wave_sum(sum) / (float)d;
  float sq = 0.f;
#pragma unroll
  for (int i = 0; i < MAXI; ++i) {
    const int c = lane + 64 * i;
    if (c < nch) {
      const float a = v[i].x - mean, b2 = v[i].y - mean, cc = v[i].z - mean, dd = v[i].w - mean;
      sq += (a * a + b2 * b2) + (cc * cc + dd * dd);
    }
  }
  const float rstd = rsqrtf(wave_sum(sq) / (float)d + eps);
#pragma unroll
  for (int i = 0; i < MAXI; ++i) {
    const int c = lane + 64 * i;
    if (c < nch) {
      float4 g4, b4;
      if (EARLY) {
        g4 = gg[EARLY ? i : 0];
        b4 = bb[EARLY ? i : 0];
      } else {
        g4 = load4<TW>(g + 4 * c);
        b4 = b ? load4<TW>(b + 4 * c) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
      v[i].x = (v[i].x - mean) * rstd * g4.x + b4.x;
      v[i].y = (v[i].y - mean) * rstd * g4.y + b4.y;
      v[i].z = (v[i].z - mean) * rstd * g4.z + b4.z;
      v[i].w = (v[i].w - mean) * rstd * g4.w + b4.w;
    }
  }
}

// Few rows (decode): one 256-thread block per row, MAXC float4 chunks per
// thread, block reductions through LDS, so a small batch still keeps every
// CU busy.
// Normalise one row held by a 256-thread block (MAXC float4 chunks per
// thread in v) and store it; block reductions through red.
template <typename T, int MAXC>
__device__ inline void norm_block_row(const float4 (&v)[MAXC], int d, const T* __restrict__ g,
                                      const T* __restrict__ b, int kind, float eps, T* __restrict__ o,
                                      float (&red)[2][4]) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nch = d >> 2;
  float4 gg[MAXC], bb[MAXC];
  float sum = 0.f;
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = tid + 256 * i;
    if (c < nch) {
      gg[i] = load4<T>(g + 4 * c);
      bb[i] = b ? load4<T>(b + 4 * c) : make_float4(0.f, 0.f, 0.f, 0.f);
      sum += (v[i].x + v[i].y) + (v[i].z + v[i].w);
    }
  }
  float mean = 0.f;
  if (kind == VFM_NORM_LAYER) {
    sum = wave_sum(sum);
    if (lane == 0) red[0][wave] = sum;
    __syncthreads();
    mean = ((red[0][0] + red[0][1]) + (red[0][2] + red[0][3])) / (float)d;
  }
  float sq = 0.f;
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = tid + 256 * i;
    if (c < nch) {
      const float a = v[i].x - mean, b2 = v[i].y - mean, cc = v[i].z - mean, dd = v[i].w - mean;
      sq += (a * a + b2 * b2) + (cc * cc + dd * dd);
    }
  }
  sq = wave_sum(sq);
  if (lane == 0) red[1][wave] = sq;
  __syncthreads();
  const float rstd = rsqrtf(((red[1][0] + red[1][1]) + (red[1][2] + red[1][3])) / (float)d + eps);
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = tid + 256 * i;
    if (c < nch) {
      float4 y;
      y.x = (v[i].x - mean) * rstd * gg[i].x + bb[i].x;
      y.y = (v[i].y - mean) * rstd * gg[i].y + bb[i].y;
      y.z = (v[i].z - mean) * rstd * gg[i].z + bb[i].z;
      y.w = (v[i].w - mean) * rstd * gg[i].w + bb[i].w;
      store4<T>(o + 4 * c, y);
    }
  }
}

template <typename T, int MAXC>
__global__ __launch_bounds__(256) void norm_rows_block_kernel(const float* __restrict__ x, int d,
                                                              const T* __restrict__ g,
                                                              const T* __restrict__ b, int kind,
                                                              float eps, T* __restrict__ out) {
  __shared__ float red[2][4];
  const int row = blockIdx.x, tid = threadIdx.x;
  const int nch = d >> 2;
  const float* xr = x + (int64_t)row * d;
  float4 v[MAXC];
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = tid + 256 * i;
    v[i] = c < nch ? *reinterpret_cast<const float4*>(xr + 4 * c) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  norm_block_row<T, MAXC>(v, d, g, b, kind, eps, out + (int64_t)row * d, red);
}

// Residual finalize + pre-norm, one block per row: x += (sum of the partial
// slices) + bias, then the row is normalised into h.
template <typename T, int MAXC>
__global__ __launch_bounds__(256) void finalize_norm_kernel(FinalizeArgs a, const T* __restrict__ g,
                                                            const T* __restrict__ b, int kind, float eps,
                                                            T* __restrict__ h) {
  __shared__ float red[2][4];
  __shared__ float Us[3 * VFM_MAX_RANK], ured[256];
  // block b takes row (b % 8) * per + b / 8: consecutive rows (often one
  // task's) run on one XCD, so the task's B rows come from that XCD's L2
  const int per = gridDim.x / 8;
  const int row = (blockIdx.x % 8) * per + blockIdx.x / 8, tid = threadIdx.x;
  if (row >= a.M) return;                     // block-uniform
  const int nch = a.N >> 2;
  const int64_t zs = (int64_t)a.M * a.N;
  float* xr = (float*)a.out + (int64_t)row * a.ldo;
  int t = 0, r = 0;
  FinB bp = {};
  if (a.lora.enabled) {                       // block-uniform
    t = a.lora.row_task[row];
    bp = fin_lora_bptrs(a.lora, t);
    r = fin_lora_u(a.lora, row, Us, ured);
  }
  float4 v[MAXC];
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = tid + 256 * i;
    v[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (c < nch) {
      float4 s4 = sum_slices(a.Z + (int64_t)row * a.N + 4 * c, zs, a.nslices);
      if (a.lora.enabled) {
        const int slot = min(4 * c / a.lora.slot_width, 2);
        add4(s4, fin_lora_delta(a.lora, bp, r, slot, 4 * c - slot * a.lora.slot_width, Us));
      }
      if (a.bias) {
        const bf16x4 bv = *reinterpret_cast<const bf16x4*>((const bf16*)a.bias + 4 * c);
        s4.x += (float)bv[0]; s4.y += (float)bv[1]; s4.z += (float)bv[2]; s4.w += (float)bv[3];
      }
      float4 xv = *reinterpret_cast<const float4*>(xr + 4 * c);
      add4(xv, s4);
      *reinterpret_cast<float4*>(xr + 4 * c) = xv;
      v[i] = xv;
    }
  }
  norm_block_row<T, MAXC>(v, a.N, g, b, kind, eps, h + (int64_t)row * a.N, red);
}

template <typename T, int MAXI>
__global__ __launch_bounds__(256) void norm_rows_kernel(const float* __restrict__ x, int n_rows,
                                                        int d, const T* __restrict__ g,
                                                        const T* __restrict__ b, int kind,
                                                        float eps, T* __restrict__ out) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n_rows) return;
  float4 v[MAXI];
  norm_row_regs<T, MAXI>(x + (int64_t)row * d, d, g, b, kind, eps, v);
  const int lane = threadIdx.x & 63;
  T* o = out + (int64_t)row * d;
#pragma unroll
  for (int i = 0; i < MAXI; ++i) {
    const int c = lane + 64 * i;
    if (c < (d >> 2)) store4<T>(o + 4 * c, v[i]);
  }
}

// Final norm of every row, written fp32 in ORIGINAL request order.
template <typename T, int MAXI>
__global__ __launch_bounds__(256) void norm_rows_unpermute_kernel(
    Plan pl, const float* __restrict__ x, int d, const T* __restrict__ g, const T* __restrict__ b,
    int kind, float eps, float* __restrict__ out) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= pl.T) return;
  float4 v[MAXI];
  norm_row_regs<T, MAXI>(x + (int64_t)row * d, d, g, b, kind, eps, v);
  const int p = pl.row_req[row];
  const int dst = pl.cu_orig[pl.order[p]] + (row - pl.cu_seqlens[p]);
  const int lane = threadIdx.x & 63;
  float* o = out + (int64_t)dst * d;
#pragma unroll
  for (int i = 0; i < MAXI; ++i) {
    const int c = lane + 64 * i;
    if (c < (d >> 2)) store4<float>(o + 4 * c, v[i]);
  }
}

// Final norm + pooling: one block per request in plan order, 16 / 8 / 4
// waves by row width, each summing its rows in registers.
template <int MAXI>
constexpr int pool_waves() { return MAXI <= 4 ? 16 : (MAXI <= 8 ? 8 : 4); }

template <typename T, int MAXI>
__global__ __launch_bounds__((64 * pool_waves<MAXI>())) void norm_pool_kernel(
    Plan pl, const float* __restrict__ x, int d, const T* __restrict__ g, const T* __restrict__ b, int kind,
    float eps, int pool, T* __restrict__ pooled) {
  constexpr int NWV = pool_waves<MAXI>();
  constexpr bool REG = MAXI <= 8;        // narrow rows: per-wave sums stay in registers
  extern __shared__ float acc[];  // [d]
  const int p = blockIdx.x;
  const int r0 = pl.cu_seqlens[p], r1 = pl.cu_seqlens[p + 1];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nch = d >> 2;
  int first = r0, last = r1;
  if (pool == VFM_POOL_FIRST) last = r0 + 1;
  if (pool == VFM_POOL_LAST) first = r1 - 1;
  for (int i = threadIdx.x; i < d; i += 64 * NWV) acc[i] = 0.f;
  __syncthreads();
  // adds a wave's float4 chunks into acc; the callers take the waves in a
  // fixed order, so the sum does not depend on scheduling
  auto add_to_acc = [&](const float4 (&u)[MAXI]) {
#pragma unroll
    for (int i = 0; i < MAXI; ++i) {
      const int c = lane + 64 * i;
      if (c < nch) {
        float4* a4 = reinterpret_cast<float4*>(acc) + c;
        float4 o = *a4;
        o.x += u[i].x; o.y += u[i].y; o.z += u[i].z; o.w += u[i].w;
        *a4 = o;
      }
    }
  };
  if constexpr (REG) {
    // each wave sums its rows (first + wave, + NWV, ...) in registers, then
    // the wave sums are added in wave order
    float4 sum[MAXI];
#pragma unroll
    for (int i = 0; i < MAXI; ++i) sum[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int r = first + wave; r < last; r += NWV) {
      float4 v[MAXI];
      norm_row_regs<T, MAXI>(x + (int64_t)r * d, d, g, b, kind, eps, v);
#pragma unroll
      for (int i = 0; i < MAXI; ++i) {
        sum[i].x += v[i].x; sum[i].y += v[i].y; sum[i].z += v[i].z; sum[i].w += v[i].w;
      }
    }
    for (int w = 0; w < NWV; ++w) {
      if (wave == w) add_to_acc(sum);
      __syncthreads();
    }
  } else {
    // wide rows: NWV rows per round, added in row order
    for (int rb = first; rb < last; rb += NWV) {
      const int r = rb + wave;
      float4 v[MAXI];
      if (r < last) norm_row_regs<T, MAXI>(x + (int64_t)r * d, d, g, b, kind, eps, v);
      for (int w = 0; w < NWV; ++w) {
        if (wave == w && r < last) add_to_acc(v);
        __syncthreads();
      }
    }
  }
  const float inv = 1.f / (float)(last - first);
  for (int i = threadIdx.x; i < d; i += 64 * NWV)
    pooled[(int64_t)p * d + i] = from_f32<T>(acc[i] * inv);
}

// Map a plan-order row to its row in the caller's original order.
__device__ inline int orig_row(const Plan& pl, int row) {
  const int p = pl.row_req[row];
  return pl.cu_orig[pl.order[p]] + (row - pl.cu_seqlens[p]);
}

template <typename T>
__global__ __launch_bounds__(256) void embed_rows_kernel(Plan pl, const T* __restrict__ src, int d,
                                                         float* __restrict__ x) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= pl.T) return;
  const int lane = threadIdx.x & 63;
  const T* s = src + (int64_t)orig_row(pl, row) * d;
  float* o = x + (int64_t)row * d;
  for (int c = lane; c < (d >> 2); c += 64) store4<float>(o + 4 * c, load4<T>(s + 4 * c));
}

template <typename T>
__global__ __launch_bounds__(256) void embed_tokens_kernel(Plan pl, const int32_t* __restrict__ ids,
                                                           int vocab, const T* __restrict__ table,
                                                           int d, float* __restrict__ x) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= pl.T) return;
  const int lane = threadIdx.x & 63;
  const int id = ids[orig_row(pl, row)];
  float* o = x + (int64_t)row * d;
  if (id < 0 || id >= vocab) {
    for (int c = lane; c < (d >> 2); c += 64) store4<float>(o + 4 * c, make_float4(0.f, 0.f, 0.f, 0.f));
    return;
  }
  const T* s = table + (int64_t)id * d;
  for (int c = lane; c < (d >> 2); c += 64) store4<float>(o + 4 * c, load4<T>(s + 4 * c));
}

// Patch embedding x = W_pe patch + b_pe, one wave per row, width <= 64.
// 8 consecutive weights (16-byte aligned for bf16, 32-byte for fp32) as floats
__device__ inline void load8w(const bf16* p, float (&v)[8]) {
  const bf16x8 q = *reinterpret_cast<const bf16x8*>(p);
#pragma unroll
  for (int k = 0; k < 8; ++k) v[k] = (float)q[k];
}
__device__ inline void load8w(const float* p, float (&v)[8]) {
  const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

template <typename T>
__global__ __launch_bounds__(256) void embed_patches_kernel(Plan pl, const float* __restrict__ src,
                                                            int width, const T* __restrict__ W,
                                                            const T* __restrict__ bias, int d,
                                                            float* __restrict__ x) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= pl.T) return;
  const int lane = threadIdx.x & 63;
  const float* s = src + (int64_t)orig_row(pl, row) * width;
  float* o = x + (int64_t)row * d;
  if (width == 8 && (d & 3) == 0) {
    // 8-wide patches: the patch in registers, 4 outputs per lane and pass,
    // each output's weight row one 16-byte load
    float pv[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) pv[k] = s[k];
    for (int n0 = 4 * lane; n0 < d; n0 += 256) {
      float r4[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float wv[8];
        load8w(W + (int64_t)(n0 + j) * 8, wv);
        float acc = bias ? to_f32(bias[n0 + j]) : 0.f;
#pragma unroll
        for (int k = 0; k < 8; ++k) acc += wv[k] * pv[k];
        r4[j] = acc;
      }
      *reinterpret_cast<float4*>(o + n0) = make_float4(r4[0], r4[1], r4[2], r4[3]);
    }
    return;
  }
  const float mine = lane < width ? s[lane] : 0.f;
  for (int n = lane; n < d; n += 64) {
    const T* w = W + (int64_t)n * width;
    float acc = bias ? to_f32(bias[n]) : 0.f;
    for (int k = 0; k < width; ++k) acc += to_f32(w[k]) * __shfl(mine, k, 64);
    o[n] = acc;
  }
}

inline int maxi_for(int d) { return d <= 1024 ? 4 : (d <= 4096 ? 16 : 32); }

}  // namespace

hipError_t launch_norm(int dtype, const float* x, int T, int d, const void* g, const void* b,
                       int kind, float eps, void* out, hipStream_t s) {
  if (T == 0) return hipSuccess;
  // Small bf16 batches (the small-batch path's side of VFM_SMALL_BATCH_ROWS):
  // a block per row (d <= 8192: <= 8 chunks per thread).  The choice follows
  // that threshold and nothing else, since the two kernels sum a row in
  // different orders: a row's result depends only on which side its batch is.
  if (dtype == VFM_BF16 && T < VFM_SMALL_BATCH_ROWS && d >= 1024) {
#define NORM_BLOCK(TT)                                                                           \
  hipLaunchKernelGGL((norm_rows_block_kernel<TT, 8>), dim3(T), dim3(256), 0, s, x, d, (const TT*)g, \
                     (const TT*)b, kind, eps, (TT*)out)
    if (dtype == VFM_BF16) NORM_BLOCK(bf16); else NORM_BLOCK(float);
#undef NORM_BLOCK
    return hipGetLastError();
  }
  dim3 grid((T + 3) / 4), block(256);
  const int mi = maxi_for(d);
#define NORM_LAUNCH(TT, MI)                                                                   \
  hipLaunchKernelGGL((norm_rows_kernel<TT, MI>), grid, block, 0, s, x, T, d, (const TT*)g,  \
                     (const TT*)b, kind, eps, (TT*)out)
  if (dtype == VFM_BF16) {
    if (mi == 4) NORM_LAUNCH(bf16, 4); else if (mi == 16) NORM_LAUNCH(bf16, 16); else NORM_LAUNCH(bf16, 32);
  } else {
    if (mi == 4) NORM_LAUNCH(float, 4); else if (mi == 16) NORM_LAUNCH(float, 16); else NORM_LAUNCH(float, 32);
  }
#undef NORM_LAUNCH
  return hipGetLastError();
}

hipError_t launch_finalize_norm(int dtype, const FinalizeArgs& a, const void* g, const void* b, int kind,
                                float eps, void* h, hipStream_t s) {
  if (a.M == 0) return hipSuccess;
  if (a.epi != EPI_RESID || dtype != VFM_BF16 || a.N % 4 || a.N > 8192 || a.ldo != a.N)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL((finalize_norm_kernel<bf16, 8>), dim3((a.M + 7) / 8 * 8), dim3(256), 0, s, a, (const bf16*)g,
                     (const bf16*)b, kind, eps, (bf16*)h);
  return hipGetLastError();
}

hipError_t launch_norm_pool(int dtype, const Plan& pl, const float* x, int d, const void* g,
                            const void* b, int kind, float eps, int pool, void* pooled,
                            float* rows_out, hipStream_t s) {
  const int mi = maxi_for(d);
  if (pool < 0) {
    dim3 grid((pl.T + 3) / 4), block(256);
#define NP_LAUNCH(TT, MI)                                                                      \
  hipLaunchKernelGGL((norm_rows_unpermute_kernel<TT, MI>), grid, block, 0, s, pl, x, d,      \
                     (const TT*)g, (const TT*)b, kind, eps, rows_out)
    if (dtype == VFM_BF16) {
      if (mi == 4) NP_LAUNCH(bf16, 4); else if (mi == 16) NP_LAUNCH(bf16, 16); else NP_LAUNCH(bf16, 32);
    } else {
      if (mi == 4) NP_LAUNCH(float, 4); else if (mi == 16) NP_LAUNCH(float, 16); else NP_LAUNCH(float, 32);
    }
#undef NP_LAUNCH
    return hipGetLastError();
  }
  dim3 grid(pl.n_req);
  const size_t lds = (size_t)d * sizeof(float);
#define PL_LAUNCH(TT, MI)                                                                            \
  hipLaunchKernelGGL((norm_pool_kernel<TT, MI>), grid, dim3(64 * pool_waves<MI>()), lds, s, pl, x, d, \
                     (const TT*)g, (const TT*)b, kind, eps, pool, (TT*)pooled)
  if (dtype == VFM_BF16) {
    if (mi == 4) PL_LAUNCH(bf16, 4); else if (mi == 16) PL_LAUNCH(bf16, 16); else PL_LAUNCH(bf16, 32);
  } else {
    if (mi == 4) PL_LAUNCH(float, 4); else if (mi == 16) PL_LAUNCH(float, 16); else PL_LAUNCH(float, 32);
  }
#undef PL_LAUNCH
  return hipGetLastError();
}

hipError_t launch_embed(int dtype, const Plan& pl, int mode, const void* src, int width,
                        const void* table, const void* bias, int d, float* x, hipStream_t s) {
  dim3 grid((pl.T + 3) / 4), block(256);
  if (mode == VFM_EMBED_ROWS) {
    if (dtype == VFM_BF16)
      hipLaunchKernelGGL(embed_rows_kernel<bf16>, grid, block, 0, s, pl, (const bf16*)src, d, x);
    else
      hipLaunchKernelGGL(embed_rows_kernel<float>, grid, block, 0, s, pl, (const float*)src, d, x);
  } else if (mode == VFM_EMBED_TOKENS) {
    if (dtype == VFM_BF16)
      hipLaunchKernelGGL(embed_tokens_kernel<bf16>, grid, block, 0, s, pl, (const int32_t*)src,
                         width, (const bf16*)table, d, x);
    else
      hipLaunchKernelGGL(embed_tokens_kernel<float>, grid, block, 0, s, pl, (const int32_t*)src,
                         width, (const float*)table, d, x);
  } else {
    if (dtype == VFM_BF16)
      hipLaunchKernelGGL(embed_patches_kernel<bf16>, grid, block, 0, s, pl, (const float*)src,
                         width, (const bf16*)table, (const bf16*)bias, d, x);
    else
      hipLaunchKernelGGL(embed_patches_kernel<float>, grid, block, 0, s, pl, (const float*)src,
                         width, (const float*)table, (const float*)bias, d, x);
  }
  return hipGetLastError();
}
