// Per-task input encoders fused with the shared patch embedding (paper
// Section 2.2 and Section 4.1 task extensions; the linear channel combiner
// of Section 4.3's pipeline example).  A request of task t arrives as C
// channels of its series; each embedded row first combines its patch's C
// channels with the task's weights, s = b_t + sum_c W_t[c] x_c, then applies
// the shared patch embedding x = W_pe s + b_pe.  The combined series never
// goes to HBM: one pass reads the raw channels and writes the rows.
#include "vfm_internal.h"

namespace {

struct SeriesArgs {
  const float* src;
  int patch, C;
  const float* const* W;        // encoder table: per task W_t [C] or NULL
  const float* const* b;        // per task b_t [1] or NULL; or NULL
  const void* W_pe;
  const void* b_pe;
  int d;
  float* x;
};

// One wave per embedded row (plan order), 4 rows per block.  Lane j < patch
// holds sample j of the row's combined patch; the output loop broadcasts it.
template <typename T>
__global__ __launch_bounds__(256) void embed_series_kernel(Plan pl, SeriesArgs a) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= pl.T) return;                                  // wave-uniform
  const int lane = threadIdx.x & 63;
  const int p = pl.row_req[row];
  const int t = pl.task[p];
  const int64_t len = pl.cu_seqlens[p + 1] - pl.cu_seqlens[p];
  const int64_t k = row - pl.cu_seqlens[p];                 // patch index within the request
  // channel c of the request starts at C * cu_orig[i] * patch + c * len * patch
  const float* s = a.src + (int64_t)pl.cu_orig[pl.order[p]] * a.C * a.patch + k * a.patch;
  const float* wt = a.W[t];
  float v = 0.f;
  if (lane < a.patch) {
    if (wt) {
      const float* bt = a.b ? a.b[t] : nullptr;
      v = bt ? bt[0] : 0.f;
      for (int c = 0; c < a.C; ++c) v = fmaf(wt[c], s[(int64_t)c * len * a.patch + lane], v);
    } else {
      v = s[lane];                                          // no encoder: channel 0
    }
  }
  const T* W = static_cast<const T*>(a.W_pe);
  const T* bias = static_cast<const T*>(a.b_pe);
  float* o = a.x + (int64_t)row * a.d;
  for (int n = lane; n < a.d; n += 64) {                    // d % 64 == 0: every lane runs each pass
    const T* w = W + (int64_t)n * a.patch;
    float acc = bias ? to_f32(bias[n]) : 0.f;
    for (int j = 0; j < a.patch; ++j) acc = fmaf(to_f32(w[j]), __shfl(v, j, 64), acc);
    o[n] = acc;
  }
}

__global__ void encoder_attach_kernel(const float** W, const float** b, int task, const float* w_new,
                                      const float* b_new) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  W[task] = w_new;
  if (b) b[task] = b_new;
}

}  // namespace

extern "C" int vfm_embed_series(const vfm_cfg* cfg, const vfm_batch* batch, const vfm_encoder_table* enc,
                                const float* src, int32_t patch, const void* W_pe, const void* b_pe, float* x,
                                void* stream) {
  if (!cfg || !batch || !enc || !src || !W_pe || !x || !enc->W) return VFM_ERR_ARG;
  if (cfg->dtype != VFM_F32 && cfg->dtype != VFM_BF16) return VFM_ERR_ARG;
  if (cfg->d_model < 64 || cfg->d_model % 64 || cfg->d_model > 8192) return VFM_ERR_SHAPE;
  // the same plan checks as every other entry point
  if (!batch->plan_host || !batch->plan_dev) return VFM_ERR_ARG;
  if (batch->n_ints < VFM_PLAN_HEADER) return VFM_ERR_SHAPE;
  const int32_t* h = batch->plan_host;
  if (h[0] < 1 || h[1] < 1 || h[2] < h[0]) return VFM_ERR_SHAPE;
  if ((size_t)plan_offsets(h[0], h[1], h[2]).total > batch->n_ints) return VFM_ERR_SHAPE;
  const Plan pl = make_plan(h, batch->plan_dev);
  if (enc->n_tasks != pl.n_tasks) return VFM_ERR_SHAPE;
  if (enc->n_channels < 1 || enc->n_channels > 64 || patch < 1 || patch > 64) return VFM_ERR_SHAPE;
  SeriesArgs a = {src, patch, enc->n_channels, enc->W, enc->b, W_pe, b_pe, cfg->d_model, x};
  const dim3 grid((pl.T + 3) / 4), block(256);
  if (cfg->dtype == VFM_BF16)
    hipLaunchKernelGGL(embed_series_kernel<bf16>, grid, block, 0, (hipStream_t)stream, pl, a);
  else
    hipLaunchKernelGGL(embed_series_kernel<float>, grid, block, 0, (hipStream_t)stream, pl, a);
  return hipGetLastError() == hipSuccess ? VFM_OK : VFM_ERR_HIP;
}

extern "C" int vfm_encoder_attach(const vfm_encoder_table* table, int32_t task, const float* W, const float* b,
                                  void* stream) {
  if (!table || !table->W) return VFM_ERR_ARG;
  if (task < 0 || task >= table->n_tasks) return VFM_ERR_TASK;
  if (b && !table->b) return VFM_ERR_ARG;
  hipLaunchKernelGGL(encoder_attach_kernel, dim3(1), dim3(64), 0, (hipStream_t)stream,
                     const_cast<const float**>(table->W), const_cast<const float**>(table->b), task, W,
                     W ? b : nullptr);
  return hipGetLastError() == hipSuccess ? VFM_OK : VFM_ERR_HIP;
}
