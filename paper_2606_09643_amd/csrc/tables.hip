// Runtime attach / remove of one task's extensions (paper Section 4.1 task
// extensions; Table 1 attach_adapter / remove_adapter / add_decoder): the
// per-task entries of the caller's device tables are rewritten by a
// one-thread kernel on the caller's stream, so the update is ordered with the
// forward calls on that stream, needs no host synchronisation, and leaves the
// backbone weights and every other task's entries untouched.  The new values
// travel as kernel arguments (nothing to keep alive on the host).
#include "vfm_internal.h"

namespace {

struct LoraEntry {
  int32_t* rank; float* scale;
  const void** A[VFM_NPROJ];
  const void** B[VFM_NPROJ];
  int32_t task, new_rank; float new_scale;
  const void* a[VFM_NPROJ];
  const void* b[VFM_NPROJ];
};

__global__ void lora_attach_kernel(LoraEntry e) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  for (int p = 0; p < VFM_NPROJ; ++p) {
    if (e.A[p]) e.A[p][e.task] = e.a[p];
    if (e.B[p]) e.B[p][e.task] = e.b[p];
  }
  e.scale[e.task] = e.new_scale;
  e.rank[e.task] = e.new_rank;
}

struct HeadEntry {
  int32_t* n_out;
  const void** W;
  const void** b;
  const void** W1;
  const void** b1;
  int32_t task, new_n_out;
  const void* w_new;
  const void* b_new;
  const void* w1_new;
  const void* b1_new;
};

__global__ void head_attach_kernel(HeadEntry e) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  e.W[e.task] = e.w_new;
  if (e.b) e.b[e.task] = e.b_new;
  if (e.W1) e.W1[e.task] = e.w1_new;
  if (e.b1) e.b1[e.task] = e.b1_new;
  e.n_out[e.task] = e.new_n_out;
}

}  // namespace

extern "C" int vfm_lora_attach(const vfm_lora_table* table, int32_t task, int32_t rank, float scale,
                               const void* const* A, const void* const* B, void* stream) {
  if (!table || !table->rank || !table->scale) return VFM_ERR_ARG;
  if (task < 0 || task >= table->n_tasks) return VFM_ERR_TASK;
  if (rank < 0 || rank % 8 || rank > table->max_rank) return VFM_ERR_SHAPE;
  LoraEntry e = {};
  e.rank = const_cast<int32_t*>(table->rank);
  e.scale = const_cast<float*>(table->scale);
  e.task = task;
  e.new_rank = rank;
  e.new_scale = scale;
  for (int p = 0; p < VFM_NPROJ; ++p) {
    e.A[p] = const_cast<const void**>(table->A[p]);
    e.B[p] = const_cast<const void**>(table->B[p]);
    const void* a = (rank > 0 && A) ? A[p] : nullptr;
    const void* b = (rank > 0 && B) ? B[p] : nullptr;
    if ((a != nullptr) != (b != nullptr)) return VFM_ERR_ARG;          // A and B come in pairs
    if (a && (!table->A[p] || !table->B[p])) return VFM_ERR_ARG;       // projection without adapters
    e.a[p] = a;
    e.b[p] = b;
  }
  hipLaunchKernelGGL(lora_attach_kernel, dim3(1), dim3(64), 0, (hipStream_t)stream, e);
  return hipGetLastError() == hipSuccess ? VFM_OK : VFM_ERR_HIP;
}

extern "C" int vfm_head_attach(const vfm_head_table* table, int32_t task, int32_t n_out, const void* W,
                               const void* b, const void* W1, const void* b1, void* stream) {
  if (!table || !table->n_out || !table->W) return VFM_ERR_ARG;
  if (task < 0 || task >= table->n_tasks) return VFM_ERR_TASK;
  if (n_out < 0 || n_out > table->max_out) return VFM_ERR_SHAPE;
  if (n_out > 0 && !W) return VFM_ERR_ARG;
  if (b && !table->b) return VFM_ERR_ARG;
  if ((W1 || b1) && !table->W1) return VFM_ERR_ARG;   // MLP head without MLP tables
  if (b1 && !table->b1) return VFM_ERR_ARG;
  if (b1 && !W1) return VFM_ERR_ARG;
  HeadEntry e = {};
  e.n_out = const_cast<int32_t*>(table->n_out);
  e.W = const_cast<const void**>(table->W);
  e.b = const_cast<const void**>(table->b);
  e.W1 = const_cast<const void**>(table->W1);
  e.b1 = const_cast<const void**>(table->b1);
  e.task = task;
  e.new_n_out = n_out;
  e.w_new = n_out > 0 ? W : nullptr;
  e.b_new = n_out > 0 ? b : nullptr;
  e.w1_new = n_out > 0 ? W1 : nullptr;
  e.b1_new = n_out > 0 ? b1 : nullptr;
  hipLaunchKernelGGL(head_attach_kernel, dim3(1), dim3(64), 0, (hipStream_t)stream, e);
  return hipGetLastError() == hipSuccess ? VFM_OK : VFM_ERR_HIP;
}
