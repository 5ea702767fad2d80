// a0: segmenting a mixed batch by task (host, integer).
//
// The scheduler's batch mixes requests of several vFMs; the backbone runs
// once over all rows and each task's adapter difference is applied per task
// (paper Section 4.2, adapter handling in "Batch-aware Fair Scheduling").
// Sorting the requests by task id (stable) makes every task's rows one
// contiguous segment, so the per-task kernels work on segments, not on
// scattered rows.
#include <vector>

#include "vfm_internal.h"

extern "C" int vfm_plan_size(int32_t n_req, int32_t n_tasks, int64_t total_rows, size_t* n_ints) {
  if (!n_ints) return VFM_ERR_ARG;
  if (n_req < 1 || n_tasks < 1 || total_rows < n_req || total_rows > INT32_MAX)
    return VFM_ERR_SHAPE;
  *n_ints = (size_t)plan_offsets(n_req, n_tasks, total_rows).total;
  return VFM_OK;
}

extern "C" int vfm_plan(const int32_t* task_id, const int32_t* seq_len, const int32_t* ctx_len,
                        const int32_t* kv_start, const int32_t* n_out, int32_t n_req,
                        int32_t n_tasks, int32_t* plan, size_t n_ints) {
  if (!task_id || !seq_len || !plan) return VFM_ERR_ARG;
  if (n_req < 1 || n_tasks < 1) return VFM_ERR_SHAPE;
  int64_t T = 0;
  int32_t max_len = 0;
  for (int32_t i = 0; i < n_req; ++i) {
    if (task_id[i] < 0 || task_id[i] >= n_tasks) return VFM_ERR_TASK;
    if (seq_len[i] < 1) return VFM_ERR_SHAPE;
    if (ctx_len && ctx_len[i] < 0) return VFM_ERR_SHAPE;
    if (kv_start && kv_start[i] < 0) return VFM_ERR_SHAPE;
    if (n_out && (n_out[task_id[i]] < 0)) return VFM_ERR_SHAPE;
    T += seq_len[i];
    if (seq_len[i] > max_len) max_len = seq_len[i];
  }
  if (T > INT32_MAX) return VFM_ERR_SHAPE;
  const PlanOffsets o = plan_offsets(n_req, n_tasks, T);
  if (n_ints < (size_t)o.total) return VFM_ERR_SHAPE;

  int32_t* order = plan + o.order;
  int32_t* task = plan + o.task;
  int32_t* cu = plan + o.cu_seqlens;
  int32_t* seg_req = plan + o.seg_req;
  int32_t* seg_row = plan + o.seg_row;
  int32_t* cu_orig = plan + o.cu_orig;
  int32_t* out_off = plan + o.out_off;
  int32_t* ctx = plan + o.ctx;
  int32_t* kvs = plan + o.kv_start;
  int32_t* qblk = plan + o.qblk_off;
  int32_t* rtile = plan + o.rtile_off;
  int32_t* row_task = plan + o.row_task;
  int32_t* row_req = plan + o.row_req;
  int32_t* pos = plan + o.pos;

  // counting sort by task id; filling positions in arrival order keeps it stable
  std::vector<int32_t> next(n_tasks + 1, 0);
  for (int32_t i = 0; i < n_req; ++i) next[task_id[i] + 1]++;
  for (int32_t t = 0; t < n_tasks; ++t) next[t + 1] += next[t];
  for (int32_t t = 0; t <= n_tasks; ++t) seg_req[t] = next[t];
  for (int32_t i = 0; i < n_req; ++i) order[next[task_id[i]]++] = i;

  cu[0] = 0;
  qblk[0] = 0;
  for (int32_t p = 0; p < n_req; ++p) {
    const int32_t i = order[p];
    task[p] = task_id[i];
    cu[p + 1] = cu[p] + seq_len[i];
    qblk[p + 1] = qblk[p] + (seq_len[i] + VFM_ROW_TILE - 1) / VFM_ROW_TILE;
    ctx[p] = ctx_len ? ctx_len[i] : 0;
    kvs[p] = kv_start ? kv_start[i] : 0;
    for (int32_t j = 0; j < seq_len[i]; ++j) {
      row_task[cu[p] + j] = task_id[i];
      row_req[cu[p] + j] = p;
      pos[cu[p] + j] = ctx[p] + j;
    }
  }
  rtile[0] = 0;
  for (int32_t t = 0; t <= n_tasks; ++t) seg_row[t] = cu[seg_req[t]];
  for (int32_t t = 0; t < n_tasks; ++t) {
    const int32_t rows = seg_row[t + 1] - seg_row[t];
    rtile[t + 1] = rtile[t] + (rows + VFM_ROW_TILE - 1) / VFM_ROW_TILE;
  }
  cu_orig[0] = 0;
  out_off[0] = 0;
  for (int32_t i = 0; i < n_req; ++i) {
    cu_orig[i + 1] = cu_orig[i] + seq_len[i];
    out_off[i + 1] = out_off[i] + (n_out ? n_out[task_id[i]] : 0);
  }

  for (int h = 0; h < VFM_PLAN_HEADER; ++h) plan[h] = 0;
  plan[0] = n_req;
  plan[1] = n_tasks;
  plan[2] = (int32_t)T;
  plan[3] = max_len;
  plan[4] = qblk[n_req];
  plan[5] = rtile[n_tasks];
  plan[6] = out_off[n_req];
  return VFM_OK;
}
