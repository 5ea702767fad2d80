// Batch-aware fair queueing (BFQ) on the host: forms the mixed-task batches
// that the backbone kernels run (paper Section 4.2, "Batch-aware Fair
// Scheduling": start / finish tags of Eq. 1-2 derived from start-time fair
// queueing, batch growth bounded by b_max and the requests' deadlines, the
// re-tagging of Eq. 3 with the batch-dependent per-request service time, and
// for token-based FMs the token-level work charged in service-time units).
//
// State layout in the caller's buffer (all 8-byte fields):
//   Header | weight[n] | T[b_max + 1] | f_disp[n] | f_last[n] | head[n] |
//   count[n] | disp[n] | taken[n] | ring[n][max_queued] of Entry
// Each task's queue is a ring in arrival order; within a task the start tags
// never decrease, so the batch scan is a merge of the n queue heads by
// (start tag, task id).
#include <cmath>
#include <cstring>

#include "vfm.h"
#include "vfm_bfq.h"

namespace {

constexpr uint64_t BFQ_MAGIC = 0x4246513176666d31ull;   // identifies an initialised state

struct Header {
  uint64_t magic;
  int32_t n_tasks, b_max, max_queued, pad;
  double v;             // largest finish tag of the tasks' last dispatched requests
};

struct Entry {
  int64_t request;
  double arrival, deadline;
  double va;            // v when the request arrived
  double S, F;
};

struct View {
  Header* h;
  double *weight, *T, *f_disp, *f_last;
  int64_t *head, *count;
  int64_t* disp;        // != 0: the task has dispatched a request
  int64_t* taken;       // per call of vfm_bfq_next_batch: the task's requests in the batch
  Entry* ring;
  Entry& at(int t, int64_t k) const {   // k-th queued request of task t
    const int64_t q = h->max_queued;
    return ring[(int64_t)t * q + (head[t] + k) % q];
  }
};

size_t layout(int32_t n, int32_t b_max, int32_t q) {
  size_t off = sizeof(Header);
  off += sizeof(double) * ((size_t)n * 3 + (size_t)b_max + 1);    // weight, f_disp, f_last, T
  off += sizeof(int64_t) * (size_t)n * 4;                          // head, count, disp, taken
  off += sizeof(Entry) * (size_t)n * (size_t)q;
  return off;
}

View view(void* state) {
  View v;
  char* p = static_cast<char*>(state);
  v.h = reinterpret_cast<Header*>(p);
  const int32_t n = v.h->n_tasks, b = v.h->b_max;
  p += sizeof(Header);
  v.weight = reinterpret_cast<double*>(p); p += sizeof(double) * n;
  v.T = reinterpret_cast<double*>(p);      p += sizeof(double) * (b + 1);
  v.f_disp = reinterpret_cast<double*>(p); p += sizeof(double) * n;
  v.f_last = reinterpret_cast<double*>(p); p += sizeof(double) * n;
  v.head = reinterpret_cast<int64_t*>(p);  p += sizeof(int64_t) * n;
  v.count = reinterpret_cast<int64_t*>(p); p += sizeof(int64_t) * n;
  v.disp = reinterpret_cast<int64_t*>(p);  p += sizeof(int64_t) * n;
  v.taken = reinterpret_cast<int64_t*>(p); p += sizeof(int64_t) * n;
  v.ring = reinterpret_cast<Entry*>(p);
  return v;
}

bool valid_config(const vfm_bfq_config* c) {
  return c->n_tasks >= 1 && c->n_tasks <= (1 << 20) && c->b_max >= 1 && c->b_max <= (1 << 20) &&
         c->max_queued >= 1 && c->max_queued <= (1 << 24);
}

bool live(const void* state) {
  return state != nullptr && (reinterpret_cast<uintptr_t>(state) % 8) == 0 &&
         static_cast<const Header*>(state)->magic == BFQ_MAGIC;
}

}  // namespace

extern "C" int vfm_bfq_state_size(const vfm_bfq_config* cfg, size_t* bytes) {
  if (!cfg || !bytes) return VFM_ERR_ARG;
  if (!valid_config(cfg)) return VFM_ERR_SHAPE;
  *bytes = layout(cfg->n_tasks, cfg->b_max, cfg->max_queued);
  return VFM_OK;
}

extern "C" int vfm_bfq_init(const vfm_bfq_config* cfg, void* state, size_t bytes) {
  if (!cfg || !state || !cfg->weight || !cfg->batch_time) return VFM_ERR_ARG;
  if (reinterpret_cast<uintptr_t>(state) % 8) return VFM_ERR_ARG;
  if (!valid_config(cfg)) return VFM_ERR_SHAPE;
  if (bytes < layout(cfg->n_tasks, cfg->b_max, cfg->max_queued)) return VFM_ERR_SHAPE;
  for (int32_t i = 0; i < cfg->n_tasks; ++i)
    if (!(cfg->weight[i] > 0.0) || !std::isfinite(cfg->weight[i])) return VFM_ERR_SHAPE;
  for (int32_t b = 1; b <= cfg->b_max; ++b)
    if (!(cfg->batch_time[b] > 0.0) || !std::isfinite(cfg->batch_time[b])) return VFM_ERR_SHAPE;
  Header* h = static_cast<Header*>(state);
  std::memset(state, 0, layout(cfg->n_tasks, cfg->b_max, cfg->max_queued));
  h->n_tasks = cfg->n_tasks;
  h->b_max = cfg->b_max;
  h->max_queued = cfg->max_queued;
  const View v = view(state);
  for (int32_t i = 0; i < cfg->n_tasks; ++i) v.weight[i] = cfg->weight[i];
  v.T[0] = 0.0;
  for (int32_t b = 1; b <= cfg->b_max; ++b) v.T[b] = cfg->batch_time[b];
  h->magic = BFQ_MAGIC;
  return VFM_OK;
}

extern "C" int vfm_bfq_enqueue(void* state, int32_t task, int64_t request, double arrival,
                               double deadline) {
  if (!live(state)) return VFM_ERR_ARG;
  const View v = view(state);
  if (task < 0 || task >= v.h->n_tasks) return VFM_ERR_TASK;
  if (v.count[task] >= v.h->max_queued) return VFM_ERR_SHAPE;
  if (std::isnan(arrival) || std::isnan(deadline)) return VFM_ERR_SHAPE;
  v.count[task] += 1;
  Entry& e = v.at(task, v.count[task] - 1);
  e.request = request;
  e.arrival = arrival;
  e.deadline = deadline;
  e.va = v.h->v;                                  // v at arrival
  e.S = std::fmax(v.f_last[task], e.va);          // Eq. 1
  e.F = e.S + v.T[1] / v.weight[task];            // Eq. 2: one request's expected service
  v.f_last[task] = e.F;
  return VFM_OK;
}

extern "C" int vfm_bfq_next_batch(void* state, double now, int64_t* requests, int32_t* tasks,
                                  int32_t capacity, int32_t* n) {
  if (!live(state) || !requests || !tasks || !n) return VFM_ERR_ARG;
  const View v = view(state);
  const int32_t nt = v.h->n_tasks, b_max = v.h->b_max;
  if (capacity < b_max) return VFM_ERR_SHAPE;
  // Merge of the task queues by (start tag, task id): taken[t] requests of
  // task t are in the batch so far, all from the front of its queue.
  for (int32_t t = 0; t < nt; ++t) v.taken[t] = 0;
  int32_t b = 0;
  double min_deadline = INFINITY;
  while (b < b_max) {
    int32_t best = -1;
    double best_s = 0.0;
    for (int32_t t = 0; t < nt; ++t) {
      if (v.taken[t] >= v.count[t]) continue;
      const double s = v.at(t, v.taken[t]).S;
      if (best < 0 || s < best_s) { best = t; best_s = s; }   // ties keep the lower task id
    }
    if (best < 0) break;                                     // every queue is drained
    const Entry& cand = v.at(best, v.taken[best]);
    const double done = now + v.T[b + 1];
    const double md = std::fmin(min_deadline, cand.deadline);
    if (b > 0 && done > md) break;                           // would pass a deadline
    requests[b] = cand.request;
    tasks[b] = best;
    v.taken[best] += 1;
    min_deadline = md;
    ++b;
  }
  *n = b;
  if (b == 0) return VFM_OK;
  // Eq. 3: re-tag every contributing task with l(b) = T(b) / b, its
  // dispatched requests first (realised service), then its queued ones.
  const double lb = v.T[b] / b;
  for (int32_t t = 0; t < nt; ++t) {
    const int64_t k = v.taken[t];
    if (k == 0) continue;
    double prev = v.disp[t] ? v.f_disp[t] : 0.0;
    for (int64_t j = 0; j < v.count[t]; ++j) {
      Entry& e = v.at(t, j);
      e.S = std::fmax(prev, e.va);
      e.F = e.S + lb / v.weight[t];
      prev = e.F;
      if (j == k - 1) v.f_disp[t] = e.F;                  // the task's last dispatched request
    }
    v.f_last[t] = prev;
    v.disp[t] = 1;
    v.head[t] = (v.head[t] + k) % v.h->max_queued;
    v.count[t] -= k;
  }
  double vmax = 0.0;
  for (int32_t t = 0; t < nt; ++t)
    if (v.disp[t]) vmax = std::fmax(vmax, v.f_disp[t]);
  v.h->v = vmax;
  return VFM_OK;
}

extern "C" int vfm_bfq_charge(void* state, int32_t task, double service) {
  if (!live(state)) return VFM_ERR_ARG;
  const View v = view(state);
  if (task < 0 || task >= v.h->n_tasks) return VFM_ERR_TASK;
  if (!(service >= 0.0) || !std::isfinite(service)) return VFM_ERR_SHAPE;
  // the realised work extends the task's last dispatched request: its finish
  // tag moves by service / w, and the queued requests' tags follow, chained
  // as Eq. 1 from their own arrival-time v with their own service lengths
  const double w = v.weight[task];
  double prev = (v.disp[task] ? v.f_disp[task] : 0.0) + service / w;
  v.f_disp[task] = prev;
  v.disp[task] = 1;
  for (int64_t j = 0; j < v.count[task]; ++j) {
    Entry& e = v.at(task, j);
    const double len = e.F - e.S;
    e.S = std::fmax(prev, e.va);
    e.F = e.S + len;
    prev = e.F;
  }
  v.f_last[task] = prev;
  double vmax = 0.0;
  for (int32_t t = 0; t < v.h->n_tasks; ++t)
    if (v.disp[t]) vmax = std::fmax(vmax, v.f_disp[t]);
  v.h->v = vmax;
  return VFM_OK;
}

extern "C" int vfm_bfq_queued(const void* state, int32_t task, int32_t* n) {
  if (!live(state) || !n) return VFM_ERR_ARG;
  const View v = view(const_cast<void*>(state));
  if (task < 0 || task >= v.h->n_tasks) return VFM_ERR_TASK;
  *n = (int32_t)v.count[task];
  return VFM_OK;
}

extern "C" int vfm_bfq_tags(const void* state, int32_t task, int32_t k, double* start, double* finish) {
  if (!live(state) || !start || !finish) return VFM_ERR_ARG;
  const View v = view(const_cast<void*>(state));
  if (task < 0 || task >= v.h->n_tasks) return VFM_ERR_TASK;
  if (k < 0 || k >= v.count[task]) return VFM_ERR_SHAPE;
  *start = v.at(task, k).S;
  *finish = v.at(task, k).F;
  return VFM_OK;
}
