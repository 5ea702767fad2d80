// Optional per-class kernel timing with hipEvents (benchmarks only).
#include <mutex>
#include <vector>

#include "vfm_internal.h"

namespace {

struct Rec {
  int cls;
  hipEvent_t a, b;
};

std::mutex g_mu;
uint32_t g_mask = 0;
std::vector<Rec> g_recs;
std::vector<hipEvent_t> g_pool;

hipEvent_t take_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

}  // namespace

int prof_begin(int cls, hipStream_t s) {
  if (!(g_mask & (1u << cls))) return -1;
  std::lock_guard<std::mutex> lk(g_mu);
  Rec r{cls, take_event(), take_event()};
  if (!r.a || !r.b) return -1;
  hipEventRecord(r.a, s);
  g_recs.push_back(r);
  return (int)g_recs.size() - 1;
}

void prof_end(int idx, hipStream_t s) {
  if (idx < 0) return;
  std::lock_guard<std::mutex> lk(g_mu);
  hipEventRecord(g_recs[idx].b, s);
}

extern "C" int vfm_profile_enable(uint32_t class_mask) {
  std::lock_guard<std::mutex> lk(g_mu);
  for (auto& r : g_recs) {
    hipEventSynchronize(r.b);
    g_pool.push_back(r.a);
    g_pool.push_back(r.b);
  }
  g_recs.clear();
  g_mask = class_mask;
  return VFM_OK;
}

extern "C" int vfm_profile_read(double* ms, int64_t* launches, int32_t n_classes) {
  if (!ms || !launches || n_classes < 1) return VFM_ERR_ARG;
  std::lock_guard<std::mutex> lk(g_mu);
  for (int c = 0; c < n_classes; ++c) {
    ms[c] = 0.0;
    launches[c] = 0;
  }
  for (auto& r : g_recs) {
    if (r.cls >= n_classes) continue;
    if (hipEventSynchronize(r.b) != hipSuccess) return VFM_ERR_HIP;
    float t = 0.f;
    if (hipEventElapsedTime(&t, r.a, r.b) != hipSuccess) return VFM_ERR_HIP;
    ms[r.cls] += t;
    launches[r.cls] += 1;
  }
  return VFM_OK;
}
