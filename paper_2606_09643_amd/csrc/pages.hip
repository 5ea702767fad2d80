// KV page allocator on the host: page ids of one paged KV pool handed to
// sequences as they grow and taken back when they finish (continuous
// batching of token-based FMs, paper Section 4.2 and Section 6).
//
// State layout in the caller's buffer:
//   Header | free stack int32[n_pages] | held int32[max_seqs] |
//   pages int32[max_seqs][max_pages]
// The free stack's top is the next page handed out.
#include <cstring>

#include "vfm.h"
#include "vfm_pages.h"

namespace {

constexpr uint64_t PAGES_MAGIC = 0x7061676573766d31ull;   // identifies an initialised state

struct Header {
  uint64_t magic;
  int32_t n_pages, page_size, max_seqs, max_pages;
  int32_t n_free, pad;
};

struct View {
  Header* h;
  int32_t* free_stack;   // [n_pages], entries 0 .. n_free - 1 are free, top last
  int32_t* held;         // [max_seqs]
  int32_t* pages;        // [max_seqs][max_pages]
  int32_t* row(int s) const { return pages + (int64_t)s * h->max_pages; }
};

bool valid(const vfm_pages_config* c) {
  return c->n_pages >= 1 && c->n_pages <= (1 << 30) && c->page_size >= 1 && c->max_seqs >= 1 &&
         c->max_seqs <= (1 << 24) && c->max_pages >= 1 && c->max_pages <= (1 << 30) &&
         (int64_t)c->max_seqs * c->max_pages <= ((int64_t)1 << 32);
}

size_t layout(const vfm_pages_config* c) {
  return sizeof(Header) + sizeof(int32_t) * ((size_t)c->n_pages + (size_t)c->max_seqs +
                                             (size_t)c->max_seqs * (size_t)c->max_pages);
}

View view(void* state) {
  View v;
  char* p = static_cast<char*>(state);
  v.h = reinterpret_cast<Header*>(p);
  p += sizeof(Header);
  v.free_stack = reinterpret_cast<int32_t*>(p); p += sizeof(int32_t) * v.h->n_pages;
  v.held = reinterpret_cast<int32_t*>(p);       p += sizeof(int32_t) * v.h->max_seqs;
  v.pages = reinterpret_cast<int32_t*>(p);
  return v;
}

bool live(const void* state) {
  return state != nullptr && (reinterpret_cast<uintptr_t>(state) % 8) == 0 &&
         static_cast<const Header*>(state)->magic == PAGES_MAGIC;
}

}  // namespace

extern "C" int vfm_pages_state_size(const vfm_pages_config* cfg, size_t* bytes) {
  if (!cfg || !bytes) return VFM_ERR_ARG;
  if (!valid(cfg)) return VFM_ERR_SHAPE;
  *bytes = layout(cfg);
  return VFM_OK;
}

extern "C" int vfm_pages_init(const vfm_pages_config* cfg, void* state, size_t bytes) {
  if (!cfg || !state || (reinterpret_cast<uintptr_t>(state) % 8)) return VFM_ERR_ARG;
  if (!valid(cfg) || bytes < layout(cfg)) return VFM_ERR_SHAPE;
  std::memset(state, 0, layout(cfg));
  Header* h = static_cast<Header*>(state);
  h->n_pages = cfg->n_pages;
  h->page_size = cfg->page_size;
  h->max_seqs = cfg->max_seqs;
  h->max_pages = cfg->max_pages;
  h->n_free = cfg->n_pages;
  const View v = view(state);
  for (int32_t i = 0; i < cfg->n_pages; ++i) v.free_stack[i] = cfg->n_pages - 1 - i;   // page 0 on top
  h->magic = PAGES_MAGIC;
  return VFM_OK;
}

extern "C" int vfm_pages_reserve(void* state, int32_t seq, int64_t n_tokens) {
  if (!live(state)) return VFM_ERR_ARG;
  const View v = view(state);
  if (seq < 0 || seq >= v.h->max_seqs) return VFM_ERR_TASK;
  if (n_tokens < 0) return VFM_ERR_SHAPE;
  const int64_t need = (n_tokens + v.h->page_size - 1) / v.h->page_size;
  const int32_t have = v.held[seq];
  if (need <= have) return VFM_OK;
  if (need > v.h->max_pages || need - have > v.h->n_free) return VFM_ERR_SHAPE;
  int32_t* r = v.row(seq);
  for (int64_t j = have; j < need; ++j) r[j] = v.free_stack[--v.h->n_free];
  v.held[seq] = (int32_t)need;
  return VFM_OK;
}

extern "C" int vfm_pages_release(void* state, int32_t seq) {
  if (!live(state)) return VFM_ERR_ARG;
  const View v = view(state);
  if (seq < 0 || seq >= v.h->max_seqs) return VFM_ERR_TASK;
  const int32_t* r = v.row(seq);
  // pushed last page first, so the sequence's first page is handed out next
  for (int32_t j = v.held[seq] - 1; j >= 0; --j) v.free_stack[v.h->n_free++] = r[j];
  v.held[seq] = 0;
  return VFM_OK;
}

extern "C" int vfm_pages_table(const void* state, const int32_t* seqs, int32_t n, int32_t* table,
                               int32_t max_cols) {
  if (!live(state) || (n > 0 && (!seqs || !table))) return VFM_ERR_ARG;
  if (n < 0 || max_cols < 1) return VFM_ERR_SHAPE;
  const View v = view(const_cast<void*>(state));
  for (int32_t i = 0; i < n; ++i) {
    if (seqs[i] < 0 || seqs[i] >= v.h->max_seqs) return VFM_ERR_TASK;
    if (v.held[seqs[i]] > max_cols) return VFM_ERR_SHAPE;
  }
  for (int32_t i = 0; i < n; ++i) {
    const int32_t s = seqs[i], k = v.held[s];
    int32_t* out = table + (int64_t)i * max_cols;
    std::memcpy(out, v.row(s), sizeof(int32_t) * k);
    for (int32_t j = k; j < max_cols; ++j) out[j] = -1;
  }
  return VFM_OK;
}

extern "C" int vfm_pages_count(const void* state, int32_t seq, int32_t* held, int32_t* free_pages) {
  if (!live(state) || !held || !free_pages) return VFM_ERR_ARG;
  const View v = view(const_cast<void*>(state));
  if (seq < 0 || seq >= v.h->max_seqs) return VFM_ERR_TASK;
  *held = v.held[seq];
  *free_pages = v.h->n_free;
  return VFM_OK;
}
