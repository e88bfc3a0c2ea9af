// Host-only C entry points over the page table, for CPU tests of the cache
// bookkeeping (built into libws_host.so with g++; no HIP involved).
#include <cstdint>

#include "pagetable.hpp"

#define WSH_API extern "C" __attribute__((visibility("default")))

WSH_API void* wsh_create(int32_t page_tokens, int32_t max_pages) {
  return new ws::PageTable(page_tokens, max_pages);
}
WSH_API void wsh_destroy(void* pt) { delete static_cast<ws::PageTable*>(pt); }

// 0 ok, 1 out of pages, 2 unknown, 3 committed, 4 shape
static int code(ws::PtStatus s) {
  switch (s) {
    case ws::PtStatus::ok: return 0;
    case ws::PtStatus::out_of_pages: return 1;
    case ws::PtStatus::unknown: return 2;
    case ws::PtStatus::committed: return 3;
    case ws::PtStatus::shape: return 4;
  }
  return -1;
}

WSH_API int wsh_acquire(void* pt, int32_t unit, int32_t kind, int32_t n_tokens, int32_t* created) {
  ws::Segment* s = nullptr;
  bool c = false;
  int r = code(static_cast<ws::PageTable*>(pt)->acquire(unit, kind, n_tokens, &s, &c));
  *created = c ? 1 : 0;
  return r;
}
WSH_API void wsh_commit(void* pt, int32_t unit) { static_cast<ws::PageTable*>(pt)->commit(unit); }
WSH_API int32_t wsh_evict_before(void* pt, int32_t unit) {
  return static_cast<ws::PageTable*>(pt)->evict_before(unit);
}
WSH_API int wsh_release(void* pt, int32_t unit, int32_t kind) {
  return code(static_cast<ws::PageTable*>(pt)->release(unit, kind));
}
WSH_API void wsh_reset(void* pt) { static_cast<ws::PageTable*>(pt)->reset(); }
WSH_API int32_t wsh_free_pages(void* pt) { return static_cast<ws::PageTable*>(pt)->free_pages(); }
WSH_API uint64_t wsh_version(void* pt) { return static_cast<ws::PageTable*>(pt)->version(); }
WSH_API int32_t wsh_n_segments(void* pt) {
  return static_cast<int32_t>(static_cast<ws::PageTable*>(pt)->segments().size());
}

// Writes up to cap (page, n_valid) pairs; returns the full count.
WSH_API int32_t wsh_visible(void* pt, int32_t q_unit, int32_t min_unit, uint32_t kind_mask,
                            int32_t* pages, int32_t* n_valid, int32_t cap) {
  std::vector<ws::PageRef> out;
  static_cast<ws::PageTable*>(pt)->visible_pages(ws::MaskSpec{q_unit, min_unit, kind_mask}, &out);
  for (int32_t i = 0; i < cap && i < static_cast<int32_t>(out.size()); ++i) {
    pages[i] = out[static_cast<size_t>(i)].page;
    n_valid[i] = out[static_cast<size_t>(i)].n_valid;
  }
  return static_cast<int32_t>(out.size());
}

// Page ids of one segment; returns the count, or -1 if absent.
WSH_API int32_t wsh_segment_pages(void* pt, int32_t unit, int32_t kind, int32_t* pages, int32_t cap) {
  const ws::Segment* s = static_cast<const ws::PageTable*>(pt)->find(unit, kind);
  if (!s) return -1;
  for (int32_t i = 0; i < cap && i < static_cast<int32_t>(s->pages.size()); ++i)
    pages[i] = s->pages[static_cast<size_t>(i)];
  return static_cast<int32_t>(s->pages.size());
}
