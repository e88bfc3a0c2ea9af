// Host-side page table of the paged K/V cache (pure C++, no HIP).
//
// The performer keeps a pre-allocated local K/V cache that the thinker's
// slices and the generated units are written into (Wan-Streamer v0.2,
// Abstract; Sec. 3).  Here the cache is a pool of fixed-size pages; every
// (unit, kind) segment owns a list of whole pages (a segment always starts on
// a fresh page, so a unit's last page may be partly filled).  This file keeps
// that bookkeeping and turns a block-causal mask into the list of visible
// pages the attention kernels walk.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace ws {

struct PageRef {
  int32_t page;     // page id in the pool
  int32_t n_valid;  // valid tokens in the page, 1..page_tokens
};

struct Segment {
  int32_t unit = 0;
  int32_t kind = 0;
  int32_t n_tokens = 0;
  bool committed = false;
  uint64_t serial = 0;          // creation order
  std::vector<int32_t> pages;   // page ids in token order
};

struct MaskSpec {
  int32_t q_unit;
  int32_t min_visible_unit;
  uint32_t kind_mask;
};

enum class PtStatus { ok, out_of_pages, unknown, committed, shape };

class PageTable {
 public:
  PageTable(int32_t page_tokens, int32_t max_pages);

  int32_t page_tokens() const { return page_tokens_; }
  int32_t max_pages() const { return max_pages_; }
  int32_t free_pages() const { return n_free_; }
  const std::vector<Segment>& segments() const { return segments_; }
  // Bumped on every change of the segment structure (not on rewrites).
  uint64_t version() const { return version_; }

  Segment* find(int32_t unit, int32_t kind);
  const Segment* find(int32_t unit, int32_t kind) const;

  // Creates (unit, kind) with n_tokens on fresh pages, or validates a rewrite
  // of an existing uncommitted segment.  *created tells which happened.
  PtStatus acquire(int32_t unit, int32_t kind, int32_t n_tokens, Segment** seg, bool* created);
  void commit(int32_t unit);                         // VIDEO and AUDIO segments of unit
  int32_t evict_before(int32_t unit);                // returns freed segment count
  PtStatus release(int32_t unit, int32_t kind);
  void reset();

  // Pages visible to a query set of mask.q_unit, in segment creation order.
  void visible_pages(const MaskSpec& mask, std::vector<PageRef>* out) const;
  // The same list, appended to *out (for the concatenated lists of a call
  // whose queries belong to several units).
  void visible_pages_append(const MaskSpec& mask, std::vector<PageRef>* out) const;
  static bool segment_visible(const Segment& s, const MaskSpec& mask);

 private:
  void free_segment_pages(const Segment& s);

  int32_t page_tokens_;
  int32_t max_pages_;
  int32_t n_free_;
  std::vector<uint8_t> used_;
  std::vector<Segment> segments_;
  uint64_t serial_ = 0;
  uint64_t version_ = 1;
};

}  // namespace ws
