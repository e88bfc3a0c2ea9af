// Host-side page table of the paged K/V cache (pure C++, no HIP).
#include "pagetable.hpp"

#include <algorithm>

namespace ws {

namespace {
constexpr int32_t kKindCond = 0;
}

PageTable::PageTable(int32_t page_tokens, int32_t max_pages)
    : page_tokens_(page_tokens), max_pages_(max_pages), n_free_(max_pages),
      used_(static_cast<size_t>(max_pages), 0) {}

Segment* PageTable::find(int32_t unit, int32_t kind) {
  for (auto& s : segments_)
    if (s.unit == unit && s.kind == kind) return &s;
  return nullptr;
}

const Segment* PageTable::find(int32_t unit, int32_t kind) const {
  for (const auto& s : segments_)
    if (s.unit == unit && s.kind == kind) return &s;
  return nullptr;
}

PtStatus PageTable::acquire(int32_t unit, int32_t kind, int32_t n_tokens, Segment** seg,
                            bool* created) {
  *created = false;
  if (Segment* s = find(unit, kind)) {
    if (s->committed) return PtStatus::committed;
    if (s->n_tokens != n_tokens) return PtStatus::shape;
    *seg = s;
    return PtStatus::ok;
  }
  const int32_t need = (n_tokens + page_tokens_ - 1) / page_tokens_;
  if (need > n_free_) return PtStatus::out_of_pages;
  Segment s;
  s.unit = unit;
  s.kind = kind;
  s.n_tokens = n_tokens;
  s.serial = ++serial_;
  s.pages.reserve(static_cast<size_t>(need));
  // Lowest free page ids first: a unit's pages stay contiguous whenever a
  // same-sized unit was evicted before it, which keeps reads sequential.
  for (int32_t p = 0; p < max_pages_ && static_cast<int32_t>(s.pages.size()) < need; ++p) {
    if (!used_[static_cast<size_t>(p)]) {
      used_[static_cast<size_t>(p)] = 1;
      s.pages.push_back(p);
    }
  }
  n_free_ -= need;
  segments_.push_back(std::move(s));
  ++version_;
  *seg = &segments_.back();
  *created = true;
  return PtStatus::ok;
}

void PageTable::commit(int32_t unit) {
  for (auto& s : segments_)
    if (s.unit == unit && s.kind != kKindCond) s.committed = true;
}

void PageTable::free_segment_pages(const Segment& s) {
  for (int32_t p : s.pages) used_[static_cast<size_t>(p)] = 0;
  n_free_ += static_cast<int32_t>(s.pages.size());
}

int32_t PageTable::evict_before(int32_t unit) {
  int32_t n = 0;
  std::vector<Segment> keep;
  keep.reserve(segments_.size());
  for (auto& s : segments_) {
    if (s.kind != kKindCond && s.unit < unit) {
      free_segment_pages(s);
      ++n;
    } else {
      keep.push_back(std::move(s));
    }
  }
  segments_.swap(keep);
  if (n) ++version_;
  return n;
}

PtStatus PageTable::release(int32_t unit, int32_t kind) {
  for (size_t i = 0; i < segments_.size(); ++i) {
    if (segments_[i].unit == unit && segments_[i].kind == kind) {
      free_segment_pages(segments_[i]);
      segments_.erase(segments_.begin() + static_cast<std::ptrdiff_t>(i));
      ++version_;
      return PtStatus::ok;
    }
  }
  return PtStatus::unknown;
}

void PageTable::reset() {
  segments_.clear();
  std::fill(used_.begin(), used_.end(), 0);
  n_free_ = max_pages_;
  ++version_;
}

bool PageTable::segment_visible(const Segment& s, const MaskSpec& mask) {
  if (s.kind < 0 || s.kind > 31 || !((mask.kind_mask >> s.kind) & 1u)) return false;
  if (s.unit > mask.q_unit) return false;                       // block-causal
  if (s.kind != kKindCond && s.unit < mask.min_visible_unit) return false;  // window
  return true;
}

void PageTable::visible_pages(const MaskSpec& mask, std::vector<PageRef>* out) const {
  out->clear();
  visible_pages_append(mask, out);
}

void PageTable::visible_pages_append(const MaskSpec& mask, std::vector<PageRef>* out) const {
  for (const auto& s : segments_) {
    if (!segment_visible(s, mask)) continue;
    int32_t left = s.n_tokens;
    for (int32_t p : s.pages) {
      const int32_t n = std::min(left, page_tokens_);
      out->push_back(PageRef{p, n});
      left -= n;
    }
  }
}

}  // namespace ws
