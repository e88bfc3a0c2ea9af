// C ABI of the performer unit-attention library (declared in include/ws.h).
//
// Host responsibilities: argument validation (before anything is enqueued),
// the page table, the visible-page lists (uploaded once per change of the
// cache structure and reused by every denoising step in between), the choice
// of key-range splits, and the kernel launches.  Nothing here computes
// attention: every arithmetic step runs in kernels.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "pagetable.hpp"
#include "ws.h"
#include "ws_internal.hpp"
#include "ws_kernels.hpp"

namespace ws_internal {

namespace {
thread_local std::string g_last_error;
}  // namespace

ws_status fail(ws_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

ws_status hip_fail(hipError_t e, const char* what) {
  return fail(WS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

const char* last_error() { return g_last_error.c_str(); }

}  // namespace ws_internal

namespace {

using ws_internal::fail;
using ws_internal::hip_fail;

#define WS_HIP(call)                                  \
  do {                                                \
    hipError_t e_ = (call);                           \
    if (e_ != hipSuccess) return hip_fail(e_, #call); \
  } while (0)

using ws::kMaxVideoSplits;
// Blocks per CU of an append launch; each loops over the launch's tiles.
constexpr int kAppendBlocksPerCu = 4;
// Fewest waves without rows in the video call's last query tile (with the
// audio rows) for the video kernel to attend the audio rows' own pages.
constexpr int kRiderMinIdleWaves = 2;
// Pages per key range of the audio kernel when the step's audio rows ride in
// the video kernel and it walks only the audio-token pages (one page per
// wave: measured 1.5 us faster per step than two).
constexpr int kRiderPagesPerRange = 4;
constexpr int kMaxAudioSplits = 512;
using ws::kMaxAudioQ;

struct TimingRing {
  int32_t cap = 0;
  int32_t next = 0;   // slot of the next call
  int32_t count = 0;  // recorded calls, <= cap
  std::vector<hipEvent_t> ev;  // 3 per slot
  std::vector<ws_call_timing> meta;
};

// A call's query groups: rows of one unit each, with that unit's mask.
struct QueryGroup {
  ws::MaskSpec mask;
  int32_t n_q;
};

// A page list uploaded to the device arena: the concatenated visible lists
// of a call's query groups (one per group with rows), kept while the cache
// structure does not change.
struct ListCacheEntry {
  bool valid = false;
  int32_t n_masks = 0;
  ws::MaskSpec masks[ws::kMaxClasses]{};
  uint64_t version = 0;
  size_t offset = 0;
  int32_t n = 0;
};

bool same_mask(const ws::MaskSpec& a, const ws::MaskSpec& b) {
  return a.q_unit == b.q_unit && a.min_visible_unit == b.min_visible_unit && a.kind_mask == b.kind_mask;
}

}  // namespace

struct ws_cache {
  ws_cache_config cfg{};
  int device = 0;
  int num_cus = 256;
  ws::PageTable pt;
  uint16_t* kpool = nullptr;
  uint16_t* vpool = nullptr;
  float2* rope_dev = nullptr;
  ws::RopeTables rope{};
  uint32_t* flags_dev = nullptr;
  int2* arena_dev = nullptr;
  int2* arena_host = nullptr;  // pinned
  size_t arena_cap = 0;
  size_t arena_used = 0;
  uint64_t arena_wraps = 0;  // times the arena started over (every cached list dropped)
  ListCacheEntry lists[4];
  int list_next = 0;
  float* part_o = nullptr;    // video key-range partials
  float* part_lse = nullptr;
  float* apart_o = nullptr;   // audio key-range partials (a separate workspace, so
  float* apart_lse = nullptr; // that one step's two paths can be merged together)
  int64_t part_rows = 0;  // capacity of each workspace in (split, head, query) rows
  int32_t opt_video_splits = 0;
  int32_t opt_audio_splits = 0;
  int32_t opt_running_max = 0;
  int32_t opt_class_cus = 0;  // 0: classes share one round of the CUs, 1: each sized for all CUs
  int32_t opt_separate_audio = 0;  // 1: ws_step_attention never lets audio rows ride in the video kernel
  float* knorm2 = nullptr;  // [max_pages][H] squared key-norm maxima
  uint16_t* zeros = nullptr;  // 1 KB of zeros (direct-load source of empty blocks)
  void* static_ws = nullptr;  // device address of the static split-KV workspace on this device
  std::vector<ws::PageRef> scratch_list;
  std::vector<ws::PageRef> rider_video, rider_audio;  // the step's two visible lists (host)
  std::vector<uint8_t> page_mark;                     // per page id, all zero between calls
  TimingRing timing;

  ws_cache(int32_t page_tokens, int32_t max_pages) : pt(page_tokens, max_pages) {}
};

namespace ws_internal {

// Timing ring slot of the next call (or -1), with its first event recorded
// unless the kernel launch stamps it (stamped: the library's own kernels
// take events 0 and 1 as their dispatch's start and end).
ws_status timing_begin_path(ws_cache* c, int32_t path, int32_t splits, hipStream_t stream, int* slot,
                            bool stamped) {
  TimingRing& tr = c->timing;
  *slot = tr.cap > 0 ? tr.next : -1;
  if (*slot >= 0) {
    tr.meta[*slot] = ws_call_timing{path, splits, 0.f, 0.f};
    if (!stamped) WS_HIP(hipEventRecord(tr.ev[3 * *slot], stream));
    tr.next = (tr.next + 1) % tr.cap;
    tr.count = std::min(tr.count + 1, tr.cap);
  }
  return WS_OK;
}

ws_status timing_mark(ws_cache* c, int slot, int k, hipStream_t stream) {
  if (slot >= 0) WS_HIP(hipEventRecord(c->timing.ev[3 * slot + k], stream));
  return WS_OK;
}

// Event k of a timing slot, or nullptr when the call is not timed.
hipEvent_t timing_event(ws_cache* c, int slot, int k) { return slot >= 0 ? c->timing.ev[3 * slot + k] : nullptr; }

int32_t cache_heads(const ws_cache* c) { return c->cfg.num_heads; }
int32_t cache_max_q(const ws_cache* c) { return c->cfg.max_q_tokens; }
int32_t free_pages(const ws_cache* c) { return c->pt.free_pages(); }

ws_status precheck_append(const ws_cache* c, int32_t unit, ws_kind kind, int32_t n_tokens,
                          int32_t* pages_needed) {
  const ws::Segment* seg = c->pt.find(unit, kind);
  if (!seg) {
    *pages_needed += (n_tokens + ws::kPageTokens - 1) / ws::kPageTokens;
    if (*pages_needed > c->pt.free_pages())
      return fail(WS_ERR_OUT_OF_PAGES, "pool has %d free pages, the step needs %d", c->pt.free_pages(),
                  *pages_needed);
    return WS_OK;
  }
  if (seg->committed)
    return fail(WS_ERR_COMMITTED, "unit %d kind %d is committed history", unit, static_cast<int>(kind));
  if (seg->n_tokens != n_tokens)
    return fail(WS_ERR_SHAPE, "rewrite of unit %d kind %d with %d tokens (segment has %d)", unit,
                static_cast<int>(kind), n_tokens, seg->n_tokens);
  return WS_OK;
}

}  // namespace ws_internal

using ws_internal::timing_begin_path;
using ws_internal::timing_mark;
using ws_internal::timing_event;

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

ws_status check_device(const ws_cache* c) {
  int dev = -1;
  WS_HIP(hipGetDevice(&dev));
  if (dev != c->device)
    return fail(WS_ERR_INVALID_ARG, "cache lives on device %d but device %d is current", c->device,
                dev);
  return WS_OK;
}

ws_status check_kind(int kind) {
  if (kind < WS_KIND_COND || kind > WS_KIND_AUDIO) return fail(WS_ERR_INVALID_ARG, "bad kind %d", kind);
  return WS_OK;
}

ws_status check_strides(const char* what, const void* p, int64_t tok_stride, int64_t head_stride,
                        int32_t n_tok, int32_t n_heads) {
  if (!p) return fail(WS_ERR_INVALID_ARG, "%s is NULL", what);
  if (!aligned16(p)) return fail(WS_ERR_INVALID_ARG, "%s is not 16-byte aligned", what);
  if (tok_stride < 0 || head_stride < 0 || tok_stride % 8 || head_stride % 8)
    return fail(WS_ERR_INVALID_ARG, "%s strides must be non-negative multiples of 8 elements", what);
  if (n_tok > 1 && tok_stride < ws::kHeadDim)
    return fail(WS_ERR_INVALID_ARG, "%s token stride %lld overlaps a head row", what,
                static_cast<long long>(tok_stride));
  if (n_heads > 1 && head_stride < ws::kHeadDim)
    return fail(WS_ERR_INVALID_ARG, "%s head stride %lld overlaps a head row", what,
                static_cast<long long>(head_stride));
  // the kernels index with 32-bit token offsets times a 64-bit stride
  const long double span = static_cast<long double>(tok_stride) * n_tok +
                           static_cast<long double>(head_stride) * n_heads;
  if (span > 9.0e18L) return fail(WS_ERR_INVALID_ARG, "%s strides overflow", what);
  return WS_OK;
}

// Uploads a page list into the device arena (async, on `stream`) and returns
// its element offset.  A full arena wraps after waiting for the device.
ws_status upload_list(ws_cache* c, const std::vector<ws::PageRef>& list, hipStream_t stream,
                      size_t* offset) {
  const size_t n = std::max<size_t>(list.size(), 1);
  if (n > c->arena_cap) return fail(WS_ERR_SHAPE, "page list of %zu entries exceeds arena", n);
  if (c->arena_used + n > c->arena_cap) {
    WS_HIP(hipDeviceSynchronize());
    c->arena_used = 0;
    ++c->arena_wraps;
    for (auto& e : c->lists) e.valid = false;
  }
  const size_t off = c->arena_used;
  for (size_t i = 0; i < list.size(); ++i)
    c->arena_host[off + i] = make_int2(list[i].page, list[i].n_valid);
  if (list.empty()) c->arena_host[off] = make_int2(0, 0);
  WS_HIP(hipMemcpyAsync(c->arena_dev + off, c->arena_host + off, n * sizeof(int2),
                        hipMemcpyHostToDevice, stream));
  c->arena_used += (n + 63) & ~size_t(63);
  if (c->arena_used > c->arena_cap) c->arena_used = c->arena_cap;
  *offset = off;
  return WS_OK;
}

// The concatenated visible page lists of masks[0..n_masks) (c->scratch_list
// holds them, built by the caller) in the device arena: reused while the
// cache structure and the masks are unchanged, else uploaded once.
ws_status arena_list(ws_cache* c, const ws::MaskSpec* masks, int n_masks, hipStream_t stream,
                     const int2** dev) {
  const uint64_t ver = c->pt.version();
  for (auto& e : c->lists) {
    if (!e.valid || e.version != ver || e.n_masks != n_masks) continue;
    bool same = true;
    for (int i = 0; i < n_masks && same; ++i) same = same_mask(e.masks[i], masks[i]);
    if (same) {
      *dev = c->arena_dev + e.offset;
      return WS_OK;
    }
  }
  size_t off = 0;
  ws_status st = upload_list(c, c->scratch_list, stream, &off);
  if (st != WS_OK) return st;
  ListCacheEntry& e = c->lists[c->list_next];
  c->list_next = (c->list_next + 1) % 4;
  e.valid = true;
  e.n_masks = n_masks;
  for (int i = 0; i < n_masks; ++i) e.masks[i] = masks[i];
  e.version = ver;
  e.offset = off;
  e.n = static_cast<int32_t>(c->scratch_list.size());
  *dev = c->arena_dev + off;
  return WS_OK;
}

ws_status fill_rope(ws_cache* c) {
  const ws_cache_config& g = c->cfg;
  size_t total = 0;
  for (int b = 0; b < 3; ++b) total += static_cast<size_t>(g.rope_max_pos[b]) * g.rope_pairs[b];
  std::vector<float2> host(std::max<size_t>(total, 1));
  size_t off[3];
  size_t o = 0;
  for (int b = 0; b < 3; ++b) {
    off[b] = o;
    const int np = g.rope_pairs[b];
    for (int pos = 0; pos < g.rope_max_pos[b]; ++pos)
      for (int pb = 0; pb < np; ++pb) {
        // angle in double precision, rounded once to fp32 per cos/sin
        const double ang = static_cast<double>(pos) *
                           std::pow(g.rope_theta, -static_cast<double>(pb) / static_cast<double>(np));
        host[o++] = make_float2(static_cast<float>(std::cos(ang)), static_cast<float>(std::sin(ang)));
      }
  }
  WS_HIP(hipMalloc(&c->rope_dev, host.size() * sizeof(float2)));
  WS_HIP(hipMemcpy(c->rope_dev, host.data(), host.size() * sizeof(float2), hipMemcpyHostToDevice));
  for (int b = 0; b < 3; ++b) {
    c->rope.tab[b] = c->rope_dev + off[b];
    c->rope.max_pos[b] = g.rope_max_pos[b];
    c->rope.pairs[b] = g.rope_pairs[b];
  }
  return WS_OK;
}

void timing_free(ws_cache* c) {
  for (hipEvent_t e : c->timing.ev) (void)hipEventDestroy(e);
  c->timing = TimingRing{};
}

void free_all(ws_cache* c) {
  timing_free(c);
  if (c->kpool) (void)hipFree(c->kpool);
  if (c->vpool) (void)hipFree(c->vpool);
  if (c->rope_dev) (void)hipFree(c->rope_dev);
  if (c->flags_dev) (void)hipFree(c->flags_dev);
  if (c->arena_dev) (void)hipFree(c->arena_dev);
  if (c->arena_host) (void)hipHostFree(c->arena_host);
  if (c->part_o) (void)hipFree(c->part_o);
  if (c->part_lse) (void)hipFree(c->part_lse);
  if (c->apart_o) (void)hipFree(c->apart_o);
  if (c->apart_lse) (void)hipFree(c->apart_lse);
  if (c->knorm2) (void)hipFree(c->knorm2);
  if (c->zeros) (void)hipFree(c->zeros);
  c->knorm2 = nullptr;
  c->zeros = nullptr;
  c->kpool = c->vpool = nullptr;
  c->rope_dev = nullptr;
  c->flags_dev = nullptr;
  c->arena_dev = c->arena_host = nullptr;
  c->part_o = c->part_lse = c->apart_o = c->apart_lse = nullptr;
}

ws_status create_impl(const ws_cache_config* cfg, ws_cache** out) {
  if (!cfg || !out) return fail(WS_ERR_INVALID_ARG, "NULL argument");
  *out = nullptr;
  if (cfg->head_dim != ws::kHeadDim)
    return fail(WS_ERR_UNSUPPORTED, "head_dim %d unsupported (only 128)", cfg->head_dim);
  if (cfg->page_tokens != ws::kPageTokens)
    return fail(WS_ERR_UNSUPPORTED, "page_tokens %d unsupported (only 64)", cfg->page_tokens);
  if (cfg->num_heads < 1 || cfg->num_heads > 4096)
    return fail(WS_ERR_SHAPE, "num_heads %d out of range [1, 4096]", cfg->num_heads);
  if (cfg->max_pages < 1 || cfg->max_q_tokens < 1 || cfg->max_q_tokens > (1 << 20))
    return fail(WS_ERR_SHAPE, "max_pages and max_q_tokens must be >= 1 (max_q_tokens <= 2^20)");
  int pair_sum = 0;
  for (int b = 0; b < 3; ++b) {
    if (cfg->rope_max_pos[b] < 1 || cfg->rope_max_pos[b] > (1 << 24))
      return fail(WS_ERR_SHAPE, "rope_max_pos[%d] = %d out of range", b, cfg->rope_max_pos[b]);
    if (cfg->rope_pairs[b] < 0) return fail(WS_ERR_SHAPE, "rope_pairs[%d] negative", b);
    pair_sum += cfg->rope_pairs[b];
  }
  if (pair_sum != ws::kHeadDim / 2)
    return fail(WS_ERR_SHAPE, "rope_pairs sum to %d, need %d", pair_sum, ws::kHeadDim / 2);
  if (!(cfg->rope_theta > 1.0) || !std::isfinite(cfg->rope_theta))
    return fail(WS_ERR_INVALID_ARG, "rope_theta must be a finite value > 1");

  ws_cache* c = new ws_cache(cfg->page_tokens, cfg->max_pages);
  c->cfg = *cfg;
  auto bail = [&](ws_status st) {
    free_all(c);
    delete c;
    return st;
  };
  hipError_t e = hipGetDevice(&c->device);
  if (e != hipSuccess) return bail(hip_fail(e, "hipGetDevice"));
  e = hipDeviceGetAttribute(&c->num_cus, hipDeviceAttributeMultiprocessorCount, c->device);
  if (e != hipSuccess) return bail(hip_fail(e, "hipDeviceGetAttribute"));

  const size_t pool_elems =
      static_cast<size_t>(cfg->max_pages) * cfg->num_heads * static_cast<size_t>(ws::kPageHeadElems);
  if ((e = hipMalloc(&c->kpool, pool_elems * 2)) != hipSuccess) return bail(hip_fail(e, "hipMalloc(K pool)"));
  if ((e = hipMalloc(&c->vpool, pool_elems * 2)) != hipSuccess) return bail(hip_fail(e, "hipMalloc(V pool)"));
  if ((e = hipMemset(c->kpool, 0, pool_elems * 2)) != hipSuccess) return bail(hip_fail(e, "hipMemset"));
  if ((e = hipMemset(c->vpool, 0, pool_elems * 2)) != hipSuccess) return bail(hip_fail(e, "hipMemset"));
  const size_t norm_elems = static_cast<size_t>(cfg->max_pages) * cfg->num_heads;
  if ((e = hipMalloc(&c->knorm2, norm_elems * sizeof(float))) != hipSuccess)
    return bail(hip_fail(e, "hipMalloc(key norms)"));
  if ((e = hipMemset(c->knorm2, 0, norm_elems * sizeof(float))) != hipSuccess)
    return bail(hip_fail(e, "hipMemset"));
  if ((e = hipMalloc(&c->zeros, 1024)) != hipSuccess) return bail(hip_fail(e, "hipMalloc(zeros)"));
  if ((e = hipMemset(c->zeros, 0, 1024)) != hipSuccess) return bail(hip_fail(e, "hipMemset"));
  if (ws_status st = fill_rope(c); st != WS_OK) return bail(st);
  if ((e = ws::static_scratch(&c->static_ws)) != hipSuccess)
    return bail(hip_fail(e, "hipGetSymbolAddress(static split-KV workspace)"));
  if ((e = hipMalloc(&c->flags_dev, sizeof(uint32_t))) != hipSuccess) return bail(hip_fail(e, "hipMalloc"));
  if ((e = hipMemset(c->flags_dev, 0, sizeof(uint32_t))) != hipSuccess) return bail(hip_fail(e, "hipMemset"));
  c->arena_cap = std::max<size_t>(65536, 16 * static_cast<size_t>(cfg->max_pages));
  if ((e = hipMalloc(&c->arena_dev, c->arena_cap * sizeof(int2))) != hipSuccess)
    return bail(hip_fail(e, "hipMalloc(arena)"));
  if ((e = hipHostMalloc(reinterpret_cast<void**>(&c->arena_host), c->arena_cap * sizeof(int2),
                         hipHostMallocDefault)) != hipSuccess)
    return bail(hip_fail(e, "hipHostMalloc(arena)"));
  c->part_rows = static_cast<int64_t>(kMaxVideoSplits) * cfg->num_heads *
                 std::max<int64_t>(cfg->max_q_tokens, kMaxAudioQ);
  if ((e = hipMalloc(&c->part_o, static_cast<size_t>(c->part_rows) * ws::kHeadDim * sizeof(float))) != hipSuccess)
    return bail(hip_fail(e, "hipMalloc(partials)"));
  if ((e = hipMalloc(&c->part_lse, static_cast<size_t>(c->part_rows) * sizeof(float))) != hipSuccess)
    return bail(hip_fail(e, "hipMalloc(partials)"));
  if ((e = hipMalloc(&c->apart_o, static_cast<size_t>(c->part_rows) * ws::kHeadDim * sizeof(float))) != hipSuccess)
    return bail(hip_fail(e, "hipMalloc(partials)"));
  if ((e = hipMalloc(&c->apart_lse, static_cast<size_t>(c->part_rows) * sizeof(float))) != hipSuccess)
    return bail(hip_fail(e, "hipMalloc(partials)"));
  *out = c;
  return WS_OK;
}

// Number of workgroup groups of the video kernel (a group is one workgroup
// per query tile; together the groups share the (head, page) units evenly;
// one round of groups fits the CUs when groups * n_qtiles <= CUs): the cost
// model of ws::video_group_count.  A forced split count s gives H * s
// groups: every head in s equal key ranges.
// Partition cost of starting a head's segment inside a workgroup's share, in
// pages: the segment switch (epilogue stores, query load, key-norm bound,
// pipeline refill) takes about as long as six pages of the main loop.
constexpr int kVideoSegCostPages = 6;

int choose_video_groups(const ws_cache* c, int n_heads, int n_qtiles, int n_pages, int n_cus) {
  if (n_pages == 0) return n_heads;
  if (c->opt_video_splits > 0) return n_heads * c->opt_video_splits;
  return static_cast<int>(ws::video_group_count(n_heads, n_qtiles, n_pages, n_cus));
}

int choose_audio_splits(const ws_cache* c, int n_items, int n_pages) {
  if (c->opt_audio_splits > 0) return c->opt_audio_splits;
  // Two 4-wave workgroups per CU (8 streaming waves): as many key ranges as
  // fill the CUs once, each wave keeping at least one page.
  const int target = std::max(1, 2 * c->num_cus / std::max(n_items, 1));
  return std::max(1, std::min({target, std::max(1, n_pages / 4), kMaxAudioSplits}));
}

// The logit scale times log2(e), folded into Q'' (0 selects 1/sqrt(128)).
float scale_log2_of(float softmax_scale) {
  const double scale = softmax_scale > 0.f ? static_cast<double>(softmax_scale)
                                           : 1.0 / std::sqrt(static_cast<double>(ws::kHeadDim));
  return static_cast<float>(scale * 1.4426950408889634);
}

// One attention call, validated and resolved into launch arguments.
struct AttnPlan {
  bool audio = false;
  ws::AttnArgs a{};
  bool merge = false;
  ws::CombineArgs cb{};
  int splits = 1;  // audio: key ranges; video: workgroup groups
  int64_t part_rows = 0;  // (range, head, query) partial rows the kernel may write
};

ws_status plan_attention(bool audio, const void* q, int64_t q_tok_stride, int64_t q_head_stride,
                         int32_t n_groups, const QueryGroup* groups, const ws_query_desc* qd, ws_cache* c,
                         void* out, int64_t out_tok_stride, int64_t out_head_stride,
                         hipStream_t stream, AttnPlan* plan) {
  if (!c || !qd || !groups) return fail(WS_ERR_INVALID_ARG, "NULL argument");
  if (ws_status st = check_device(c); st != WS_OK) return st;
  if (n_groups < 1 || n_groups > (audio ? 1 : ws::kMaxClasses))
    return fail(WS_ERR_INVALID_ARG, "query group count %d outside [1, %d]", n_groups, audio ? 1 : ws::kMaxClasses);
  int32_t n_q = 0;
  for (int g = 0; g < n_groups; ++g) {
    if (groups[g].n_q < 0) return fail(WS_ERR_SHAPE, "query group %d has a negative row count", g);
    n_q += groups[g].n_q;
  }
  const int H = c->cfg.num_heads;
  const int max_q = audio ? std::min(c->cfg.max_q_tokens, kMaxAudioQ) : c->cfg.max_q_tokens;
  if (n_q < 1 || n_q > max_q) return fail(WS_ERR_SHAPE, "n_q %d out of range [1, %d]", n_q, max_q);
  if (ws_status st = check_strides("q", q, q_tok_stride, q_head_stride, n_q, H); st != WS_OK) return st;
  if (ws_status st = check_strides("out", out, out_tok_stride, out_head_stride, n_q, H); st != WS_OK)
    return st;
  if (qd->mode != WS_APPEND_RAW && qd->mode != WS_APPEND_NORM_ROPE && qd->mode != WS_QUERY_PREPARED)
    return fail(WS_ERR_INVALID_ARG, "bad query mode %d", static_cast<int>(qd->mode));
  if (qd->mode == WS_APPEND_NORM_ROPE) {
    if (!qd->positions || !qd->gamma) return fail(WS_ERR_INVALID_ARG, "NORM_ROPE needs positions and gamma");
    if (!aligned16(qd->gamma)) return fail(WS_ERR_INVALID_ARG, "gamma is not 16-byte aligned");
    if (!(qd->eps >= 0.f) || !std::isfinite(qd->eps)) return fail(WS_ERR_INVALID_ARG, "bad eps");
  }
  if (!std::isfinite(qd->softmax_scale) || qd->softmax_scale < 0.f)
    return fail(WS_ERR_INVALID_ARG, "bad softmax_scale");

  // Each group with rows is a query class with its own visible page list;
  // the lists are concatenated.  The whole list goes into the kernel
  // arguments when it fits, else into the device arena (one upload per
  // distinct list).
  plan->audio = audio;
  ws::AttnArgs& a = plan->a;
  a = ws::AttnArgs{};
  const int2* plist = nullptr;
  ws::MaskSpec masks[ws::kMaxClasses];
  int n_cls = 0;
  c->scratch_list.clear();
  for (int g = 0, r0 = 0; g < n_groups; r0 += groups[g].n_q, ++g) {
    if (groups[g].n_q == 0) continue;
    ws::AttnClass& cl = a.cls[n_cls];
    masks[n_cls++] = groups[g].mask;
    cl.q0 = r0;
    cl.n_q = groups[g].n_q;
    cl.page0 = static_cast<int32_t>(c->scratch_list.size());
    c->pt.visible_pages_append(groups[g].mask, &c->scratch_list);
    cl.n_pages = static_cast<int32_t>(c->scratch_list.size()) - cl.page0;
  }
  const int32_t n_pages = static_cast<int32_t>(c->scratch_list.size());
  if (n_pages <= ws::AttnArgs::kInlinePages) {
    for (int32_t i = 0; i < n_pages; ++i)
      a.inline_pages[i] = make_int2(c->scratch_list[static_cast<size_t>(i)].page,
                                    c->scratch_list[static_cast<size_t>(i)].n_valid);
  } else if (ws_status st = arena_list(c, masks, n_cls, stream, &plist); st != WS_OK) {
    return st;
  }
  a.n_classes = n_cls;
  a.q = static_cast<const uint16_t*>(q);
  a.q_tok_stride = q_tok_stride;
  a.q_head_stride = q_head_stride;
  a.n_q = n_q;
  a.num_heads = H;
  a.mode = static_cast<int32_t>(qd->mode);
  a.positions = qd->positions;
  a.gamma = qd->gamma;
  a.eps = qd->eps;
  a.scale_log2 = scale_log2_of(qd->softmax_scale);
  a.rope = c->rope;
  a.kpool = c->kpool;
  a.vpool = c->vpool;
  a.knorm2 = c->knorm2;
  a.zeros = c->zeros;
  a.fixed_shift = c->opt_running_max ? 0 : 1;
  a.pages = plist;
  a.n_pages = n_pages;
  a.out = static_cast<uint16_t*>(out);
  a.out_tok_stride = out_tok_stride;
  a.out_head_stride = out_head_stride;
  a.part_o = audio ? c->apart_o : c->part_o;
  a.part_lse = audio ? c->apart_lse : c->part_lse;
  a.flags = c->flags_dev;
  const int qtile = audio ? ws::kAudioQTile : ws::kVideoQTile;
  a.n_qtiles = (n_q + qtile - 1) / qtile;
  const int n_items = a.n_qtiles * H;
  const int64_t cap = c->part_rows / (static_cast<int64_t>(H) * n_q);
  int splits = 1;         // audio: key ranges; video: workgroup groups
  bool merge = audio;
  if (audio) {
    splits = choose_audio_splits(c, n_items, n_pages);
    splits = std::max(1, std::min(splits, std::max(1, n_pages)));
    splits = static_cast<int>(std::min<int64_t>(splits, std::max<int64_t>(cap, 1)));
    const int pps = n_pages > 0 ? (n_pages + splits - 1) / splits : 0;
    splits = pps > 0 ? (n_pages + pps - 1) / pps : 1;  // no empty splits
    if (cap < splits) return fail(WS_ERR_SHAPE, "split-KV workspace too small");
    a.n_splits = splits;
    a.pages_per_split = pps;
    plan->part_rows = static_cast<int64_t>(splits) * H * n_q;
  } else {
    // Per class: query tiles, and groups of workgroups sharing the class's
    // (head, page) units.  The classes share one round of the CUs in
    // proportion to their work (a catch-up of three 920-query units over
    // 8536 keys each, measured with the clocks settled: 480 us, against 500
    // us when every class is partitioned as if it had all CUs and the
    // launch runs several rounds of workgroups; the option selects the
    // latter).
    int64_t work = 0;
    for (int k = 0; k < n_cls; ++k) {
      a.cls[k].n_qtiles = (a.cls[k].n_q + ws::kVideoQTile - 1) / ws::kVideoQTile;
      work += static_cast<int64_t>(a.cls[k].n_qtiles) * a.cls[k].n_pages;
    }
    int64_t max_ranges = 1;
    int32_t wg = 0, total_groups = 0;
    merge = false;
    for (int k = 0; k < n_cls; ++k) {
      ws::AttnClass& cl = a.cls[k];
      const int64_t w = static_cast<int64_t>(cl.n_qtiles) * cl.n_pages;
      const int cus = c->opt_class_cus == 1 || n_cls == 1 || work == 0
                          ? c->num_cus
                          : static_cast<int>(std::max<int64_t>(cl.n_qtiles, c->num_cus * w / work));
      cl.n_groups = choose_video_groups(c, H, cl.n_qtiles, cl.n_pages, cus);
      cl.wg0 = wg;
      wg += cl.n_groups * cl.n_qtiles;
      total_groups += cl.n_groups;
      // ranges per head: exactly the forced split count, else at most
      // ceil(groups / H) + 1 (a share of at most one head's pages meets at
      // most two heads); a single range writes bf16 directly, and no head
      // is split when the group count divides H
      if (cl.n_pages > 0 && ws::video_heads_split(H, cl.n_groups)) {
        merge = true;
        max_ranges = std::max<int64_t>(max_ranges, c->opt_video_splits > 0
                                                       ? c->opt_video_splits
                                                       : std::max(2, (cl.n_groups + H - 1) / H + 1));
      }
    }
    if (cap < max_ranges) return fail(WS_ERR_SHAPE, "split-KV workspace too small");
    plan->part_rows = max_ranges * H * n_q;
    a.n_groups = total_groups;
    a.n_wg = wg;
    a.n_qtiles = 0;
    for (int k = 0; k < n_cls; ++k) a.n_qtiles += a.cls[k].n_qtiles;
    // forced splits keep equal ranges per head
    a.seg_cost = c->opt_video_splits > 0 ? 0 : kVideoSegCostPages;
    a.n_splits = 1;
    splits = total_groups;
  }

  plan->splits = splits;
  plan->merge = merge;
  if (merge) {
    ws::CombineArgs& cb = plan->cb;
    cb = ws::CombineArgs{};
    cb.part_o = a.part_o;
    cb.part_lse = a.part_lse;
    cb.n_splits = audio ? splits : kMaxVideoSplits;
    cb.n_groups = audio ? 0 : splits;
    cb.n_classes = audio ? 0 : a.n_classes;
    if (!audio)
      for (int k = 0; k < a.n_classes; ++k) cb.cls[k] = a.cls[k];
    cb.seg_cost = a.seg_cost;
    cb.n_q = n_q;
    cb.num_heads = H;
    cb.out = a.out;
    cb.out_tok_stride = out_tok_stride;
    cb.out_head_stride = out_head_stride;
  }
  return WS_OK;
}

hipError_t launch_plan_kernel(const AttnPlan& p, hipStream_t stream, hipEvent_t start = nullptr,
                              hipEvent_t stop = nullptr) {
  return p.audio ? ws::launch_audio_attention(p.a, stream, start, stop)
                 : ws::launch_unit_attention(p.a, stream, start, stop);
}


// A timed attention call: events 0 and 1 are the kernel's own dispatch
// timestamps (see launch_plan_kernel), event 2 follows the merge.
ws_status timing_begin(ws_cache* c, const AttnPlan& p, hipStream_t stream, int* slot) {
  return timing_begin_path(c, p.audio ? 1 : 0, p.splits, stream, slot, true);
}


ws_status attention_impl(bool audio, const void* q, int64_t q_tok_stride, int64_t q_head_stride,
                         int32_t n_groups, const QueryGroup* groups, const ws_query_desc* qd, ws_cache* c,
                         void* out, int64_t out_tok_stride, int64_t out_head_stride,
                         void* hip_stream) {
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  AttnPlan p;
  if (ws_status st = plan_attention(audio, q, q_tok_stride, q_head_stride, n_groups, groups, qd, c, out,
                                    out_tok_stride, out_head_stride, stream, &p);
      st != WS_OK)
    return st;
  int slot = -1;
  if (ws_status st = timing_begin(c, p, stream, &slot); st != WS_OK) return st;
  hipError_t e = launch_plan_kernel(p, stream, timing_event(c, slot, 0), timing_event(c, slot, 1));
  if (e != hipSuccess) return hip_fail(e, audio ? "audio_attn launch" : "unit_attn launch");
  if (p.merge) {
    e = ws::launch_combine(p.cb, stream);
    if (e != hipSuccess) return hip_fail(e, "combine launch");
  }
  return timing_mark(c, slot, 2, stream);
}

// Puts both calls' split-KV partials into the static workspace: video bf16
// O rows, audio fp32 O rows, and their fp32 log-sum-exp, each region
// 256-byte aligned.  Fails (before anything is enqueued) when they do not fit.
ws_status use_static_workspace(ws_cache* c, AttnPlan& pv, AttnPlan& pa) {
  if (!c->static_ws) return fail(WS_ERR_HIP, "static split-KV workspace unavailable");
  uint8_t* base = static_cast<uint8_t*>(c->static_ws);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    uint8_t* p = base + off;
    off += (bytes + 255) & ~size_t(255);
    return p;
  };
  const size_t rv = static_cast<size_t>(pv.part_rows), ra = static_cast<size_t>(pa.part_rows);
  float* vo = reinterpret_cast<float*>(take(rv * ws::kHeadDim * sizeof(uint16_t)));
  float* vl = reinterpret_cast<float*>(take(rv * sizeof(float)));
  float* ao = reinterpret_cast<float*>(take(ra * ws::kHeadDim * sizeof(float)));
  float* al = reinterpret_cast<float*>(take(ra * sizeof(float)));
  if (off > ws::kStaticScratchBytes)
    return fail(WS_ERR_SHAPE,
                "this step needs %zu bytes of split-KV workspace (%zu video and %zu audio partial rows); "
                "the static workspace holds %zu",
                off, rv, ra, ws::kStaticScratchBytes);
  pv.a.part_o = vo;
  pv.a.part_lse = vl;
  pa.a.part_o = ao;
  pa.a.part_lse = al;
  pv.cb.part_o = vo;
  pv.cb.part_lse = vl;
  pa.cb.part_o = ao;
  pa.cb.part_lse = al;
  return WS_OK;
}

// Audio rows riding in the video kernel.  The audio queries of a step see
// the pages the video queries see plus the unit's audio pages (Sec. 3: both
// latent streams of a unit attend over the same cache; the audio tokens are
// visible to audio queries only).  When the audio call's visible pages
// include every page of the video call's, its queries come prepared (Q''),
// and the spare rows of the video call's last 256-row query tile hold them,
// the video kernel computes the audio rows over the shared pages while it
// streams those pages for the video rows, and the audio kernel walks only
// the pages the video call does not see.  The merge then folds, per (head,
// row), the audio kernel's ranges and the ranges the video kernel wrote.
// Fills the fused plans and *rider_ranges (the most video ranges of a head);
// false (plans untouched) when the step does not qualify.
bool plan_riders(ws_cache* c, const ws_attn_call* video, const ws_attn_call* audio, AttnPlan& pv, AttnPlan& pa,
                 int* rider_ranges) {
  if (c->opt_separate_audio || audio->desc.mode != WS_QUERY_PREPARED) return false;
  if (pv.a.n_classes != 1 || pv.a.cls[0].n_pages == 0) return false;
  const ws::AttnClass& cl = pv.a.cls[0];
  const int H = c->cfg.num_heads;
  const int n_rq = audio->n_q;
  const int rq_row0 = video->n_q;
  if (rq_row0 + n_rq > cl.n_qtiles * ws::kVideoQTile) return false;
  // the audio call's pages that the video call does not see; every video
  // page must be among the audio call's
  c->pt.visible_pages(ws::MaskSpec{video->mask.q_unit, video->mask.min_visible_unit, video->mask.kind_mask},
                      &c->rider_video);
  c->pt.visible_pages(ws::MaskSpec{audio->mask.q_unit, audio->mask.min_visible_unit, audio->mask.kind_mask},
                      &c->rider_audio);
  std::vector<uint8_t>& mark = c->page_mark;
  if (mark.size() != static_cast<size_t>(c->cfg.max_pages)) mark.assign(static_cast<size_t>(c->cfg.max_pages), 0);
  for (const ws::PageRef& r : c->rider_video) mark[static_cast<size_t>(r.page)] = 1;
  size_t shared = 0;
  c->scratch_list.clear();
  for (const ws::PageRef& r : c->rider_audio) {
    if (mark[static_cast<size_t>(r.page)] == 1) {
      mark[static_cast<size_t>(r.page)] = 2;
      ++shared;
    } else {
      c->scratch_list.push_back(r);
    }
  }
  for (const ws::PageRef& r : c->rider_video) mark[static_cast<size_t>(r.page)] = 0;
  const int32_t n_extra = static_cast<int32_t>(c->scratch_list.size());
  if (shared != c->rider_video.size() || n_extra > ws::AttnArgs::kInlinePages) return false;
  // key ranges: the audio kernel's over the extra pages, then the video
  // kernel's (at most rmax per head)
  const ws::VideoPartition part{H, cl.n_pages, pv.a.seg_cost, cl.n_groups};
  int rmax = 1;
  for (int64_t h = 0; h < H; ++h) {
    const int64_t h0 = h * cl.n_pages;
    rmax = std::max(rmax, static_cast<int>(ws::video_group_of(part, h0 + cl.n_pages - 1) -
                                           ws::video_group_of(part, h0) + 1));
  }
  // The rows' own pages go to the video kernel when its last query tile
  // leaves at least kRiderMinIdleWaves waves without rows (they attend the
  // pages while the others start their first segment) and the page list
  // stays inline; otherwise to the audio kernel.
  const int last_rows = rq_row0 + n_rq - (cl.n_qtiles - 1) * ws::kVideoQTile;
  const int idle_waves = ws::kVideoWaves - (last_rows + 31) / 32;
  const bool in_video = n_extra > 0 && c->opt_audio_splits == 0 && pv.a.pages == nullptr &&
                        idle_waves >= kRiderMinIdleWaves &&
                        pv.a.n_pages + n_extra <= ws::AttnArgs::kInlinePages;
  const int rx_waves = in_video ? std::min(idle_waves, n_extra) : 0;
  int splits = 0, pps = 0;
  if (n_extra > 0 && !in_video) {
    // few pages (latency-bound): as many ranges as give each wave of the
    // audio kernel at most kRiderPagesPerRange / 4 pages
    splits = c->opt_audio_splits > 0 ? c->opt_audio_splits
                                     : (n_extra + kRiderPagesPerRange - 1) / kRiderPagesPerRange;
    splits = std::max(1, std::min(splits, n_extra));
    pps = (n_extra + splits - 1) / splits;
    splits = (n_extra + pps - 1) / pps;
  }
  const int ranges = splits + rmax + rx_waves;
  if (static_cast<int64_t>(ranges) * H * n_rq > c->part_rows) return false;

  ws::AttnArgs& aa = pa.a;
  for (int32_t i = 0; i < n_extra; ++i)
    aa.inline_pages[i] = make_int2(c->scratch_list[static_cast<size_t>(i)].page,
                                   c->scratch_list[static_cast<size_t>(i)].n_valid);
  aa.pages = nullptr;
  aa.n_pages = n_extra;
  aa.n_splits = std::max(splits, 1);
  aa.pages_per_split = pps;
  pa.splits = splits;
  pa.part_rows = static_cast<int64_t>(ranges) * H * n_rq;
  pa.merge = true;
  pa.cb.n_splits = splits;
  pa.cb.r_pages = cl.n_pages;
  pa.cb.r_groups = cl.n_groups;
  pa.cb.seg_cost = pv.a.seg_cost;
  pa.cb.r_extra = rx_waves;
  ws::AttnArgs& av = pv.a;
  if (in_video) {
    av.rx_page0 = pv.a.n_pages;
    av.rx_pages = n_extra;
    av.rx_waves = rx_waves;
    for (int32_t i = 0; i < n_extra; ++i)
      av.inline_pages[av.rx_page0 + i] = make_int2(c->scratch_list[static_cast<size_t>(i)].page,
                                                   c->scratch_list[static_cast<size_t>(i)].n_valid);
  }
  av.rq = static_cast<const uint16_t*>(audio->q);
  av.rq_tok_stride = audio->q_tok_stride;
  av.rq_head_stride = audio->q_head_stride;
  av.n_rq = n_rq;
  av.rq_row0 = rq_row0;
  *rider_ranges = rmax;
  return true;
}

ws_status step_attention_impl(ws_cache* c, const ws_attn_call* video, const ws_attn_call* audio,
                              void* hip_stream, bool static_workspace) {
  if (!c || !video || !audio) return fail(WS_ERR_INVALID_ARG, "NULL argument");
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  AttnPlan pv, pa;
  const QueryGroup gv{ws::MaskSpec{video->mask.q_unit, video->mask.min_visible_unit, video->mask.kind_mask},
                      video->n_q};
  const QueryGroup ga{ws::MaskSpec{audio->mask.q_unit, audio->mask.min_visible_unit, audio->mask.kind_mask},
                      audio->n_q};
  auto plan_video = [&]() {
    return plan_attention(false, video->q, video->q_tok_stride, video->q_head_stride, 1, &gv, &video->desc, c,
                          video->out, video->out_tok_stride, video->out_head_stride, stream, &pv);
  };
  if (ws_status st = plan_video(); st != WS_OK) return st;
  const uint64_t wraps = c->arena_wraps;
  if (ws_status st = plan_attention(true, audio->q, audio->q_tok_stride, audio->q_head_stride, 1, &ga,
                                    &audio->desc, c, audio->out, audio->out_tok_stride, audio->out_head_stride,
                                    stream, &pa);
      st != WS_OK)
    return st;
  // A page list uploaded by the audio plan that started the arena over may
  // sit where the video plan's list was: plan the video call again (its list
  // then goes in after the audio one; the arena holds at least 16 lists of
  // the longest possible length, so it cannot start over a second time).
  if (c->arena_wraps != wraps) {
    if (ws_status st = plan_video(); st != WS_OK) return st;
    if (c->arena_wraps != wraps + 1) return fail(WS_ERR_SHAPE, "page-list arena too small for one step");
  }
  int rider_ranges = 0;
  const bool riders = plan_riders(c, video, audio, pv, pa, &rider_ranges);
  if (static_workspace)
    if (ws_status st = use_static_workspace(c, pv, pa); st != WS_OK) return st;
  if (riders) {  // the video kernel's ranges of the audio rows follow the audio kernel's
    const int64_t off = static_cast<int64_t>(pa.splits) * c->cfg.num_heads * audio->n_q;
    pv.a.rpart_o = pa.a.part_o + off * ws::kHeadDim;
    pv.a.rpart_lse = pa.a.part_lse + off;
  }
  // video kernel, audio kernel (over the extra pages only when the audio
  // rows ride in the video kernel), then one launch merging both
  int sv = -1, sa = -1;
  if (ws_status st = timing_begin(c, pv, stream, &sv); st != WS_OK) return st;
  hipError_t e = launch_plan_kernel(pv, stream, timing_event(c, sv, 0), timing_event(c, sv, 1));
  if (e != hipSuccess) return hip_fail(e, "unit_attn launch");
  if (ws_status st = timing_mark(c, sv, 2, stream); st != WS_OK) return st;
  const bool audio_kernel = !riders || pa.splits > 0;
  if (ws_status st = timing_begin_path(c, riders ? 5 : 1, pa.splits, stream, &sa, audio_kernel); st != WS_OK)
    return st;
  if (audio_kernel) {
    e = launch_plan_kernel(pa, stream, timing_event(c, sa, 0), timing_event(c, sa, 1));
    if (e != hipSuccess) return hip_fail(e, "audio_attn launch");
  } else if (ws_status st = timing_mark(c, sa, 1, stream); st != WS_OK) {
    return st;
  }
  if (pv.merge || pa.merge) {
    ws::CombineArgs none{};
    e = ws::launch_step_combine(pv.merge ? pv.cb : none, pa.merge ? pa.cb : none, stream);
    if (e != hipSuccess) return hip_fail(e, "combine launch");
  }
  return timing_mark(c, sa, 2, stream);
}

}  // namespace

extern "C" {

ws_status ws_cache_create(const ws_cache_config* cfg, ws_cache** out) {
  try {
    return create_impl(cfg, out);
  } catch (...) {
    return fail(WS_ERR_INVALID_ARG, "host allocation failed");
  }
}

ws_status ws_cache_destroy(ws_cache* cache) {
  if (!cache) return WS_OK;
  hipError_t e = hipDeviceSynchronize();
  free_all(cache);
  delete cache;
  if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
  return WS_OK;
}

ws_status ws_cache_reset(ws_cache* cache) {
  if (!cache) return fail(WS_ERR_INVALID_ARG, "NULL cache");
  cache->pt.reset();
  return WS_OK;
}

ws_status ws_kv_append(ws_cache* c, const void* k, const void* v, int64_t tok_stride,
                       int64_t head_stride, const ws_append_desc* d, void* hip_stream) {
  if (!d) return fail(WS_ERR_INVALID_ARG, "NULL argument");
  const ws_append_item item{k, v, tok_stride, head_stride, *d};
  return ws_kv_append_many(c, 1, &item, hip_stream);
}

ws_status ws_kv_append_many(ws_cache* c, int32_t n, const ws_append_item* items, void* hip_stream) {
  if (!c || !items) return fail(WS_ERR_INVALID_ARG, "NULL argument");
  if (n < 1 || n > WS_MAX_APPEND_ITEMS)
    return fail(WS_ERR_INVALID_ARG, "append item count %d outside [1, %d]", n, WS_MAX_APPEND_ITEMS);
  return ws_step_append(c, n, items, 0, nullptr, hip_stream);
}

ws_status ws_step_append(ws_cache* c, int32_t n, const ws_append_item* items, int32_t n_q,
                         const ws_query_item* qs, void* hip_stream) {
  if (!c) return fail(WS_ERR_INVALID_ARG, "NULL cache");
  if (n < 0 || n > WS_MAX_APPEND_ITEMS)
    return fail(WS_ERR_INVALID_ARG, "append item count %d outside [0, %d]", n, WS_MAX_APPEND_ITEMS);
  if (n_q < 0 || n_q > WS_MAX_QUERY_ITEMS)
    return fail(WS_ERR_INVALID_ARG, "query item count %d outside [0, %d]", n_q, WS_MAX_QUERY_ITEMS);
  if (n + n_q < 1) return fail(WS_ERR_INVALID_ARG, "nothing to do: no append and no query item");
  if ((n > 0 && !items) || (n_q > 0 && !qs)) return fail(WS_ERR_INVALID_ARG, "NULL item array");
  if (ws_status st = check_device(c); st != WS_OK) return st;
  const int H = c->cfg.num_heads;
  // Every item is checked before any page is taken.
  for (int i = 0; i < n; ++i) {
    const ws_append_item& it = items[i];
    const ws_append_desc* d = &it.desc;
    if (ws_status st = check_kind(d->kind); st != WS_OK) return st;
    if (d->mode != WS_APPEND_RAW && d->mode != WS_APPEND_NORM_ROPE)
      return fail(WS_ERR_INVALID_ARG, "item %d: bad append mode %d", i, static_cast<int>(d->mode));
    if (d->n_tokens < 1) return fail(WS_ERR_SHAPE, "item %d: n_tokens must be >= 1", i);
    if (ws_status st = check_strides("k", it.k, it.tok_stride, it.head_stride, d->n_tokens, H); st != WS_OK)
      return st;
    if (ws_status st = check_strides("v", it.v, it.tok_stride, it.head_stride, d->n_tokens, H); st != WS_OK)
      return st;
    if (d->mode == WS_APPEND_NORM_ROPE) {
      if (!d->positions || !d->gamma)
        return fail(WS_ERR_INVALID_ARG, "item %d: NORM_ROPE needs positions and gamma", i);
      if (!aligned16(d->gamma)) return fail(WS_ERR_INVALID_ARG, "item %d: gamma is not 16-byte aligned", i);
      if (!(d->eps >= 0.f) || !std::isfinite(d->eps)) return fail(WS_ERR_INVALID_ARG, "item %d: bad eps", i);
    }
    for (int j = 0; j < i; ++j)
      if (items[j].desc.unit == d->unit && items[j].desc.kind == d->kind)
        return fail(WS_ERR_INVALID_ARG, "items %d and %d name the same unit %d kind %d", j, i, d->unit,
                    static_cast<int>(d->kind));
  }
  for (int i = 0; i < n_q; ++i) {
    const ws_query_item& it = qs[i];
    const ws_query_desc* d = &it.desc;
    if (d->mode != WS_APPEND_RAW && d->mode != WS_APPEND_NORM_ROPE)
      return fail(WS_ERR_INVALID_ARG, "query item %d: bad mode %d", i, static_cast<int>(d->mode));
    if (it.n_q < 1) return fail(WS_ERR_SHAPE, "query item %d: n_q must be >= 1", i);
    if (ws_status st = check_strides("q", it.q, it.tok_stride, it.head_stride, it.n_q, H); st != WS_OK)
      return st;
    if (ws_status st = check_strides("q_out", it.q_out, it.out_tok_stride, it.out_head_stride, it.n_q, H);
        st != WS_OK)
      return st;
    if (d->mode == WS_APPEND_NORM_ROPE) {
      if (!d->positions || !d->gamma)
        return fail(WS_ERR_INVALID_ARG, "query item %d: NORM_ROPE needs positions and gamma", i);
      if (!aligned16(d->gamma)) return fail(WS_ERR_INVALID_ARG, "query item %d: gamma is not 16-byte aligned", i);
      if (!(d->eps >= 0.f) || !std::isfinite(d->eps)) return fail(WS_ERR_INVALID_ARG, "query item %d: bad eps", i);
    }
    if (!std::isfinite(d->softmax_scale) || d->softmax_scale < 0.f)
      return fail(WS_ERR_INVALID_ARG, "query item %d: bad softmax_scale", i);
  }
  // Pages: all items or none.  Page lists are copied out at once (the table's
  // segment storage may move on the next creation).
  std::vector<std::vector<int32_t>> pages(static_cast<size_t>(n));
  std::vector<int> created_items;
  auto roll_back = [&]() {
    for (auto it = created_items.rbegin(); it != created_items.rend(); ++it)
      c->pt.release(items[*it].desc.unit, items[*it].desc.kind);
  };
  for (int i = 0; i < n; ++i) {
    const ws_append_desc* d = &items[i].desc;
    ws::Segment* seg = nullptr;
    bool created = false;
    const ws::PtStatus st = c->pt.acquire(d->unit, d->kind, d->n_tokens, &seg, &created);
    if (st != ws::PtStatus::ok) {
      roll_back();
      switch (st) {
        case ws::PtStatus::out_of_pages:
          return fail(WS_ERR_OUT_OF_PAGES, "item %d: pool has %d free pages, segment needs %d", i,
                      c->pt.free_pages(), (d->n_tokens + ws::kPageTokens - 1) / ws::kPageTokens);
        case ws::PtStatus::committed:
          return fail(WS_ERR_COMMITTED, "item %d: unit %d kind %d is committed history", i, d->unit,
                      static_cast<int>(d->kind));
        case ws::PtStatus::shape:
          return fail(WS_ERR_SHAPE, "item %d: rewrite of unit %d kind %d with %d tokens (segment has %d)", i,
                      d->unit, static_cast<int>(d->kind), d->n_tokens, seg ? seg->n_tokens : -1);
        default: return fail(WS_ERR_INVALID_ARG, "item %d: page table error", i);
      }
    }
    if (created) created_items.push_back(i);
    pages[static_cast<size_t>(i)] = seg->pages;
  }

  // Launches of up to kMaxSegs segments and kMaxAppendPages pages each; a
  // segment longer than that continues in the next launch.
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  ws::AppendArgs a{};
  a.num_heads = H;
  a.grid_blocks = kAppendBlocksPerCu * c->num_cus;
  a.kpool = c->kpool;
  a.vpool = c->vpool;
  a.knorm2 = c->knorm2;
  a.rope = c->rope;
  a.flags = c->flags_dev;
  int n_segs = 0;
  int tslot = -1;
  if (ws_status st = timing_begin_path(c, 2, n + n_q, stream, &tslot, true); st != WS_OK) {
    roll_back();
    return st;
  }
  // the first launch stamps event 0 with its start, the final one event 1
  // with its end; one recorded by hand below when no launch takes it
  bool started = false, stopped = false;
  auto flush = [&](bool final_launch) -> hipError_t {
    if (a.n_blocks == 0) return hipSuccess;
    hipEvent_t ev0 = started ? nullptr : timing_event(c, tslot, 0);
    hipEvent_t ev1 = final_launch ? timing_event(c, tslot, 1) : nullptr;
    const hipError_t e = ws::launch_kv_append(a, stream, ev0, ev1);
    started = started || ev0 != nullptr;
    stopped = stopped || ev1 != nullptr;
    a.n_blocks = 0;
    n_segs = 0;
    return e;
  };
  for (int i = 0; i < n; ++i) {
    const ws_append_item& it = items[i];
    const std::vector<int32_t>& pl = pages[static_cast<size_t>(i)];
    int slot = -1;
    for (size_t p = 0; p < pl.size(); ++p) {
      if (a.n_blocks == ws::AppendArgs::kMaxAppendPages) {
        if (hipError_t e = flush(false); e != hipSuccess) {
          roll_back();
          return hip_fail(e, "kv_append launch");
        }
        slot = -1;
      }
      if (slot < 0) {
        if (n_segs == ws::AppendArgs::kMaxSegs) {
          if (hipError_t e = flush(false); e != hipSuccess) {
            roll_back();
            return hip_fail(e, "kv_append launch");
          }
        }
        slot = n_segs++;
        ws::AppendSeg& sg = a.seg[slot];
        sg = ws::AppendSeg{};
        sg.k = static_cast<const uint16_t*>(it.k);
        sg.v = static_cast<const uint16_t*>(it.v);
        sg.tok_stride = it.tok_stride;
        sg.head_stride = it.head_stride;
        sg.n_tokens = it.desc.n_tokens;
        sg.mode = static_cast<int32_t>(it.desc.mode);
        sg.positions = it.desc.positions;
        sg.gamma = it.desc.gamma;
        sg.eps = it.desc.eps;
      }
      a.pages[a.n_blocks] = pl[p];
      a.blk_page[a.n_blocks] = static_cast<int32_t>(p);
      a.blk_seg[a.n_blocks] = static_cast<uint8_t>(slot);
      ++a.n_blocks;
    }
  }
  // query sets: 64-token chunks, no pages
  for (int i = 0; i < n_q; ++i) {
    const ws_query_item& it = qs[i];
    const int chunks = (it.n_q + ws::kPageTokens - 1) / ws::kPageTokens;
    int slot = -1;
    for (int ch = 0; ch < chunks; ++ch) {
      if (a.n_blocks == ws::AppendArgs::kMaxAppendPages) {
        if (hipError_t e = flush(false); e != hipSuccess) {
          roll_back();
          return hip_fail(e, "kv_append launch");
        }
        slot = -1;
      }
      if (slot < 0) {
        if (n_segs == ws::AppendArgs::kMaxSegs) {
          if (hipError_t e = flush(false); e != hipSuccess) {
            roll_back();
            return hip_fail(e, "kv_append launch");
          }
        }
        slot = n_segs++;
        ws::AppendSeg& sg = a.seg[slot];
        sg = ws::AppendSeg{};
        sg.k = static_cast<const uint16_t*>(it.q);
        sg.tok_stride = it.tok_stride;
        sg.head_stride = it.head_stride;
        sg.n_tokens = it.n_q;
        sg.mode = ws::kAppendQuery | (it.desc.mode == WS_APPEND_NORM_ROPE ? 1 : 0);
        sg.positions = it.desc.positions;
        sg.gamma = it.desc.gamma;
        sg.eps = it.desc.eps;
        sg.scale_log2 = scale_log2_of(it.desc.softmax_scale);
        sg.q_out = static_cast<uint16_t*>(it.q_out);
        sg.out_tok_stride = it.out_tok_stride;
        sg.out_head_stride = it.out_head_stride;
      }
      a.pages[a.n_blocks] = -1;
      a.blk_page[a.n_blocks] = ch;
      a.blk_seg[a.n_blocks] = static_cast<uint8_t>(slot);
      ++a.n_blocks;
    }
  }
  if (hipError_t e = flush(true); e != hipSuccess) {
    roll_back();
    return hip_fail(e, "kv_append launch");
  }
  if (!started)
    if (ws_status st = timing_mark(c, tslot, 0, stream); st != WS_OK) return st;
  if (!stopped)
    if (ws_status st = timing_mark(c, tslot, 1, stream); st != WS_OK) return st;
  return timing_mark(c, tslot, 2, stream);
}

ws_status ws_unit_commit(ws_cache* c, int32_t unit) {
  if (!c) return fail(WS_ERR_INVALID_ARG, "NULL cache");
  c->pt.commit(unit);
  return WS_OK;
}

ws_status ws_kv_evict_before(ws_cache* c, int32_t unit) {
  if (!c) return fail(WS_ERR_INVALID_ARG, "NULL cache");
  c->pt.evict_before(unit);
  return WS_OK;
}

ws_status ws_kv_release(ws_cache* c, int32_t unit, ws_kind kind) {
  if (!c) return fail(WS_ERR_INVALID_ARG, "NULL cache");
  if (ws_status st = check_kind(kind); st != WS_OK) return st;
  if (c->pt.release(unit, kind) != ws::PtStatus::ok)
    return fail(WS_ERR_UNKNOWN_UNIT, "no segment for unit %d kind %d", unit, static_cast<int>(kind));
  return WS_OK;
}

ws_status ws_unit_attention(const void* q, int64_t q_tok_stride, int64_t q_head_stride, int32_t n_q,
                            const ws_query_desc* qdesc, ws_cache* cache, const ws_mask_spec* mask,
                            void* out, int64_t out_tok_stride, int64_t out_head_stride,
                            void* hip_stream) {
  if (!mask) return fail(WS_ERR_INVALID_ARG, "NULL argument");
  const QueryGroup g{ws::MaskSpec{mask->q_unit, mask->min_visible_unit, mask->kind_mask}, n_q};
  return attention_impl(false, q, q_tok_stride, q_head_stride, 1, &g, qdesc, cache, out, out_tok_stride,
                        out_head_stride, hip_stream);
}

ws_status ws_unit_attention_groups(const void* q, int64_t q_tok_stride, int64_t q_head_stride,
                                   int32_t n_groups, const ws_query_group* groups, const ws_query_desc* qdesc,
                                   ws_cache* cache, void* out, int64_t out_tok_stride, int64_t out_head_stride,
                                   void* hip_stream) {
  if (!groups) return fail(WS_ERR_INVALID_ARG, "NULL argument");
  if (n_groups < 1 || n_groups > WS_MAX_QUERY_GROUPS)
    return fail(WS_ERR_INVALID_ARG, "query group count %d outside [1, %d]", n_groups, WS_MAX_QUERY_GROUPS);
  QueryGroup g[WS_MAX_QUERY_GROUPS];
  for (int i = 0; i < n_groups; ++i)
    g[i] = QueryGroup{ws::MaskSpec{groups[i].mask.q_unit, groups[i].mask.min_visible_unit,
                                   groups[i].mask.kind_mask},
                      groups[i].n_q};
  return attention_impl(false, q, q_tok_stride, q_head_stride, n_groups, g, qdesc, cache, out, out_tok_stride,
                        out_head_stride, hip_stream);
}

ws_status ws_audio_attention(const void* q, int64_t q_tok_stride, int64_t q_head_stride, int32_t n_q,
                             const ws_query_desc* qdesc, ws_cache* cache, const ws_mask_spec* mask,
                             void* out, int64_t out_tok_stride, int64_t out_head_stride,
                             void* hip_stream) {
  if (!mask) return fail(WS_ERR_INVALID_ARG, "NULL argument");
  const QueryGroup g{ws::MaskSpec{mask->q_unit, mask->min_visible_unit, mask->kind_mask}, n_q};
  return attention_impl(true, q, q_tok_stride, q_head_stride, 1, &g, qdesc, cache, out, out_tok_stride,
                        out_head_stride, hip_stream);
}

ws_status ws_step_attention(ws_cache* c, const ws_attn_call* video, const ws_attn_call* audio, void* hip_stream) {
  return step_attention_impl(c, video, audio, hip_stream, false);
}

ws_status ws_step_attention_noalloc(ws_cache* c, const ws_attn_call* video, const ws_attn_call* audio,
                                    void* hip_stream) {
  return step_attention_impl(c, video, audio, hip_stream, true);
}

ws_status ws_cache_export(ws_cache* c, int32_t unit, ws_kind kind, void* k_host, void* v_host) {
  if (!c) return fail(WS_ERR_INVALID_ARG, "NULL cache");
  if (ws_status st = check_device(c); st != WS_OK) return st;
  if (ws_status st = check_kind(kind); st != WS_OK) return st;
  const ws::Segment* s = c->pt.find(unit, kind);
  if (!s) return fail(WS_ERR_UNKNOWN_UNIT, "no segment for unit %d kind %d", unit, static_cast<int>(kind));
  WS_HIP(hipDeviceSynchronize());
  const int H = c->cfg.num_heads;
  const size_t page_elems = static_cast<size_t>(H) * ws::kPageHeadElems;
  std::vector<uint16_t> kp(page_elems), vp(page_elems);
  uint16_t* ko = static_cast<uint16_t*>(k_host);
  uint16_t* vo = static_cast<uint16_t*>(v_host);
  for (size_t pi = 0; pi < s->pages.size(); ++pi) {
    const size_t base = static_cast<size_t>(s->pages[pi]) * page_elems;
    if (ko) WS_HIP(hipMemcpy(kp.data(), c->kpool + base, page_elems * 2, hipMemcpyDeviceToHost));
    if (vo) WS_HIP(hipMemcpy(vp.data(), c->vpool + base, page_elems * 2, hipMemcpyDeviceToHost));
    for (int slot = 0; slot < ws::kPageTokens; ++slot) {
      const size_t tok = pi * ws::kPageTokens + static_cast<size_t>(slot);
      if (tok >= static_cast<size_t>(s->n_tokens)) break;
      for (int h = 0; h < H; ++h)
        for (int d = 0; d < ws::kHeadDim; ++d) {
          const size_t dst = (tok * H + static_cast<size_t>(h)) * ws::kHeadDim + static_cast<size_t>(d);
          const size_t hb = static_cast<size_t>(h) * ws::kPageHeadElems;
          if (ko) ko[dst] = kp[hb + static_cast<size_t>(ws::k_tile_index(slot, d))];
          if (vo) vo[dst] = vp[hb + static_cast<size_t>(ws::v_tile_index(slot, d))];
        }
    }
  }
  return WS_OK;
}

ws_status ws_segment_tokens(ws_cache* c, int32_t unit, ws_kind kind, int32_t* n_tokens) {
  if (!c || !n_tokens) return fail(WS_ERR_INVALID_ARG, "NULL argument");
  const ws::Segment* s = c->pt.find(unit, kind);
  if (!s) return fail(WS_ERR_UNKNOWN_UNIT, "no segment for unit %d kind %d", unit, static_cast<int>(kind));
  *n_tokens = s->n_tokens;
  return WS_OK;
}

ws_status ws_segment_pages(ws_cache* c, int32_t unit, ws_kind kind, int32_t* pages, int32_t max,
                           int32_t* n_pages) {
  if (!c || !n_pages || max < 0 || (max > 0 && !pages)) return fail(WS_ERR_INVALID_ARG, "bad argument");
  if (ws_status st = check_kind(kind); st != WS_OK) return st;
  const ws::Segment* s = c->pt.find(unit, kind);
  if (!s) return fail(WS_ERR_UNKNOWN_UNIT, "no segment for unit %d kind %d", unit, static_cast<int>(kind));
  const int32_t n = static_cast<int32_t>(s->pages.size());
  for (int32_t i = 0; i < std::min(n, max); ++i) pages[i] = s->pages[static_cast<size_t>(i)];
  *n_pages = n;
  return WS_OK;
}

ws_status ws_cache_info(ws_cache* c, ws_cache_stats* st) {
  if (!c || !st) return fail(WS_ERR_INVALID_ARG, "NULL argument");
  st->pages_total = c->pt.max_pages();
  st->pages_free = c->pt.free_pages();
  st->n_segments = static_cast<int32_t>(c->pt.segments().size());
  st->reserved = 0;
  return WS_OK;
}

ws_status ws_cache_check(ws_cache* c, uint32_t* flags) {
  if (!c || !flags) return fail(WS_ERR_INVALID_ARG, "NULL argument");
  if (ws_status st = check_device(c); st != WS_OK) return st;
  WS_HIP(hipDeviceSynchronize());
  WS_HIP(hipMemcpy(flags, c->flags_dev, sizeof(uint32_t), hipMemcpyDeviceToHost));
  WS_HIP(hipMemset(c->flags_dev, 0, sizeof(uint32_t)));
  WS_HIP(hipDeviceSynchronize());
  return WS_OK;
}

ws_status ws_cache_set_option(ws_cache* c, ws_option opt, int32_t value) {
  if (!c) return fail(WS_ERR_INVALID_ARG, "NULL cache");
  switch (opt) {
    case WS_OPT_VIDEO_KV_SPLITS:
      if (value < 0 || value > kMaxVideoSplits) return fail(WS_ERR_INVALID_ARG, "video splits out of range");
      c->opt_video_splits = value;
      return WS_OK;
    case WS_OPT_AUDIO_KV_SPLITS:
      if (value < 0 || value > kMaxAudioSplits) return fail(WS_ERR_INVALID_ARG, "audio splits out of range");
      c->opt_audio_splits = value;
      return WS_OK;
    case WS_OPT_VIDEO_CLASS_CUS:
      if (value < 0 || value > 1) return fail(WS_ERR_INVALID_ARG, "class CU option must be 0 or 1");
      c->opt_class_cus = value;
      return WS_OK;
    case WS_OPT_STEP_SEPARATE_AUDIO:
      if (value < 0 || value > 1) return fail(WS_ERR_INVALID_ARG, "separate-audio option must be 0 or 1");
      c->opt_separate_audio = value;
      return WS_OK;
    case WS_OPT_VIDEO_RUNNING_MAX:
      if (value < 0 || value > 1) return fail(WS_ERR_INVALID_ARG, "running-max option must be 0 or 1");
      c->opt_running_max = value;
      return WS_OK;
  }
  return fail(WS_ERR_INVALID_ARG, "unknown option %d", static_cast<int>(opt));
}

ws_status ws_cache_timing_enable(ws_cache* c, int32_t capacity) {
  if (!c) return fail(WS_ERR_INVALID_ARG, "NULL cache");
  if (capacity < 0 || capacity > 65536) return fail(WS_ERR_INVALID_ARG, "timing capacity out of range");
  if (ws_status st = check_device(c); st != WS_OK) return st;
  timing_free(c);
  if (capacity == 0) return WS_OK;
  TimingRing& tr = c->timing;
  tr.ev.reserve(3 * static_cast<size_t>(capacity));
  for (int i = 0; i < 3 * capacity; ++i) {
    hipEvent_t e;
    hipError_t he = hipEventCreate(&e);
    if (he != hipSuccess) {
      timing_free(c);
      return hip_fail(he, "hipEventCreate");
    }
    tr.ev.push_back(e);
  }
  tr.meta.assign(static_cast<size_t>(capacity), ws_call_timing{});
  tr.cap = capacity;
  return WS_OK;
}

ws_status ws_cache_timing_read(ws_cache* c, ws_call_timing* out, int32_t max, int32_t* n) {
  if (!c || !n || (max > 0 && !out)) return fail(WS_ERR_INVALID_ARG, "NULL argument");
  TimingRing& tr = c->timing;
  if (tr.cap == 0) return fail(WS_ERR_INVALID_ARG, "timing is not enabled");
  const int32_t count = std::min(tr.count, std::max(max, 0));
  const int32_t first = (tr.next - tr.count + tr.cap) % tr.cap;
  for (int32_t i = 0; i < count; ++i) {
    const int32_t slot = (first + i) % tr.cap;
    WS_HIP(hipEventSynchronize(tr.ev[3 * slot + 2]));
    float a_ms = 0.f, m_ms = 0.f;
    WS_HIP(hipEventElapsedTime(&a_ms, tr.ev[3 * slot], tr.ev[3 * slot + 1]));
    WS_HIP(hipEventElapsedTime(&m_ms, tr.ev[3 * slot + 1], tr.ev[3 * slot + 2]));
    out[i] = tr.meta[slot];
    out[i].attn_us = 1e3f * a_ms;
    out[i].merge_us = 1e3f * m_ms;
  }
  *n = count;
  tr.count = 0;
  return WS_OK;
}

namespace {
ws_status probe_mfma(int32_t workgroups, int32_t iters, bool random_operands, float* sink, double* flop,
                     void* hip_stream) {
  if (!sink || !flop) return fail(WS_ERR_INVALID_ARG, "NULL argument");
  if (workgroups < 1 || workgroups > 65536 || iters < 1 || iters > (1 << 24))
    return fail(WS_ERR_INVALID_ARG, "workgroups must be in [1, 65536] and iters in [1, 2^24]");
  *flop = ws::mfma_probe_flop(workgroups, iters);
  WS_HIP(ws::launch_mfma_probe(workgroups, iters, random_operands, sink, static_cast<hipStream_t>(hip_stream)));
  return WS_OK;
}
}  // namespace

ws_status ws_probe_mfma(int32_t workgroups, int32_t iters, float* sink, double* flop,
                        void* hip_stream) {
  return probe_mfma(workgroups, iters, false, sink, flop, hip_stream);
}

ws_status ws_probe_mfma_random(int32_t workgroups, int32_t iters, float* sink, double* flop,
                               void* hip_stream) {
  return probe_mfma(workgroups, iters, true, sink, flop, hip_stream);
}

ws_status ws_probe_read(const void* buf, int64_t bytes, int32_t workgroups, uint32_t* sink,
                        void* hip_stream) {
  if (!buf || !sink) return fail(WS_ERR_INVALID_ARG, "NULL argument");
  if (bytes <= 0 || bytes % 16 != 0 || reinterpret_cast<uintptr_t>(buf) % 16 != 0)
    return fail(WS_ERR_INVALID_ARG, "buf must be 16-byte aligned and bytes a positive multiple of 16");
  if (workgroups < 1 || workgroups > 65536)
    return fail(WS_ERR_INVALID_ARG, "workgroups must be in [1, 65536]");
  WS_HIP(ws::launch_read_probe(buf, bytes / 16, workgroups, sink, static_cast<hipStream_t>(hip_stream)));
  return WS_OK;
}

const char* ws_last_error(void) { return ws_internal::last_error(); }

}  // extern "C"
