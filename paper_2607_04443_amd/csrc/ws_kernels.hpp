// Launch interface of the gfx950 kernels (host side sees only these structs
// and the launch functions; the kernels live in kernels.hip).
//
// Device memory layout of the paged cache (all bf16).  Pages hold 64 tokens;
// a (page, head) tile is 16 KB contiguous in each pool:
//   K pool: [page][head] tile = [4 d groups][64 slots][32 d]
//   V pool: [page][head] tile = [2 slot halves][128 d][32 slots]  (V stored
//           transposed: eight consecutive keys of one d, the P*V MFMA operand,
//           are one 16-byte load)
// Both tiles are arranged so that the 16-key x 32-d (K) and 16-d x 32-key
// (V^T) operand blocks of one MFMA step cover whole 128-byte lines, and the
// video kernel's direct-to-LDS loads keep a constant per-lane source offset.
// Slots past a segment's last token hold zeros (every append writes all 64
// slots of its pages), so a masked key's zero weight never meets stale data.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace ws {

constexpr int kHeadDim = 128;
constexpr int kPageTokens = 64;
constexpr int64_t kPageHeadElems = int64_t(kHeadDim) * kPageTokens;  // 8192

// Element offsets of (slot, d) within a K tile and a V tile.
__host__ __device__ constexpr int k_tile_index(int slot, int d) {
  return ((d >> 5) * kPageTokens + slot) * 32 + (d & 31);
}
__host__ __device__ constexpr int v_tile_index(int slot, int d) {
  return ((slot >> 5) * kHeadDim + d) * 32 + (slot & 31);
}

// Device error flags (ws_cache_check).
constexpr uint32_t kFlagPositionClamped = 1u;

// Video work partition.  For one query tile the (head, page) units are laid
// on a line in head-major order with seg_cost extra places in front of
// every head (the price of starting a head: query load, key-norm bound,
// pipeline refill), and group g takes the units whose place falls in
// [floor(g L / G), floor((g+1) L / G)), L = heads * (pages + seg_cost): a
// group whose share starts another head gets correspondingly fewer pages.
// The attention kernel (shares), the merge kernel (ranges per head) and the
// host (workspace bound) use these same functions.
struct VideoPartition {
  int64_t heads, pages, seg_cost, groups;
};
__host__ __device__ inline int64_t video_place(const VideoPartition& p, int64_t x) {
  const int64_t h = x / p.pages;
  return h * (p.pages + p.seg_cost) + p.seg_cost + (x - h * p.pages);
}
// The group that holds unit x, and the first unit of group g's share
// (g = groups gives the end), in 64-bit arithmetic.
__host__ __device__ inline int64_t video_group_of_wide(const VideoPartition& p, int64_t x) {
  const int64_t len = p.heads * (p.pages + p.seg_cost);
  return ((video_place(p, x) + 1) * p.groups + len - 1) / len - 1;
}
__host__ __device__ inline int64_t video_group_lo_wide(const VideoPartition& p, int64_t g) {
  const int64_t len = p.heads * (p.pages + p.seg_cost);
  const int64_t v0 = g * len / p.groups;
  const int64_t h = v0 / (p.pages + p.seg_cost), o = v0 - h * (p.pages + p.seg_cost);
  return h * p.pages + (o > p.seg_cost ? o - p.seg_cost : 0);
}
// Whether the same lookups fit 32-bit arithmetic: with len = heads * (pages
// + seg_cost), every intermediate value is at most (len + 1) * (groups + 1).
// The 32-bit form gives the same integers; on the GPU it avoids the long
// instruction sequence of a 64-bit division.
__host__ __device__ inline bool video_fits32(const VideoPartition& p) {
  const int64_t len = p.heads * (p.pages + p.seg_cost);
  return (len + 1) * (p.groups + 1) < (int64_t(1) << 32);
}
// The lookups the host and the kernels use.
__host__ __device__ inline int64_t video_group_of(const VideoPartition& p, int64_t x) {
  if (!video_fits32(p)) return video_group_of_wide(p, x);
  const uint32_t pages = static_cast<uint32_t>(p.pages), cost = static_cast<uint32_t>(p.seg_cost);
  const uint32_t stride = pages + cost, len = static_cast<uint32_t>(p.heads) * stride;
  const uint32_t ux = static_cast<uint32_t>(x), h = ux / pages;
  const uint32_t place = h * stride + cost + (ux - h * pages);
  return static_cast<int64_t>(((place + 1) * static_cast<uint32_t>(p.groups) + len - 1) / len) - 1;
}
__host__ __device__ inline int64_t video_group_lo(const VideoPartition& p, int64_t g) {
  if (!video_fits32(p)) return video_group_lo_wide(p, g);
  const uint32_t pages = static_cast<uint32_t>(p.pages), cost = static_cast<uint32_t>(p.seg_cost);
  const uint32_t stride = pages + cost, len = static_cast<uint32_t>(p.heads) * stride;
  const uint32_t v0 = static_cast<uint32_t>(g) * len / static_cast<uint32_t>(p.groups);
  const uint32_t h = v0 / stride, o = v0 - h * stride;
  return static_cast<int64_t>(h * pages + (o > cost ? o - cost : 0u));
}

struct RopeTables {
  const float2* tab[3];  // (cos, sin) per band: [max_pos[b]][pairs[b]]
  int32_t max_pos[3];
  int32_t pairs[3];
};

// One segment of an append launch: a K/V segment (mode 0 raw, 1 norm +
// rope; block x writes one page) or a query set (mode 2 raw, 3 norm + rope:
// the key path's arithmetic, then the scale, written to q_out; block x
// prepares 64 tokens, no page).
struct AppendSeg {
  const uint16_t* k;     // keys, or the queries
  const uint16_t* v;
  int64_t tok_stride;
  int64_t head_stride;
  int32_t n_tokens;      // tokens of the whole segment
  int32_t mode;
  const int32_t* positions;
  const float* gamma;
  float eps;
  float scale_log2;      // queries: softmax scale * log2(e)
  uint16_t* q_out;       // queries: prepared Q''
  int64_t out_tok_stride;
  int64_t out_head_stride;
};
constexpr int kAppendQuery = 2;  // mode bit: a query set

// Several segments in one launch: block x of the grid writes page pages[x],
// which is page blk_page[x] of segment blk_seg[x] (for a query set: token
// chunk blk_page[x]).
struct AppendArgs {
  static constexpr int kMaxSegs = 8;
  static constexpr int kMaxAppendPages = 192;
  AppendSeg seg[kMaxSegs];
  int32_t n_blocks;      // items (pages and query chunks) of the launch
  int32_t num_heads;
  int32_t grid_blocks;   // blocks of the launch (each loops over the (item, head) tiles)
  uint16_t* kpool;
  uint16_t* vpool;
  float* knorm2;
  RopeTables rope;
  uint32_t* flags;
  int32_t pages[kMaxAppendPages];
  int32_t blk_page[kMaxAppendPages];
  uint8_t blk_seg[kMaxAppendPages];
};

// Query class of a video attention call: the rows of one unit's queries in a
// call that holds queries of several units.  Rows [q0, q0 + n_q) of the call
// walk entries [page0, page0 + n_pages) of the call's page list (the pages
// their block-causal mask leaves visible), with n_groups groups of n_qtiles
// workgroups starting at workgroup wg0 (VideoPartition over this class's
// pages).  A call with queries of one unit is one class.
struct AttnClass {
  int32_t q0, n_q, page0, n_pages, n_groups, n_qtiles, wg0, pad;
};
constexpr int kMaxClasses = 8;

struct AttnArgs {
  // Visible page lists up to this length travel in the kernel arguments
  // (no upload, no copy dispatch ahead of the kernel); longer ones are
  // uploaded to device memory.
  static constexpr int kInlinePages = 384;
  const uint16_t* q;
  int64_t q_tok_stride;
  int64_t q_head_stride;
  int32_t n_q;
  int32_t num_heads;
  int32_t mode;          // query prologue: 0 raw, 1 norm + rope, 2 prepared (Q'' as given)
  const int32_t* positions;
  const float* gamma;
  float eps;
  float scale_log2;      // softmax scale * log2(e)
  RopeTables rope;
  const uint16_t* kpool;
  const uint16_t* vpool;
  const float* knorm2;
  int32_t fixed_shift;   // 1: softmax shift from the key-norm bound when it is small enough
  const int2* pages;     // visible pages (page id, valid tokens) in device memory, or
                         // nullptr: the first n_pages entries of inline_pages
  const uint16_t* zeros; // 1 KB of zeros (direct-load source for empty blocks)
  int32_t n_pages;
  int32_t n_splits;      // audio: key-range splits (the combine kernel merges them)
  int32_t pages_per_split;
  int32_t n_groups;      // video: workgroup groups sharing the (head, page) units (all classes)
  int32_t seg_cost;      // video: partition cost of starting a head (VideoPartition)
  int32_t n_qtiles;      // audio: query tiles; video: all classes' query tiles
  int32_t n_classes;     // video: query classes (1..kMaxClasses)
  int32_t n_wg;          // video: workgroups of the launch (all classes)
  AttnClass cls[kMaxClasses];
  uint16_t* out;
  int64_t out_tok_stride;
  int64_t out_head_stride;
  float* part_o;         // [split][head][n_q][128], normalised: fp32 (audio), bf16 (video)
  float* part_lse;       // [split][head][n_q], log2 domain (scaled logits)
  // Video: rider rows, a second query set (prepared Q'') that walks the same
  // pages in the spare rows of the last query tile: rows rq_row0 .. rq_row0 +
  // n_rq - 1 of the call's row space (rq_row0 = n_q, a single query class)
  // are rows 0 .. n_rq - 1 of rq.  Their key ranges always go out as fp32
  // partials, [range][head][n_rq][128] and [range][head][n_rq].
  const uint16_t* rq;
  int64_t rq_tok_stride;
  int64_t rq_head_stride;
  int32_t n_rq;          // 0: no rider rows
  int32_t rq_row0;
  float* rpart_o;
  float* rpart_lse;
  // The rider rows' own pages (visible to them only), entries rx_page0 ..
  // rx_page0 + rx_pages - 1 of the inline page list (rx_pages = 0: none, or
  // attended elsewhere): attended by the last rx_waves waves (which have no
  // rows) of the last query tile's workgroup of the group holding each
  // head's last page, one key range per wave after the head's ranges.
  int32_t rx_page0;
  int32_t rx_pages;
  int32_t rx_waves;
  uint32_t* flags;
  int2 inline_pages[kInlinePages];
};

struct CombineArgs {
  const float* part_o;
  const float* part_lse;
  int32_t n_splits;      // key ranges per head (when n_groups == 0)
  int32_t n_groups;      // > 0: video schedule, ranges per head follow from
                         //      each class's shares (VideoPartition)
  int32_t n_classes;     // video: the call's query classes (AttnArgs::cls)
  int32_t seg_cost;
  AttnClass cls[kMaxClasses];
  // Audio merge with rider rows: after the n_splits ranges of the audio
  // kernel come the ranges the video kernel wrote for the rows, as many per
  // head as the video partition over r_pages pages with r_groups groups
  // gives (r_groups = 0: none).
  int32_t r_pages;
  int32_t r_groups;
  int32_t r_extra;       // more ranges per head: the rows' own pages, from the video kernel's idle waves
  int32_t n_q;
  int32_t num_heads;
  uint16_t* out;
  int64_t out_tok_stride;
  int64_t out_head_stride;
};

hipError_t launch_kv_append(const AppendArgs& a, hipStream_t stream, hipEvent_t start = nullptr,
                            hipEvent_t stop = nullptr);
// Video path: 256-query tiles on 8 waves, 32x32x16 bf16 MFMA, LDS-staged
// pages; n_groups x n_qtiles workgroups, each with an even share of the
// (head, page) units.
hipError_t launch_unit_attention(const AttnArgs& a, hipStream_t stream, hipEvent_t start = nullptr,
                                 hipEvent_t stop = nullptr);
// Audio path: 4 independent waves per (head, 16-query tile, key range),
// pages loaded straight into registers, 16x16x32 bf16 MFMA.
hipError_t launch_audio_attention(const AttnArgs& a, hipStream_t stream, hipEvent_t start = nullptr,
                                  hipEvent_t stop = nullptr);
hipError_t launch_combine(const CombineArgs& a, hipStream_t stream);
// The merges of a video call (n_groups > 0) and an audio call (num_heads > 0)
// in one launch; either may be absent (zero-initialised).
hipError_t launch_step_combine(const CombineArgs& video, const CombineArgs& audio, hipStream_t stream);
// Calibration probes (peaks.hip).
hipError_t launch_mfma_probe(int workgroups, int iters, bool random_operands, float* sink, hipStream_t stream);
hipError_t launch_read_probe(const void* buf, int64_t n16, int workgroups, uint32_t* sink,
                             hipStream_t stream);
double mfma_probe_flop(int workgroups, int iters);

// Split-KV workspace of the no-allocation step entry point: a static device
// array of this many bytes in the library's code object (one per device).
constexpr size_t kStaticScratchBytes = size_t(32) << 20;
// Device address of that array on the current device, looked up once per
// device (hipGetSymbolAddress) and kept.
hipError_t static_scratch(void** ptr);

constexpr int kVideoQTile = 256;
constexpr int kMaxVideoSplits = 8;  // key-range splits of the video kernel

// Whether a partition into `groups` shares splits some head over more than
// one share (then a merge of the key ranges is needed): no head is split
// when the group count divides the head count.
inline bool video_heads_split(int64_t heads, int64_t groups) { return groups > heads || heads % groups != 0; }

// Group count of the video kernel for one query class (host): the G that
// minimises rounds of the CUs x (a share's pages plus a fixed cost per
// segment it holds: query prologue, or switch to the next head), plus the
// merge launch when a head is split.  Shares line up with heads when G is a
// multiple or a divisor of H, so that every group holds max(G, H) / G whole
// segments; otherwise the G shares cut G + H - 1 segments.  At most
// kMaxVideoSplits ranges per head (ceil(G / H) + 1 of them).
inline int64_t video_group_count(int64_t heads, int64_t qtiles, int64_t pages, int64_t cus) {
  if (pages == 0) return heads;
  constexpr double kSegCostPages = 9.5;   // about 15 us against about 1.6 us per page
  constexpr double kMergeCostPages = 4.0;  // the merge launch and its traffic
  const int64_t units = heads * pages;
  const int64_t one_round = cus / qtiles > 1 ? cus / qtiles : 1;
  int64_t g_max = heads * (kMaxVideoSplits - 1);
  if (units < g_max) g_max = units;
  if (4 * one_round < g_max) g_max = 4 * one_round;
  int64_t best = heads < g_max ? heads : g_max;
  double best_cost = -1.0;
  for (int64_t g = 1; g <= g_max; ++g) {
    const double rounds = static_cast<double>((g + one_round - 1) / one_round);
    const bool aligned = g % heads == 0 || heads % g == 0;
    const double segs = static_cast<double>(aligned ? (g > heads ? g : heads) : g + heads - 1) / g;
    const double cost = rounds * (static_cast<double>(units) / g + kSegCostPages * segs) +
                        (video_heads_split(heads, g) ? kMergeCostPages : 0.0);
    if (best_cost < 0 || cost < best_cost - 1e-9) {
      best = g;
      best_cost = cost;
    }
  }
  return best;
}
constexpr int kVideoWaves = kVideoQTile / 32;
constexpr int kAudioQTile = 16;
constexpr int kMaxAudioQ = 64;  // audio queries per call

}  // namespace ws
