/*
 * ws.h -- C ABI of the Wan-Streamer v0.2 performer unit-attention library
 * (libws.so, HIP on MI355X / gfx950).
 *
 * The library owns one paged K/V cache per ws_cache handle and runs the
 * performer's per-denoising-step attention of the next streaming unit over it
 * (Wan-Streamer v0.2, arXiv 2607.04443):
 *   - a per-rank K/V cache, allocated up front, receives the thinker's slices
 *     and the generated units' K/V (Abstract; Sec. 3, the performer item and
 *     the unit-k schedule paragraph);
 *   - generated latents are committed into history after every unit
 *     (Sec. 2.1); the full-history cache is updated per unit (Sec. 3);
 *   - attention is block-causal on one timeline, the block being the 160 ms
 *     unit (Fig. 1 caption; Sec. 1);
 *   - the long video latent sequence and the short, unsharded audio latent
 *     sequence are separate query sets (Sec. 3).
 * On one GPU the cache holds every head (no sequence sharding, no collectives).
 *
 * Numeric conventions (the paper states none): bf16 storage, fp32
 * accumulation; head_dim 128; 64-token pages; per-head RMS-norm over the head
 * dimension, eps and weight gamma[128] given by the caller, applied before
 * rotary positions; rotary pairs (2p, 2p+1) with the first rope_pairs[0]
 * pairs driven by t, the next rope_pairs[1] by h and the rest by w, pair p_b
 * of a band of n_b pairs turning by pos * theta^(-p_b / n_b); softmax scale
 * 1/sqrt(head_dim) unless given.
 *
 * Conventions common to every call:
 *   - Pointers named "device" are HIP device pointers (e.g. from torch
 *     tensors); the caller owns them and keeps them alive until the work
 *     enqueued on the given stream has completed.
 *   - Tensors are bf16 with element strides given in elements; the innermost
 *     (head_dim) stride is 1.  Pointers must be 16-byte aligned and strides
 *     multiples of 8 elements.
 *   - Calls that take a hip_stream (a hipStream_t; NULL = the null stream)
 *     enqueue work and return without waiting.  Host-side validation happens
 *     before anything is enqueued; a call that fails validation changes no
 *     state.  After a failed launch the call returns WS_ERR_HIP.
 *   - ws_last_error() returns a thread-local message for the last non-OK
 *     status of the calling thread.
 *   - One ws_cache is used from one host thread at a time.  Calls on one
 *     cache must be issued on one stream (or be ordered by the caller).
 *   - The attention calls allocate nothing: pools, page tables and split-KV
 *     workspaces are allocated by ws_cache_create.
 */
#ifndef WS_H_
#define WS_H_

#include <stdint.h>

#if defined(__GNUC__) || defined(__clang__)
#define WS_API __attribute__((visibility("default")))
#else
#define WS_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ws_cache ws_cache; /* opaque; owned by the library */

typedef enum ws_status {
  WS_OK = 0,
  WS_ERR_INVALID_ARG = 1,   /* null pointer, bad enum, misaligned pointer or stride */
  WS_ERR_SHAPE = 2,         /* sizes outside the supported range, token count mismatch */
  WS_ERR_OUT_OF_PAGES = 3,  /* the page pool cannot hold the new segment */
  WS_ERR_UNKNOWN_UNIT = 4,  /* no segment for the named (unit, kind) */
  WS_ERR_COMMITTED = 5,     /* rewrite of a segment already committed to history */
  WS_ERR_UNSUPPORTED = 6,   /* head_dim != 128, page_tokens != 64, ... */
  WS_ERR_HIP = 7            /* a HIP runtime call or kernel launch failed */
} ws_status;

/* Segment kinds: the thinker's conditioning slice, and a unit's generated
 * video or audio latents. */
typedef enum ws_kind { WS_KIND_COND = 0, WS_KIND_VIDEO = 1, WS_KIND_AUDIO = 2 } ws_kind;
#define WS_KIND_BIT(kind) (1u << (unsigned)(kind))

/* RAW: keys stored as given (the thinker's slice arrives in final form).
 * NORM_ROPE: keys RMS-normed per head, weighted by gamma, then rotated.
 * PREPARED (queries of the attention calls only): the queries are already
 * Q'' = RoPE(RMSNorm(Q) * gamma, positions) * softmax_scale * log2(e) in
 * bf16 (or Q * softmax_scale * log2(e) for RAW), as ws_step_append writes
 * them; the attention uses them as given. */
typedef enum ws_append_mode {
  WS_APPEND_RAW = 0,
  WS_APPEND_NORM_ROPE = 1,
  WS_QUERY_PREPARED = 2
} ws_append_mode;

typedef struct ws_cache_config {
  int32_t num_heads;       /* H >= 1 */
  int32_t head_dim;        /* must be 128 */
  int32_t page_tokens;     /* must be 64 */
  int32_t max_pages;       /* pool capacity; each page holds 64 tokens of every head */
  int32_t max_q_tokens;    /* largest n_q accepted by the attention calls (>= 1) */
  int32_t rope_max_pos[3]; /* exclusive bounds of the t, h, w positions (each >= 1) */
  int32_t rope_pairs[3];   /* rotary pairs per band t, h, w; must sum to head_dim / 2 */
  double rope_theta;       /* rotary base (> 1), e.g. 10000 */
} ws_cache_config;

typedef struct ws_append_desc {
  int32_t unit;              /* streaming unit the tokens belong to */
  ws_kind kind;
  int32_t n_tokens;          /* >= 1; a rewrite must repeat the first append's count */
  ws_append_mode mode;
  const int32_t* positions;  /* device int32 [n_tokens][3] (t, h, w); NORM_ROPE only */
  const float* gamma;        /* device fp32 [head_dim]; NORM_ROPE only */
  float eps;                 /* RMS-norm epsilon (>= 0); NORM_ROPE only */
} ws_append_desc;

/* One segment of a batched append (ws_kv_append_many): the K/V buffers and
 * strides of ws_kv_append plus its descriptor. */
typedef struct ws_append_item {
  const void* k;
  const void* v;
  int64_t tok_stride;
  int64_t head_stride;
  ws_append_desc desc;
} ws_append_item;

#define WS_MAX_APPEND_ITEMS 16

typedef struct ws_query_desc {
  ws_append_mode mode;       /* NORM_ROPE: RMS-norm + rotary on Q; RAW: Q used as given;
                                PREPARED: Q'' from ws_step_append (the fields below unused) */
  const int32_t* positions;  /* device int32 [n_q][3]; NORM_ROPE only */
  const float* gamma;        /* device fp32 [head_dim]; NORM_ROPE only */
  float eps;
  float softmax_scale;       /* logit scale; 0 selects 1/sqrt(head_dim) */
} ws_query_desc;

/* One query set prepared by ws_step_append: q (mode RAW or NORM_ROPE in
 * desc) is turned into Q'' (see WS_QUERY_PREPARED) and written to q_out.
 *   q:     device bf16 [n_q][H][128], strides (tok_stride, head_stride);
 *   q_out: device bf16 [n_q][H][128], strides (out_tok_stride, out_head_stride),
 *          not overlapping q. */
typedef struct ws_query_item {
  const void* q;
  int64_t tok_stride;
  int64_t head_stride;
  int32_t n_q;               /* >= 1 */
  ws_query_desc desc;
  void* q_out;
  int64_t out_tok_stride;
  int64_t out_head_stride;
} ws_query_item;

#define WS_MAX_QUERY_ITEMS 4

/* Block-causal visibility for a query set that belongs to unit q_unit.  A
 * segment (unit u, kind k) is visible iff bit k of kind_mask is set, u <= q_unit,
 * and, for VIDEO and AUDIO segments, u >= min_visible_unit (history window;
 * INT32_MIN for no window).  Within a unit keys are visible in both
 * directions.  A query with no visible key gets a zero output. */
typedef struct ws_mask_spec {
  int32_t q_unit;
  int32_t min_visible_unit;
  uint32_t kind_mask;        /* OR of WS_KIND_BIT(...) */
} ws_mask_spec;

typedef struct ws_cache_stats {
  int32_t pages_total;
  int32_t pages_free;
  int32_t n_segments;
  int32_t reserved;
} ws_cache_stats;

/* Tuning knobs (0 = automatic choice).  They change scheduling only, never
 * results beyond floating-point summation order. */
typedef enum ws_option {
  WS_OPT_VIDEO_KV_SPLITS = 0,  /* video kernel: split every head's keys into this many
                                  equal ranges (1..8) instead of the balanced share */
  WS_OPT_AUDIO_KV_SPLITS = 1,  /* key-range splits of the audio kernel (1..512) */
  /* Softmax shift of the video kernel: 0 = automatic (a query row's logit
   * bound |q''| * max |k| when it is at most 40 in log2 units, else a lazily
   * raised running maximum), 1 = always the running maximum. */
  WS_OPT_VIDEO_RUNNING_MAX = 2,
  /* ws_unit_attention_groups: 0 = the query groups share one round of the
   * CUs in proportion to their work, 1 = every group is partitioned as if it
   * had all CUs (several rounds of workgroups in one launch). */
  WS_OPT_VIDEO_CLASS_CUS = 3,
  /* ws_step_attention: 0 = the audio rows ride in the video kernel when the
   * step allows it (see there), 1 = always the separate audio kernel. */
  WS_OPT_STEP_SEPARATE_AUDIO = 4
} ws_option;

/* Creates a cache: allocates the K and V page pools (2 * max_pages * H * 64 *
 * 128 * 2 bytes), a per-(page, head) table of key-norm maxima (max_pages * H
 * floats, written by ws_kv_append with each page), the rotary cos/sin tables
 * (built in double precision on the host, stored as fp32), page-list arenas
 * and split-KV workspaces, and clears the pools to zero.  Uses the current HIP device.  Synchronous.
 * On success *out owns all of it until ws_cache_destroy. */
WS_API ws_status ws_cache_create(const ws_cache_config* cfg, ws_cache** out);

/* Waits for the device, then frees everything the cache owns.  NULL is a no-op. */
WS_API ws_status ws_cache_destroy(ws_cache* cache);

/* Drops every segment and returns all pages to the pool (host-side only;
 * the pool contents are left as they are). */
WS_API ws_status ws_cache_reset(ws_cache* cache);

/* Writes n_tokens K/V of one (unit, kind) into the cache: a thinker slice
 * (Sec. 3: ranks write incoming K/V into their cache) or a generated unit's
 * K/V at a denoising step.  The first append of a (unit, kind) takes fresh
 * pages (WS_ERR_OUT_OF_PAGES if the pool is short); a later append of the same
 * uncommitted (unit, kind) rewrites its slots in place (same n_tokens, else
 * WS_ERR_SHAPE; WS_ERR_COMMITTED after ws_unit_commit).
 *   k, v: device bf16, element (t, h, d) at [t * tok_stride + h * head_stride + d],
 *         t < n_tokens, h < num_heads, d < 128.
 * NORM_ROPE keys: K' = RoPE(RMSNorm(K) * gamma, positions), computed in fp32,
 * rounded to bf16.  Values are always stored as given.  Positions outside
 * [0, rope_max_pos) are clamped and flagged (ws_cache_check).  Each written
 * page also records, per head, the largest squared norm of its stored keys. */
WS_API ws_status ws_kv_append(ws_cache* cache, const void* k, const void* v, int64_t tok_stride,
                       int64_t head_stride, const ws_append_desc* desc, void* hip_stream);

/* ws_kv_append for n (1..WS_MAX_APPEND_ITEMS) segments at once, e.g. a
 * denoising step's video and audio K/V together with a thinker slice (Sec. 3):
 * the writes of all items share kernel launches (one launch per 8 items and 192
 * pages).  Each item obeys the rules of ws_kv_append and is stored exactly as a
 * separate ws_kv_append of it would store it.  All items are checked before any
 * page is taken, and if one item fails (bad argument, two items naming the same
 * (unit, kind), WS_ERR_OUT_OF_PAGES, WS_ERR_COMMITTED, WS_ERR_SHAPE) the
 * segments this call created are released again and nothing is launched.
 * items: host array of n entries, read before the call returns. */
WS_API ws_status ws_kv_append_many(ws_cache* cache, int32_t n, const ws_append_item* items,
                                   void* hip_stream);

/* A denoising step's input stage in one launch (Sec. 3: the performer writes
 * the step's K/V into its cache and attends with the step's queries): the K/V
 * appends of ws_kv_append_many (n_kv items, 0..WS_MAX_APPEND_ITEMS) and the
 * query preparation of n_q query sets (0..WS_MAX_QUERY_ITEMS; RMS-norm, gamma
 * and rotary as for NORM_ROPE keys, then the softmax scale and log2(e),
 * rounded once to bf16).  n_kv + n_q >= 1.  The K/V items follow every rule
 * of ws_kv_append_many (and are all checked, with the query items, before any
 * page is taken); ws_unit_attention / ws_audio_attention then take q_out
 * with mode WS_QUERY_PREPARED and give the same result as NORM_ROPE (or RAW)
 * on q, up to the summation order of the RMS norm.  kv and qs: host arrays,
 * read before the call returns (either may be NULL when its count is 0). */
WS_API ws_status ws_step_append(ws_cache* cache, int32_t n_kv, const ws_append_item* kv,
                                int32_t n_q, const ws_query_item* qs, void* hip_stream);

/* Marks the VIDEO and AUDIO segments of `unit` as committed history
 * (Sec. 2.1); they can no longer be rewritten.  Host-only. */
WS_API ws_status ws_unit_commit(ws_cache* cache, int32_t unit);

/* Frees the VIDEO and AUDIO segments of every unit < `unit` (history window
 * advance).  Conditioning slices are kept.  Host-only; the caller must not
 * have work in flight that still reads those pages. */
WS_API ws_status ws_kv_evict_before(ws_cache* cache, int32_t unit);

/* Frees one (unit, kind) segment (e.g. a superseded conditioning slice).
 * Host-only, with the same in-flight caveat. */
WS_API ws_status ws_kv_release(ws_cache* cache, int32_t unit, ws_kind kind);

/* The performer's attention of a unit's video latent queries over the
 * visible cache (Sec. 3, the expensive latent-generation path):
 *   Q' = RoPE(RMSNorm(Q) * gamma, positions) (or Q for RAW),
 *   out[i] = sum_j softmax_j(scale * <Q'_i, K'_j>) V_j over the visible keys.
 *   q:   device bf16 [n_q][H][128] with strides (q_tok_stride, q_head_stride).
 *   out: device bf16 [n_q][H][128] with strides (out_tok_stride, out_head_stride).
 * 1 <= n_q <= max_q_tokens.  MFMA flash kernel: 256-query tiles, 64-key pages.
 * Groups of workgroups (one per query tile) take even shares of the
 * (head, page) work, so a head's keys may be split into ranges (split-KV);
 * those are merged by log-sum-exp in a second kernel.
 * The softmax shift of a query row is its logit bound |Q''_i| * max |K'_j|
 * (Cauchy-Schwarz over the pages of one key range) when that bound is at most
 * 40 in log2 units, else a lazily raised running maximum
 * (WS_OPT_VIDEO_RUNNING_MAX forces the latter); both give the same softmax. */
WS_API ws_status ws_unit_attention(const void* q, int64_t q_tok_stride, int64_t q_head_stride,
                            int32_t n_q, const ws_query_desc* qdesc, ws_cache* cache,
                            const ws_mask_spec* mask, void* out, int64_t out_tok_stride,
                            int64_t out_head_stride, void* hip_stream);

/* Queries of several units in one call (Fig. 1 caption: block-causal
 * attention on one timeline; Sec. 2.1: units committed into history), e.g. a
 * catch-up after a stall or re-encoding committed units.  The call's query
 * rows are the groups' rows in order: group g holds groups[g].n_q >= 0 rows
 * (at least one group has rows) and its rows see exactly what
 * ws_unit_attention with groups[g].mask would let them see.  Each group's
 * visible page list is built on the host and walked only by that group's
 * query tiles, so pages a group's mask hides cost it nothing; a group that
 * sees nothing gets zero rows.  Arguments as ws_unit_attention, with n_q =
 * the sum of the groups' rows (at most max_q_tokens) and qdesc's positions
 * covering all rows; 1 <= n_groups <= WS_MAX_QUERY_GROUPS.  groups: host
 * array, read before the call returns.  With a single group the call is
 * ws_unit_attention. */
typedef struct ws_query_group {
  int32_t n_q;
  ws_mask_spec mask;
} ws_query_group;

#define WS_MAX_QUERY_GROUPS 8

WS_API ws_status ws_unit_attention_groups(const void* q, int64_t q_tok_stride, int64_t q_head_stride,
                                          int32_t n_groups, const ws_query_group* groups,
                                          const ws_query_desc* qdesc, ws_cache* cache, void* out,
                                          int64_t out_tok_stride, int64_t out_head_stride,
                                          void* hip_stream);

/* The same attention for the few audio latent queries of a unit (Sec. 3:
 * short, unsharded).  Memory-bound split-KV kernel: fp32 partials over key
 * ranges, merged by log-sum-exp.  Arguments as ws_unit_attention;
 * 1 <= n_q <= min(max_q_tokens, 64). */
WS_API ws_status ws_audio_attention(const void* q, int64_t q_tok_stride, int64_t q_head_stride,
                             int32_t n_q, const ws_query_desc* qdesc, ws_cache* cache,
                             const ws_mask_spec* mask, void* out, int64_t out_tok_stride,
                             int64_t out_head_stride, void* hip_stream);

/* One attention call of ws_step_attention: the arguments of
 * ws_unit_attention / ws_audio_attention. */
typedef struct ws_attn_call {
  const void* q;
  int64_t q_tok_stride;
  int64_t q_head_stride;
  int32_t n_q;
  ws_query_desc desc;
  ws_mask_spec mask;
  void* out;
  int64_t out_tok_stride;
  int64_t out_head_stride;
} ws_attn_call;

/* A denoising step's two attentions over the cache (Sec. 3: the long video
 * latent queries and the short audio latent queries of the same unit): the
 * video kernel, the audio kernel, and one launch that merges both calls' key
 * ranges.  Both calls are validated before anything is enqueued.  video,
 * audio: host structs, read before the call returns.  The audio call's key
 * ranges use a workspace of their own.
 *
 * Audio rows riding in the video kernel: when the audio call is
 * WS_QUERY_PREPARED, every page the video call sees is visible to the audio
 * call too, and the audio rows fit the spare rows of the video call's last
 * 256-query tile (n_audio <= 256 * ceil(n_video / 256) - n_video), the video
 * kernel also computes the audio rows over the video call's pages (the pages
 * are streamed once for both); the pages the audio call alone sees (the
 * units' audio tokens) are walked by the video kernel's waves that have no
 * rows (when its last query tile leaves at least two) or else by the audio
 * kernel; the merge folds all the ranges.
 * WS_OPT_STEP_SEPARATE_AUDIO turns this off.  The video output always equals
 * what ws_unit_attention(video) writes, bit for bit; the audio output equals
 * ws_audio_attention(audio) bit for bit when the rows do not ride, and
 * otherwise agrees with it to the rounding of the bf16 softmax weights (taken
 * under another shift) and the order of fp32 sums.  With timing
 * enabled the call records two ring entries: the video kernel (merge time 0),
 * and the audio kernel with the shared merge (path 1; path 5 when the audio
 * rows ride, with the audio kernel's range count, 0 when it was not
 * launched). */
WS_API ws_status ws_step_attention(ws_cache* cache, const ws_attn_call* video, const ws_attn_call* audio,
                                   void* hip_stream);

/* ws_step_attention for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same kernels and the same outputs, bit for bit, but the two
 * calls' split-KV partials go to a static workspace in the library's code
 * object (32 MiB per device, kept until the process ends) instead of the
 * cache's workspaces.  The call itself allocates nothing.
 * Limit: the partials of both calls must fit the 32 MiB: video (ranges per
 * head) x H x n_q rows of 260 bytes, audio (key ranges, plus the video
 * kernel's ranges of the audio rows when they ride in it) x H x n_q rows of
 * 516 bytes, each region rounded up to 256 bytes; a larger step returns
 * WS_ERR_SHAPE before anything is enqueued.  (The v0.2 unit at 640x368 with
 * an 8-unit window needs about 29 MB.)  Every call on a device shares that
 * device's workspace: calls that overlap in time on one device (different
 * streams, or different threads) race and must be ordered by the caller.
 * Nothing in it has to start at zero: each call writes every partial row it
 * reads. */
WS_API ws_status ws_step_attention_noalloc(ws_cache* cache, const ws_attn_call* video,
                                           const ws_attn_call* audio, void* hip_stream);

/* The attention sub-block of one performer layer at one denoising step
 * (Sec. 3: the performer generates the next unit conditioned on its K/V
 * cache and writes the unit's own K/V into it; the whole performer step and
 * the K/V and latent transfers must fit one 160 ms unit).  A ws_block holds
 * the layer's two projection weights and the buffers of one step:
 *   [Q | K | V] = X W_qkv   (hipBLASLt GEMM, bf16 in and out, fp32 accumulation)
 *   ws_step_append: the unit's video and audio K/V (NORM_ROPE) and the
 *                   preparation of both query sets
 *   ws_step_attention (or ws_unit_attention without audio rows)
 *   Y = O W_out             (hipBLASLt GEMM)
 * X holds the unit's n_video video tokens followed by its n_audio audio
 * tokens.  Column block j of W_qkv (j = 0 Q, 1 K, 2 V) holds columns
 * [j hidden, (j + 1) hidden), head h in its columns 128 h .. 128 h + 127.
 * The weights are random here: the call measures the time of the sub-block
 * and the share of attention in it. */
typedef struct ws_block ws_block; /* opaque; owned by the library */

/* Creates a block over `cache` (hidden = 128 * num_heads of the cache):
 *   w_qkv: device bf16 [hidden][3 hidden] row-major; w_out: device bf16
 *   [hidden][hidden] row-major; both 16-byte aligned, owned by the caller and
 *   kept alive and unchanged while the block is used;
 *   max_rows: most tokens (n_video + n_audio) a step takes, 1..max_q_tokens.
 * Allocates the GEMM workspace (64 MiB) and the step's Q/K/V, prepared-query
 * and attention buffers (max_rows rows); ws_block_step allocates no device
 * memory (its first step with a new row count creates, and destroys, two
 * HIP events to time the GEMM candidates).
 * The cache must outlive the block.  Synchronous. */
WS_API ws_status ws_block_create(ws_cache* cache, const void* w_qkv, const void* w_out, int32_t max_rows,
                                 ws_block** out);

/* Waits for the device, then frees what the block owns.  NULL is a no-op. */
WS_API ws_status ws_block_destroy(ws_block* block);

typedef struct ws_block_step_args {
  const void* x;              /* device bf16 [n_video + n_audio][hidden], rows contiguous */
  int32_t n_video;            /* >= 1 */
  int32_t n_audio;            /* 0..64 */
  int32_t unit;               /* the unit the tokens belong to (the K/V append's unit) */
  const int32_t* video_positions;  /* device int32 [n_video][3] */
  const int32_t* audio_positions;  /* device int32 [n_audio][3] (NULL when n_audio = 0) */
  const float* gamma_q;       /* device fp32 [128] */
  const float* gamma_k;       /* device fp32 [128] */
  float eps;
  float softmax_scale;        /* 0 selects 1/sqrt(128) */
  ws_mask_spec video_mask;    /* visibility of the video rows (q_unit = unit) */
  ws_mask_spec audio_mask;    /* visibility of the audio rows */
  void* attn_out;             /* optional device bf16 [n][hidden]: the attention output O
                                 (NULL: kept inside the block) */
  void* y;                    /* device bf16 [n][hidden], rows contiguous */
} ws_block_step_args;

/* One sub-block step on hip_stream, in the order above.  The append follows
 * the rules of ws_kv_append (a first step of a unit takes pages, later steps
 * rewrite them; committed units are rejected); arguments, pages and the
 * rewrite rule are checked before anything is enqueued.  The first step
 * with a given row count (n_video + n_audio) asks hipBLASLt for up to 16
 * algorithms per projection, times each on this step's operands on
 * hip_stream (waiting for the stream; a few ms) and keeps the fastest; later
 * steps with that row count reuse it (run the first one outside any stream
 * capture).  With timing enabled
 * the two projections record ring entries of their own (path 3: QKV
 * projection, path 4: output projection), besides the append and attention
 * entries.  args: host struct, read before the call returns. */
WS_API ws_status ws_block_step(ws_block* block, const ws_block_step_args* args, void* hip_stream);

/* Debug read-back of one segment in logical order: k_host and v_host receive
 * bf16 [n_tokens][H][128] (contiguous host buffers owned by the caller).
 * Waits for the device.  k_host or v_host may be NULL to skip it. */
WS_API ws_status ws_cache_export(ws_cache* cache, int32_t unit, ws_kind kind, void* k_host,
                          void* v_host);

/* Token count of a segment (WS_ERR_UNKNOWN_UNIT if absent). */
WS_API ws_status ws_segment_tokens(ws_cache* cache, int32_t unit, ws_kind kind, int32_t* n_tokens);

/* Debug: the pool page ids of segment (unit, kind) in token order (page i
 * holds tokens 64 i .. 64 i + 63).  Writes min(count, max) ids to pages (host
 * int32 array owned by the caller; may be NULL when max is 0) and the
 * segment's page count to *n_pages.  Host-only; WS_ERR_UNKNOWN_UNIT if absent. */
WS_API ws_status ws_segment_pages(ws_cache* cache, int32_t unit, ws_kind kind, int32_t* pages,
                                  int32_t max, int32_t* n_pages);

/* Page-pool occupancy.  Host-only. */
WS_API ws_status ws_cache_info(ws_cache* cache, ws_cache_stats* stats);

/* Waits for the device and returns (and clears) the device-side flags:
 * bit 0 = a position outside [0, rope_max_pos) was clamped. */
WS_API ws_status ws_cache_check(ws_cache* cache, uint32_t* flags);

/* Sets a tuning knob (see ws_option); value 0 restores the automatic choice. */
WS_API ws_status ws_cache_set_option(ws_cache* cache, ws_option opt, int32_t value);

/* Launch timing of the attention entry points (for benchmarks and
 * profilers).  While enabled, every ws_unit_attention / ws_audio_attention
 * call records three HIP events on its own stream: the start and the end of
 * its attention kernel, taken by the kernel's dispatch itself
 * (hipExtLaunchKernelGGL: the kernel's execution, as a profiler's kernel
 * trace reports it), and one recorded after the split-KV merge kernel;
 * every append call (ws_kv_append, ws_kv_append_many, ws_step_append) takes
 * the start of its first launch and the end of its last (merge time 0).
 * The projections of ws_block_step are timed with events recorded before
 * and after them.  The cache keeps the events of the last `capacity` calls
 * in a ring (older calls are overwritten); recording adds no
 * synchronization. */
typedef struct ws_call_timing {
  int32_t path;      /* 0 = video attention, 1 = audio attention, 2 = append,
                        3 = QKV projection, 4 = output projection (ws_block_step),
                        5 = audio attention with its rows in the video kernel
                        (ws_step_attention) */
  int32_t n_splits;  /* audio: key-range splits; video: workgroup groups; append: items */
  float attn_us;     /* attention kernel, microseconds */
  float merge_us;    /* merge kernel, microseconds (0 when there is none) */
} ws_call_timing;

/* capacity > 0 (at most 65536) enables timing with a ring of that many calls
 * (creating 3 * capacity HIP events on the cache's device) and clears it;
 * capacity = 0 disables timing and destroys the events. */
WS_API ws_status ws_cache_timing_enable(ws_cache* cache, int32_t capacity);

/* Waits for the recorded calls, copies up to `max` of them into out[] (host
 * array owned by the caller, oldest call first), stores the count in *n and
 * clears the ring.  WS_ERR_INVALID_ARG if timing is not enabled. */
WS_API ws_status ws_cache_timing_read(ws_cache* cache, ws_call_timing* out, int32_t max,
                                      int32_t* n);

/* Calibration probes: the bf16 MFMA rate and the HBM read rate the GPU
 * sustains, so that measured rates can be set against measured ceilings as
 * well as the published peaks.  Each enqueues one kernel on hip_stream and
 * returns; the caller times it (HIP events on that stream).  Invalid
 * arguments return WS_ERR_INVALID_ARG before anything is enqueued.
 *
 * ws_probe_mfma: `workgroups` (1..65536) workgroups of 4 waves; each wave
 * issues iters (1..2^24) rounds of 4 independent 32x32x16 bf16 MFMAs on
 * register operands (small integers, the same for the 4 chains: few bits
 * switch).  *flop (host) receives the launch's FLOP count.  sink is a device
 * float[1], written only in a case the arithmetic never reaches.
 *
 * ws_probe_mfma_random: the same launch with hashed operands, random sign
 * and mantissa bits and magnitudes in [0.5, 2), different for each chain (the
 * switching activity of attention's operands, which lowers the clock the
 * chip holds under a long MFMA load).
 *
 * ws_probe_read: reads the `bytes` bytes at device address buf once
 * (16-byte aligned, bytes a positive multiple of 16) with `workgroups`
 * (1..65536) workgroups of 256 threads, each reading one contiguous chunk
 * with nontemporal loads (the form that sustains the highest read rate);
 * sink is a device uint32[1], likewise written only in a case that does not
 * occur for ordinary data. */
WS_API ws_status ws_probe_mfma(int32_t workgroups, int32_t iters, float* sink, double* flop,
                               void* hip_stream);
WS_API ws_status ws_probe_mfma_random(int32_t workgroups, int32_t iters, float* sink, double* flop,
                                      void* hip_stream);
WS_API ws_status ws_probe_read(const void* buf, int64_t bytes, int32_t workgroups, uint32_t* sink,
                               void* hip_stream);

/* Thread-local message for the last non-OK status ("" if none). */
WS_API const char* ws_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* WS_H_ */
