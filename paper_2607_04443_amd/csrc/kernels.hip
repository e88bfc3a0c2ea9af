// gfx950 (MI355X, CDNA4) kernels of the performer unit attention.
//
//  kv_append       writes a segment's K/V into its cache pages; NORM_ROPE keys
//                  get per-head RMS-norm, the gamma weight and (t,h,w) rotary
//                  positions in fp32 before the bf16 store; V is stored
//                  transposed per page ([d][slot]).
//  unit_attn       video queries: flash attention over the visible pages with
//                  v_mfma_f32_32x32x16_bf16, K/V pages staged through LDS
//                  (double-buffered), online softmax in the exp2 domain.
//  audio_attn      the few audio queries: memory-bound split-KV, one wave per
//                  key range, v_mfma_f32_16x16x32_bf16 straight from registers.
//  combine         log-sum-exp merge of split-KV partials.
//
// The attention is the performer's per-step attention over its K/V cache
// (Wan-Streamer v0.2, Sec. 3); block-causal visibility (Fig. 1 caption) is
// resolved on the host into the list of visible pages.
#include <hip/hip_ext.h>

#include <algorithm>
#include <cstddef>
#include <mutex>
#include <type_traits>

#include "ws_kernels.hpp"

namespace ws {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kNegInf = -__builtin_inff();
// Lazy-max threshold of the video softmax, log2 units.
constexpr float kLazyTau = 8.0f;
// Largest logit bound (log2 units) used as a fixed softmax shift.
constexpr float kShiftBoundMax = 40.0f;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Two fp32 -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  bf16x2 r = __builtin_convertvector((f32x2){lo, hi}, bf16x2);
  return __builtin_bit_cast(uint32_t, r);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// (cos, sin) of rotary pair p (0..63) for a token at position pos (t, h, w).
__device__ __forceinline__ float2 rope_cs(const RopeTables& r, int p, int pt, int ph, int pw) {
  const int p0 = r.pairs[0], p01 = r.pairs[0] + r.pairs[1];
  if (p < p0) return r.tab[0][pt * r.pairs[0] + p];
  if (p < p01) return r.tab[1][ph * r.pairs[1] + (p - p0)];
  return r.tab[2][pw * r.pairs[2] + (p - p01)];
}

// Clamps a token's (t, h, w) into the table; flags a clamp.
__device__ __forceinline__ void clamp_pos(const RopeTables& r, int t, int h, int w, uint32_t* flags,
                                          int& pt, int& ph, int& pw) {
  const int ct = min(max(t, 0), r.max_pos[0] - 1);
  const int ch = min(max(h, 0), r.max_pos[1] - 1);
  const int cw = min(max(w, 0), r.max_pos[2] - 1);
  if ((ct != t) | (ch != h) | (cw != w)) atomicOr(flags, kFlagPositionClamped);
  pt = ct;
  ph = ch;
  pw = cw;
}

// Loads a token's (t, h, w), clamped into the table; flags a clamp.
__device__ __forceinline__ void load_pos(const RopeTables& r, const int32_t* positions, int tok,
                                         uint32_t* flags, int& pt, int& ph, int& pw) {
  int t = positions[3 * tok + 0], h = positions[3 * tok + 1], w = positions[3 * tok + 2];
  const int ct = min(max(t, 0), r.max_pos[0] - 1);
  const int ch = min(max(h, 0), r.max_pos[1] - 1);
  const int cw = min(max(w, 0), r.max_pos[2] - 1);
  if ((ct != t) | (ch != h) | (cw != w)) atomicOr(flags, kFlagPositionClamped);
  pt = ct;
  ph = ch;
  pw = cw;
}

typedef const __attribute__((address_space(4))) AppendSeg* const_append_seg;
typedef const __attribute__((address_space(4))) AppendArgs* const_append_args;

// The append launch's arguments, read in place from the kernel argument
// segment (the kernel's only argument is the AppendArgs): with run-time
// indexes into the by-value argument the compiler copies all of it to
// private memory.
__device__ __forceinline__ const_append_args append_args() {
  return (const_append_args)__builtin_amdgcn_kernarg_segment_ptr();
}

// Query preparation, one block of an append launch: tokens 64 chunk ..
// 64 chunk + 63 of query set si, one head, 16 threads per token row as in
// the key path below.  Q'' = RoPE(RMSNorm(Q) * gamma, positions) * scale *
// log2(e) (mode 3) or Q * scale * log2(e) (mode 2), in fp32, rounded once to
// bf16: the attention kernels' own query prologue, done once per step
// instead of once per workgroup that reads the queries.
__device__ __forceinline__ void prepare_queries(const RopeTables& rope, uint32_t* flags, const_append_seg sg,
                                                int chunk, int head) {
  const uint16_t* src = sg->k;
  const int64_t tok_stride = sg->tok_stride, head_stride = sg->head_stride;
  const int n_tokens = sg->n_tokens;
  const bool norm_rope = (sg->mode & 1) != 0;
  const float scale = sg->scale_log2;
  uint16_t* dst = sg->q_out;
  const int64_t out_tok_stride = sg->out_tok_stride, out_head_stride = sg->out_head_stride;
  const int t = threadIdx.x, c = t & 15, rr = t >> 4;
  const int tok0 = chunk * kPageTokens;
  float g[8];
  float eps = 0.f;
  const int32_t* positions = nullptr;
  if (norm_rope) {
    const float* gamma = sg->gamma;
    eps = sg->eps;
    positions = sg->positions;
    const float4 g0 = *reinterpret_cast<const float4*>(gamma + 8 * c);
    const float4 g1 = *reinterpret_cast<const float4*>(gamma + 8 * c + 4);
    g[0] = g0.x; g[1] = g0.y; g[2] = g0.z; g[3] = g0.w;
    g[4] = g1.x; g[5] = g1.y; g[6] = g1.z; g[7] = g1.w;
  }
  u32x4 qx[4];
  int tpos[4][3];
#pragma unroll
  for (int pass = 0; pass < 4; ++pass) {
    const int tok = tok0 + pass * 16 + rr;
    const bool valid = tok < n_tokens;
    qx[pass] = valid ? *reinterpret_cast<const u32x4*>(src + tok * tok_stride + head * head_stride + 8 * c)
                     : (u32x4){0u, 0u, 0u, 0u};
    if (norm_rope && valid) {
      tpos[pass][0] = positions[3 * tok + 0];
      tpos[pass][1] = positions[3 * tok + 1];
      tpos[pass][2] = positions[3 * tok + 2];
    } else {
      tpos[pass][0] = tpos[pass][1] = tpos[pass][2] = 0;
    }
  }
#pragma unroll
  for (int pass = 0; pass < 4; ++pass) {
    const int tok = tok0 + pass * 16 + rr;
    const bool valid = tok < n_tokens;
    const u32x4 x = qx[pass];
    u32x4 y;
    if (norm_rope) {
      float f[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f[2 * i] = bf16_lo(x[i]);
        f[2 * i + 1] = bf16_hi(x[i]);
      }
      float ss = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) ss += f[i] * f[i];
      ss += __shfl_xor(ss, 1);
      ss += __shfl_xor(ss, 2);
      ss += __shfl_xor(ss, 4);
      ss += __shfl_xor(ss, 8);
      const float inv = rsqrtf(ss * (1.0f / kHeadDim) + eps);
      int pt = 0, ph = 0, pw = 0;
      if (valid) clamp_pos(rope, tpos[pass][0], tpos[pass][1], tpos[pass][2], flags, pt, ph, pw);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float y0 = f[2 * i] * inv * g[2 * i];
        const float y1 = f[2 * i + 1] * inv * g[2 * i + 1];
        const float2 cs = rope_cs(rope, 4 * c + i, pt, ph, pw);
        y[i] = pack_bf16((y0 * cs.x - y1 * cs.y) * scale, (y0 * cs.y + y1 * cs.x) * scale);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) y[i] = pack_bf16(bf16_lo(x[i]) * scale, bf16_hi(x[i]) * scale);
    }
    if (valid) *reinterpret_cast<u32x4*>(dst + tok * out_tok_stride + head * out_head_stride + 8 * c) = y;
  }
}

// ------------------------------------------------------------------------- //
// kv_append: one (item, head) tile of an append launch, an item being a K/V
// page or a 64-token chunk of a query set of one of up to
// AppendArgs::kMaxSegs segments.  256 threads; vt and wave_norm2 are the
// block's LDS, free again when the call returns.
// ------------------------------------------------------------------------- //
__device__ __forceinline__ void append_tile(const_append_args A, int item, int head,
                                            uint16_t (*vt)[kHeadDim + 8], float* wave_norm2) {
  const const_append_seg sg = A->seg + A->blk_seg[item];
  RopeTables rope;
#pragma unroll
  for (int b = 0; b < 3; ++b) {
    rope.tab[b] = A->rope.tab[b];
    rope.max_pos[b] = A->rope.max_pos[b];
    rope.pairs[b] = A->rope.pairs[b];
  }
  uint32_t* const flags = A->flags;
  if (sg->mode & kAppendQuery) {
    prepare_queries(rope, flags, sg, A->blk_page[item], head);
    return;
  }
  const int num_heads = A->num_heads;
  const int page = A->pages[item];
  const uint16_t* src_k = sg->k;
  const uint16_t* src_v = sg->v;
  const int64_t tok_stride = sg->tok_stride, head_stride = sg->head_stride;
  const int n_tokens = sg->n_tokens;
  const int mode = sg->mode;
  const int tok0 = A->blk_page[item] * kPageTokens;
  const int64_t tile = (static_cast<int64_t>(page) * num_heads + head) * kPageHeadElems;
  uint16_t* kdst = A->kpool + tile;
  uint16_t* vdst = A->vpool + tile;
  const int t = threadIdx.x;

  // K: 16 threads per token row, 8 consecutive d each; 16 rows per pass.
  // Alongside, the largest squared norm of the stored rows of the tile.
  const int c = t & 15;
  const int rr = t >> 4;
  float norm2 = 0.f;
  float g[8];
  float eps = 0.f;
  const int32_t* positions = nullptr;
  if (mode == 1) {
    const float* gamma = sg->gamma;
    eps = sg->eps;
    positions = sg->positions;
    const float4 g0 = *reinterpret_cast<const float4*>(gamma + 8 * c);
    const float4 g1 = *reinterpret_cast<const float4*>(gamma + 8 * c + 4);
    g[0] = g0.x; g[1] = g0.y; g[2] = g0.z; g[3] = g0.w;
    g[4] = g1.x; g[5] = g1.y; g[6] = g1.z; g[7] = g1.w;
  }
  // all loads of the tile are issued up front (K rows, V rows, positions)
  u32x4 kx[4], vx[4];
  int tpos[4][3];
#pragma unroll
  for (int pass = 0; pass < 4; ++pass) {
    const int tok = tok0 + pass * 16 + rr;
    kx[pass] = tok < n_tokens ? *reinterpret_cast<const u32x4*>(src_k + tok * tok_stride + head * head_stride + 8 * c)
                              : (u32x4){0u, 0u, 0u, 0u};
    if (mode == 1 && tok < n_tokens) {
      tpos[pass][0] = positions[3 * tok + 0];
      tpos[pass][1] = positions[3 * tok + 1];
      tpos[pass][2] = positions[3 * tok + 2];
    } else {
      tpos[pass][0] = tpos[pass][1] = tpos[pass][2] = 0;
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ch = t + 256 * i;
    const int tok = tok0 + (ch >> 4);
    vx[i] = tok < n_tokens ? *reinterpret_cast<const u32x4*>(src_v + tok * tok_stride + head * head_stride + 8 * (ch & 15))
                           : (u32x4){0u, 0u, 0u, 0u};
  }
  // V rows go to LDS ([slot][d]) as soon as they arrive, which frees their
  // registers before the key arithmetic
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ch = t + 256 * i;
    *reinterpret_cast<u32x4*>(&vt[ch >> 4][8 * (ch & 15)]) = vx[i];
  }

#pragma unroll
  for (int pass = 0; pass < 4; ++pass) {
    const int slot = pass * 16 + rr;
    const int tok = tok0 + slot;
    const bool valid = tok < n_tokens;
    const u32x4 x = kx[pass];
    u32x4 y = x;
    if (mode == 1) {
      float f[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f[2 * i] = bf16_lo(x[i]);
        f[2 * i + 1] = bf16_hi(x[i]);
      }
      float ss = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) ss += f[i] * f[i];
      // the 16 threads of a row are 16 consecutive lanes
      ss += __shfl_xor(ss, 1);
      ss += __shfl_xor(ss, 2);
      ss += __shfl_xor(ss, 4);
      ss += __shfl_xor(ss, 8);
      const float inv = rsqrtf(ss * (1.0f / kHeadDim) + eps);
      int pt = 0, ph = 0, pw = 0;
      if (valid) clamp_pos(rope, tpos[pass][0], tpos[pass][1], tpos[pass][2], flags, pt, ph, pw);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float y0 = f[2 * i] * inv * g[2 * i];
        const float y1 = f[2 * i + 1] * inv * g[2 * i + 1];
        const float2 cs = rope_cs(rope, 4 * c + i, pt, ph, pw);
        y[i] = pack_bf16(y0 * cs.x - y1 * cs.y, y0 * cs.y + y1 * cs.x);
      }
      if (!valid) y = (u32x4){0u, 0u, 0u, 0u};
    }
    *reinterpret_cast<u32x4*>(kdst + k_tile_index(slot, 8 * c)) = y;
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) ss += bf16_lo(y[i]) * bf16_lo(y[i]) + bf16_hi(y[i]) * bf16_hi(y[i]);
    ss += __shfl_xor(ss, 1);
    ss += __shfl_xor(ss, 2);
    ss += __shfl_xor(ss, 4);
    ss += __shfl_xor(ss, 8);
    norm2 = fmaxf(norm2, ss);
  }
  norm2 = fmaxf(norm2, __shfl_xor(norm2, 16));
  norm2 = fmaxf(norm2, __shfl_xor(norm2, 32));
  if ((t & 63) == 0) wave_norm2[t >> 6] = norm2;

  // V: staged [slot][d] in LDS above, written [d][slot].
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ch = t + 256 * i;
    const int d = ch >> 3, tc = ch & 7;
    u32x4 y;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      y[j] = static_cast<uint32_t>(vt[8 * tc + 2 * j][d]) |
             (static_cast<uint32_t>(vt[8 * tc + 2 * j + 1][d]) << 16);
    *reinterpret_cast<u32x4*>(vdst + v_tile_index(8 * tc, d)) = y;
  }
  if (t == 0)
    A->knorm2[static_cast<int64_t>(page) * num_heads + head] =
        fmaxf(fmaxf(wave_norm2[0], wave_norm2[1]), fmaxf(wave_norm2[2], wave_norm2[3]));
}

// The launch: a grid of a few blocks per CU that loop over the launch's
// (item, head) tiles, consecutive tiles being the heads of one item.  (One
// block per tile made the launch as long as dispatching its ~1,400 short
// blocks: their average life was about an eighth of the launch.)
__global__ __launch_bounds__(256) void kv_append_kernel(const AppendArgs args) {
  (void)args;  // read in place, through append_args()
  __shared__ __attribute__((aligned(16))) uint16_t vt[kPageTokens][kHeadDim + 8];
  __shared__ float wave_norm2[4];
  const const_append_args A = append_args();
  const int heads = A->num_heads;
  const int n_tiles = A->n_blocks * heads;
  for (int tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
    append_tile(A, tile / heads, tile % heads, vt, wave_norm2);
    __syncthreads();  // vt and wave_norm2 are rewritten by the next tile
  }
}

// ------------------------------------------------------------------------- //
// unit_attn (video): 8 waves x 32 queries, 64-key pages through LDS.
//
// Per wave and page, with lane l = 32*h + i (h = half, i = query column):
//   S^T[key][q] = K[key][:] . Q'[q][:]   2 x (32x32) tiles, 8 MFMAs of k=16 each
//   O^T[d][q]  += V^T[d][key] P^T[key][q] 4 x (32x32) tiles, 4 MFMAs of k=16 each
// Every lane owns one query column, so the softmax row statistics live in one
// lane (plus its partner l^32).  The K rows of S-tile row m are loaded from key
// swap23(m) (bits 2 and 3 exchanged), which makes accumulator register r of
// lane half h hold key 16*(r/8) + 8*h + (r%8): registers 0-7 and 8-15 are then
// directly the B operands (eight consecutive keys) of the P*V MFMAs.
// ------------------------------------------------------------------------- //
__device__ __forceinline__ int swap23(int m) { return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1); }
// LDS stages of the video kernel (a ring of five pages, 160 KB: the previous
// page, whose V^T the pipelined schedule still reads, the current page, the
// next page, already complete so that its first operands can be read before
// the page barrier, and the two after it in flight), filled by direct
// global->LDS loads (global_load_lds_dwordx4: lane l of a wave writes 16
// bytes at base + 16 l).
//   K    [64 rows][16 chunks]: row R holds key swap23(R); its logical chunk c
//        (dims 8c..8c+7) sits at position c ^ (R & 15).  Lane i of either
//        half then reads row i (+32 for the second tile), and the 16 lanes
//        of a ds_read_b128 pass hit 16 distinct 16-byte bank groups.
//   V^T  [128 d][8 chunks]: logical chunk c (keys 8c..8c+7) of row d sits at
//        position c ^ ((d >> 1) & 7).
constexpr int kStages = 5;
__shared__ __attribute__((aligned(1024))) uint16_t g_k0[kPageTokens * kHeadDim];
__shared__ __attribute__((aligned(1024))) uint16_t g_k1[kPageTokens * kHeadDim];
__shared__ __attribute__((aligned(1024))) uint16_t g_k2[kPageTokens * kHeadDim];
__shared__ __attribute__((aligned(1024))) uint16_t g_k3[kPageTokens * kHeadDim];
__shared__ __attribute__((aligned(1024))) uint16_t g_k4[kPageTokens * kHeadDim];
__shared__ __attribute__((aligned(1024))) uint16_t g_v0[kHeadDim * kPageTokens];
__shared__ __attribute__((aligned(1024))) uint16_t g_v1[kHeadDim * kPageTokens];
__shared__ __attribute__((aligned(1024))) uint16_t g_v2[kHeadDim * kPageTokens];
__shared__ __attribute__((aligned(1024))) uint16_t g_v3[kHeadDim * kPageTokens];
__shared__ __attribute__((aligned(1024))) uint16_t g_v4[kHeadDim * kPageTokens];

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

struct VideoState {
  f32x16 o[4];
  float m_run;
  float l_run;
  bool first;
};

// Read-only for a whole launch: accessed through the constant address space
// so that uniform reads become scalar loads.
typedef const __attribute__((address_space(4))) int2* const_page_list;

// The call's visible page list: in device memory, or in the kernel
// arguments themselves (the kernel's only argument is the AttnArgs, at the
// start of the kernel argument segment; addressing it through the segment
// pointer keeps the compiler from copying the argument to private memory).
__device__ __forceinline__ const_page_list page_list(const AttnArgs& a) {
  if (a.pages) return (const_page_list)a.pages;
  const __attribute__((address_space(4))) char* seg =
      (const __attribute__((address_space(4))) char*)__builtin_amdgcn_kernarg_segment_ptr();
  return (const_page_list)(seg + offsetof(AttnArgs, inline_pages));
}

struct VideoCtx {
  bool active;             // the wave has at least one real query row
  const_page_list pages;   // visible page list
  const uint16_t* kpool;   // pool base + this head's tile offset
  const uint16_t* vpool;
  int64_t page_stride;     // elements per page (all heads)
  int wave, half, l32;
  uint32_t dma_k, dma_v;   // this lane's source byte offsets within a tile (block i = 0)
  bf16x8 qreg[8];
};

// LDS byte offset of a pointer into a __shared__ object.
__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) void*)p));
}

// One direct load: each lane's 16 bytes at sbase + voff go to LDS at
// lds + 16 * lane.  Written as inline asm: with the compiler's own LDS-DMA
// intrinsic in flight, every later LDS read waits for lgkmcnt(0), which
// serializes the MFMA operand reads.  M0 is restored afterwards; completion
// is tracked by the explicit vmcnt wait in wait_dma.
__device__ __forceinline__ void dma16(const uint16_t* sbase, uint32_t voff, uint32_t lds) {
  // both are wave-uniform by construction; make that visible to the compiler
  // (readfirstlane returns int: widen through uint32_t, never sign-extend)
  lds = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(lds));
  const uint64_t b = reinterpret_cast<uint64_t>(sbase);
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b >> 32)));
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b)));
  sbase = reinterpret_cast<const uint16_t*>((static_cast<uint64_t>(hi) << 32) | lo);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "global_load_lds_dwordx4 %1, %2\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(voff), "s"(sbase), "s"(lds)
      : "memory");
}

// Issues the direct loads of page `page` (K and V^T tiles of this head) into
// the stage (k_dst, v_dst): per wave two 1 KB blocks of each, block
// b = 8 i + wave.  Block b of K is rows 4b..4b+3, lane l at row
// R = 32 i + 4 wave + l/16, position l%16; block b of V^T is rows
// d = 64 i + 8 wave + l/8, position l%8.  The lane's source offset changes
// with i only by a constant: 32 keys (1024 elements) in the K tile, 64 d
// rows (2048 elements) in the V tile.
__device__ __forceinline__ void stage_dma(const VideoCtx& c, int page, uint16_t* k_dst, uint16_t* v_dst) {
  const uint16_t* kp = c.kpool + page * c.page_stride;
  const uint16_t* vp = c.vpool + page * c.page_stride;
  const uint32_t kl = lds_offset(k_dst) + 1024 * c.wave, vl = lds_offset(v_dst) + 1024 * c.wave;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    dma16(kp + 1024 * i, c.dma_k, kl + 8192 * i);
    dma16(vp + 2048 * i, c.dma_v, vl + 8192 * i);
  }
}
constexpr int kDmaPerPage = 4;  // direct loads per wave and page

// Waits for this wave's direct loads of the page after next's predecessor:
// everything but the kDmaPerPage loads issued last (loads retire in order).
// The barrier that follows then makes every wave's share visible.
__device__ __forceinline__ void wait_dma_all_but_last_page() {
  static_assert(kDmaPerPage == 4, "vmcnt encoding below");
  __builtin_amdgcn_s_waitcnt(0x0F74);  // vmcnt(4), expcnt(7), lgkmcnt(15)
}
__device__ __forceinline__ void wait_dma_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)

// max over lanes l and l ^ 32 (v_permlane32_swap: no LDS round trip)
__device__ __forceinline__ float pair_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// v_max3 tree over one lane's 16 logits of a 32-key tile
__device__ __forceinline__ float max16(const f32x16& s) {
  const float a = fmaxf(s[0], fmaxf(s[1], s[2]));
  const float b = fmaxf(s[3], fmaxf(s[4], s[5]));
  const float c = fmaxf(s[6], fmaxf(s[7], s[8]));
  const float d = fmaxf(s[9], fmaxf(s[10], s[11]));
  const float e = fmaxf(s[12], fmaxf(s[13], s[14]));
  return fmaxf(fmaxf(a, fmaxf(b, c)), fmaxf(d, fmaxf(e, s[15])));
}

// P = exp2(s) of a 32-key tile as bf16: pa holds the lane's first eight keys,
// pb the next eight (the B operands of two P*V MFMAs).  Returns the lane's
// row sum over the same bf16 values the MFMAs consume.
__device__ __forceinline__ float exp_tile(const f32x16& s, u32x4& pa, u32x4& pb) {
  const bf16x2 ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
  float la = 0.f, lb = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    // bit-cast scalar temporaries: a bit-cast of a vector element subscript
    // is lowered to element 0 by this compiler
    const uint32_t x = pack_bf16(fast_exp2(s[2 * i]), fast_exp2(s[2 * i + 1]));
    const uint32_t y = pack_bf16(fast_exp2(s[8 + 2 * i]), fast_exp2(s[9 + 2 * i]));
    pa[i] = x;
    pb[i] = y;
    la = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, x), ones, la, false);
    lb = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, y), ones, lb, false);
  }
  return la + lb;
}

__device__ __forceinline__ void scale_o(VideoState& st, float alpha) {
#pragma unroll
  for (int t4 = 0; t4 < 4; ++t4) st.o[t4] *= alpha;
}

// Empty asm statements that make a value live in a register at this point:
// they keep the compiler from sinking the speculative softmax past the rare
// rescale branch, and a scalar page-list load from drifting next to its use.
__device__ __forceinline__ void pin_sgpr(int x) { asm volatile("" ::"s"(x)); }
__device__ __forceinline__ void pin_vgpr(u32x4& x) { asm volatile("" : "+v"(x)); }
__device__ __forceinline__ void pin_vgpr(float& x) { asm volatile("" : "+v"(x)); }

template <int kStage>
__device__ __forceinline__ uint16_t* stage_k() {
  return kStage == 0 ? g_k0 : kStage == 1 ? g_k1 : kStage == 2 ? g_k2 : kStage == 3 ? g_k3 : g_k4;
}
template <int kStage>
__device__ __forceinline__ uint16_t* stage_v() {
  return kStage == 0 ? g_v0 : kStage == 1 ? g_v1 : kStage == 2 ? g_v2 : kStage == 3 ? g_v3 : g_v4;
}
__device__ __forceinline__ const uint16_t* stage_v_at(int stage) {
  return stage == 0 ? g_v0 : stage == 1 ? g_v1 : stage == 2 ? g_v2 : stage == 3 ? g_v3 : g_v4;
}

// Page list index of the page staged three pages ahead of pi (near the
// range's end the last page re-stages itself into an idle stage: nothing
// reads that copy).
__device__ __forceinline__ int ahead3(int pi, int p_end) { return pi + 3 < p_end ? pi + 3 : p_end - 1; }

// A page for a wave whose 32 query rows are all padding (ragged last query
// tile): it only issues its share of the loads of page pi + 3.
template <int kCur>
__device__ __forceinline__ void video_page_stage_only(const VideoCtx& c, int pi, int p_end) {
  pi = __builtin_amdgcn_readfirstlane(pi);
  const int ahead = c.pages[ahead3(pi, p_end)].x;
  __syncthreads();
  stage_dma(c, ahead, stage_k<(kCur + 3) % kStages>(), stage_v<(kCur + 3) % kStages>());
  wait_dma_all_but_last_page();
}

// One 64-key page from LDS stage kCur, as two 32-key tiles (keys 0-31 in s0,
// 32-63 in s1), scheduled by hand in 32 steps of one MFMA each:
//   A: S tile 0                      B: S tile 1 + exp of tile 0
//   D: P*V tile 0 + exp of tile 1    F: P*V tile 1
// Each step issues the LDS operand read four steps ahead, its MFMA, and its
// share of the softmax VALU work (two exponentials, one pack, one dot2), and
// ends in a scheduling fence, so the emitted order is the program order.
// The S accumulators start at -m_run (or -inf past the page's valid tokens),
// so they hold the exp2 argument directly.
//   kLazy = false: m_run is a fixed upper bound of the row's logits (from the
//     key norms), so there is no running maximum and nothing to rescale.
//   kLazy = true: m_run is a running maximum raised lazily.  The
//     exponentials are taken speculatively against the current m_run; when a
//     tile raises it by more than kLazyTau (rare after the first tile), a
//     branch between the phases rescales O and l and recomputes that tile's P.
// Right after the page's barrier, the direct loads of page pi + 3 into the
// stage freed by page pi - 2 are issued; at the end of the page each wave
// waits for its loads of page pi + 2 (issued one page earlier), so every
// load has two pages to land and the next page is complete a page before it
// is used.  One barrier per page.
template <bool kLazy, int kCur>
__device__ __forceinline__ void video_page(const VideoCtx& c, VideoState& st, int pi, int p_end) {
  const uint16_t* sk = stage_k<kCur>();
  const uint16_t* sv = stage_v<kCur>();
  pi = __builtin_amdgcn_readfirstlane(pi);
  const int n_valid = c.pages[pi].y;
  const int ahead = c.pages[ahead3(pi, p_end)].x;
  // both scalars are loaded before the barrier: a scalar load left for later
  // would share lgkmcnt with the LDS operand reads
  pin_sgpr(n_valid);
  __syncthreads();
  stage_dma(c, ahead, stage_k<(kCur + 3) % kStages>(), stage_v<(kCur + 3) % kStages>());
  __builtin_amdgcn_sched_barrier(0);
  const int half = c.half, l32 = c.l32;

  const float neg_m = -st.m_run;
  f32x16 s0, s1;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    s0[r] = neg_m;
    s1[r] = neg_m;
  }
  // page tail: register r of half h holds key 16*(r/8) + 8*h + r%8 (+32 in
  // s1); keys at or past n_valid become -inf
  const bool tail = n_valid < kPageTokens;
  auto mask_tail = [&](f32x16& sc, int key0) {
    const int lim = n_valid - key0 - 8 * half;
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (16 * (r >> 3) + (r & 7) >= lim) sc[r] = kNegInf;
  };
  // operand of S step n (n < 8: tile 0, else tile 1) and of P*V step n
  // (d tile n % 4, key chunk n / 4)
  auto kread = [&](int n) {
    const int row = n < 8 ? l32 : 32 + l32;
    return as_bf16x8(*reinterpret_cast<const u32x4*>(sk + row * kHeadDim + 8 * ((2 * (n & 7) + half) ^ (l32 & 15))));
  };
  auto vread = [&](int n) {
    const int d = 32 * (n & 3) + l32;
    return as_bf16x8(*reinterpret_cast<const u32x4*>(sv + d * kPageTokens + 8 * ((2 * (n >> 2) + half) ^ ((l32 >> 1) & 7))));
  };
  const bf16x2 ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
  // two exponentials of tile register pair n, packed to bf16 (word n of P),
  // added to the row sum
  auto exp_pair = [&](const f32x16& sc, int n, float& l) {
    // bit-cast a scalar temporary: a bit-cast of a vector element subscript
    // is lowered to element 0 by this compiler
    const uint32_t w = pack_bf16(fast_exp2(sc[2 * n]), fast_exp2(sc[2 * n + 1]));
    l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), ones, l, false);
    return w;
  };

  // Operand reads run kAhead MFMA steps ahead of their use, through a ring of
  // kAhead + 1 registers: S steps 0-15 (kread), then P*V steps 0-15 (vread).
  constexpr int kAhead = 4;
  auto oread = [&](int n) { return n < 16 ? kread(n) : vread(n - 16); };
  bf16x8 ring[kAhead + 1];
#pragma unroll
  for (int n = 0; n < kAhead; ++n) ring[n] = oread(n);
  auto next_operand = [&](int n) {  // operand of step n; issues the read of step n + kAhead
    if (n + kAhead < 32) ring[(n + kAhead) % (kAhead + 1)] = oread(n + kAhead);
    return ring[n % (kAhead + 1)];
  };

  // ---- A: S tile 0 ----
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int n = 0; n < 8; ++n) {
    const bf16x8 k = next_operand(n);
    s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k, c.qreg[n], s0, 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (tail) mask_tail(s0, 0);
  __builtin_amdgcn_sched_barrier(0);

  // ---- B: S tile 1, exponentials of tile 0 ----
  u32x4 p0a, p0b;
  float l0 = 0.f, mx0 = 0.f;
#pragma unroll
  for (int n = 0; n < 8; ++n) {
    const bf16x8 k = next_operand(8 + n);
    s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k, c.qreg[n], s1, 0, 0, 0);
    if (kLazy && n == 0) mx0 = pair_max(max16(s0));
    const uint32_t w = exp_pair(s0, n, l0);
    if (n < 4) p0a[n] = w; else p0b[n - 4] = w;
    __builtin_amdgcn_sched_barrier(0);
  }
  // d0: shift of the running maximum taken at tile 0 (0 for most rows)
  const bool need0 = kLazy && (st.first || mx0 > kLazyTau);
  const float d0 = need0 ? mx0 : 0.f;
  // keep the exponentials in the MFMA shadow they were scheduled in (the
  // compiler would otherwise sink them past the branches below)
  pin_vgpr(p0a);
  pin_vgpr(p0b);
  pin_vgpr(l0);
  if constexpr (kLazy) {
    if (__any(need0)) {
      const float alpha = fast_exp2(-d0);
      st.m_run += d0;
      st.l_run *= alpha;
      scale_o(st, alpha);
#pragma unroll
      for (int r = 0; r < 16; ++r) s0[r] -= d0;
      l0 = exp_tile(s0, p0a, p0b);
    }
    st.first = false;
  }
  st.l_run += l0;
  if (tail) mask_tail(s1, 32);
  __builtin_amdgcn_sched_barrier(0);

  // ---- D: P*V tile 0, exponentials of tile 1 ----
  u32x4 p1a, p1b;
  float l1 = 0.f, mx1 = 0.f;
#pragma unroll
  for (int n = 0; n < 8; ++n) {
    const bf16x8 v = next_operand(16 + n);
    const int t4 = n & 3;
    st.o[t4] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v, as_bf16x8(n < 4 ? p0a : p0b), st.o[t4], 0, 0, 0);
    if (kLazy && n == 0) mx1 = pair_max(max16(s1));
    const uint32_t w = exp_pair(s1, n, l1);
    if (n < 4) p1a[n] = w; else p1b[n - 4] = w;
    __builtin_amdgcn_sched_barrier(0);
  }
  // d1: shift of tile 1 relative to the page's starting maximum
  const bool need1 = kLazy && mx1 - d0 > kLazyTau;
  const float d1 = need1 ? mx1 : d0;
  pin_vgpr(p1a);
  pin_vgpr(p1b);
  pin_vgpr(l1);
  if constexpr (kLazy) {
    if (__any(d1 != 0.f)) {
      const float e = d1 - d0;
      const float alpha = fast_exp2(-e);
      st.m_run += e;
      st.l_run *= alpha;
      scale_o(st, alpha);
#pragma unroll
      for (int r = 0; r < 16; ++r) s1[r] -= d1;
      l1 = exp_tile(s1, p1a, p1b);
    }
  }
  st.l_run += l1;
  __builtin_amdgcn_sched_barrier(0);

  // ---- F: P*V tile 1 ----
#pragma unroll
  for (int n = 8; n < 16; ++n) {
    const bf16x8 v = next_operand(16 + n);
    const int t4 = n & 3;
    st.o[t4] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v, as_bf16x8(n < 12 ? p1a : p1b), st.o[t4], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
  wait_dma_all_but_last_page();
}

// Fixed-shift pages, software-pipelined across pages so that the softmax
// VALU work is spread over the MFMA steps (it then runs in the shadow of the
// matrix pipe instead of piling up in a few of them).  Iteration p (page p
// from LDS stage kCur, V^T of page p-1 from the stage before it), 32 MFMA
// steps with operand reads three steps ahead through a ring of four
// registers; the last three steps read the first operands of page p + 1
// (complete since the previous barrier), so the ring runs on across the page
// barrier.  Exponentials per step in brackets ("register r" is accumulator
// register r of a tile, in both lane halves; registers 0-7 are the tile's
// first 16 keys):
//   steps  0- 3  S tile 0 of p        [2: tile 1 of p-1, registers 0-3, 8-11]
//   steps  4- 7  S tile 0 of p        [1: tile 1 of p-1, registers 4-7]
//   steps  8-11  P*V of p-1, chunk 2  [1: tile 1 of p-1, registers 12-15]
//   steps 12-15  P*V of p-1, chunk 3  [1: tile 0 of p, registers 0-3]
//   steps 16-23  S tile 1 of p        [1: tile 0 of p, registers 4-11]
//   steps 24-27  P*V of p, chunk 0    [1: tile 0 of p, registers 12-15]
//   steps 28-31  P*V of p, chunk 1
// Every P word is complete before the P*V step that reads it, and the
// previous page's tile 1 is fully exponentiated (step 11) before this
// page's tile 1 is accumulated (step 16), so their registers need not be
// live together.  The first page of a range (kFirst) has no page p-1: steps
// 0-7 S tile 0, 8-15 S tile 1 with the exponentials of tile 0 keys 0-15,
// 16-23 P*V chunks 0-1 with those of keys 16-31.  Tile 1 of the last page is
// finished by video_flush.
constexpr int kRingAhead = 3;  // operand reads issued this many MFMA steps ahead
struct PipeState {
  f32x16 s1;      // S tile 1 of the previous page (exp2 argument)
  bf16x8 ring[kRingAhead + 1];  // operands in flight (slot = step % 4)
};

template <int kCur, bool kFirst>
__device__ __forceinline__ void video_iter(const VideoCtx& c, VideoState& st, PipeState& ps,
                                           const f32x16& s_init, int pi, int p_end) {
  constexpr int kPrev = (kCur + kStages - 1) % kStages;
  const uint16_t* sk = stage_k<kCur>();
  const uint16_t* sv = stage_v<kCur>();
  const uint16_t* svp = stage_v<kPrev>();
  constexpr int kNext = (kCur + 1) % kStages;
  const uint16_t* skn = stage_k<kNext>();
  pi = __builtin_amdgcn_readfirstlane(pi);
  const int ahead = c.pages[ahead3(pi, p_end)].x;
  const int n_valid = c.pages[pi].y;
  pin_sgpr(ahead);
  pin_sgpr(n_valid);
  __syncthreads();
  stage_dma(c, ahead, stage_k<(kCur + 3) % kStages>(), stage_v<(kCur + 3) % kStages>());
  __builtin_amdgcn_sched_barrier(0);
  const int half = c.half, l32 = c.l32;
  // Page tail (only a segment's last page is partly filled): logits of slots
  // at or past n_valid become -inf before their exponentials, so they weigh
  // exactly 0.  Register r of lane half h holds key 16 (r / 8) + 8 h + r % 8
  // (+32 in tile 1).  A correction subtracted from the row sum afterwards
  // would cancel catastrophically for rows whose logits all sit far below
  // the shift.
  const bool tail = n_valid < kPageTokens;
  auto mask_tail = [&](f32x16& sc, int key0) {
    const int lim = n_valid - key0 - 8 * half;
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (16 * (r >> 3) + (r & 7) >= lim) sc[r] = kNegInf;
  };
  auto kread_at = [&](const uint16_t* k, int n) {  // S k-step n % 8 of tile n / 8
    const int row = n < 8 ? l32 : 32 + l32;
    return as_bf16x8(*reinterpret_cast<const u32x4*>(k + row * kHeadDim + 8 * ((2 * (n & 7) + half) ^ (l32 & 15))));
  };
  auto kread = [&](int n) { return kread_at(sk, n); };
  auto vread = [&](const uint16_t* v, int t4, int jc) {  // d tile t4, key chunk jc
    const int d = 32 * t4 + l32;
    return as_bf16x8(*reinterpret_cast<const u32x4*>(v + d * kPageTokens + 8 * ((2 * jc + half) ^ ((l32 >> 1) & 7))));
  };
  constexpr int kSteps = kFirst ? 24 : 32;
  static_assert(kSteps % (kRingAhead + 1) == 0, "ring slots must line up across iterations");
  auto oread = [&](int o) {
    if (o >= kSteps) return kread_at(skn, o - kSteps);  // page p + 1, first S steps
    if (kFirst) return o < 16 ? kread(o) : vread(sv, (o - 16) & 3, (o - 16) >> 2);
    if (o < 8) return kread(o);
    if (o < 12) return vread(svp, o - 8, 2);
    if (o < 16) return vread(svp, o - 12, 3);
    if (o < 24) return kread(8 + o - 16);
    return vread(sv, (o - 24) & 3, (o - 24) >> 2);
  };
  constexpr int kAhead = kRingAhead;
  bf16x8* ring = ps.ring;
  if (kFirst) {  // the range's first page: nothing was read ahead
#pragma unroll
    for (int o = 0; o < kAhead; ++o) ring[o] = oread(o);
  }
  __builtin_amdgcn_sched_barrier(0);

  // The first MFMA of each S tile takes its accumulator input from s_init
  // (-m_run in every register), so the tiles start at the exp2 argument with
  // no per-page register initialisation.
  f32x16 s0, s1;
  const bf16x2 ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
  float l = 0.f;
  // P words: w[0..3] keys 0-15 of a tile (chunk 0 or 2), w[4..7] keys 16-31
  u32x4 pp2, pp3, p0, p1;  // tile 1 of p-1 (chunks 2, 3); tile 0 of p (chunks 0, 1)
  float e_lo = 0.f;        // first exponential of a pair, waiting for its partner
  float e2_lo = 0.f, e3_lo = 0.f;  // the same for the two halves of the previous tile 1
  auto exp_one = [&](const f32x16& sc, int r, u32x4& dst, int word) {
    const float e = fast_exp2(sc[r]);
    if ((r & 1) == 0) {
      e_lo = e;
    } else {
      // bit-cast a scalar temporary: a bit-cast of a vector element subscript
      // is lowered to element 0 by this compiler
      const uint32_t w = pack_bf16(e_lo, e);
      l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), ones, l, false);
      dst[word] = w;
    }
  };

#pragma unroll
  for (int o = 0; o < kSteps; ++o) {
    const bf16x8 a = ring[o % (kAhead + 1)];
    ring[(o + kAhead) % (kAhead + 1)] = oread(o + kAhead);
    if (kFirst) {
      if (o < 8) {
        s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, c.qreg[o], o == 0 ? s_init : s0, 0, 0, 0);
      } else if (o < 16) {
        s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, c.qreg[o - 8], o == 8 ? s_init : s1, 0, 0, 0);
        if (o == 8 && tail) mask_tail(s0, 0);
        exp_one(s0, o - 8, p0, (o - 8) >> 1);
      } else if (o < 20) {
        st.o[o - 16] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, as_bf16x8(p0), st.o[o - 16], 0, 0, 0);
        exp_one(s0, 8 + 2 * (o - 16), p1, o - 16);
        exp_one(s0, 9 + 2 * (o - 16), p1, o - 16);
      } else {
        st.o[o - 20] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, as_bf16x8(p1), st.o[o - 20], 0, 0, 0);
      }
    } else {
      // exponentials of the previous page's tile 1: registers 0-7 (key chunk
      // 2) one per step in steps 0-7, registers 8-11 a second one in steps
      // 0-3 and 12-15 one per step in 8-11, all done before the P*V of
      // chunks 2 and 3 reads them; those of this page's tile 0 one per step
      // in steps 12-27 (registers 0-7 before chunk 0 is read at step 24)
      auto prev_exp = [&](int r, u32x4& dst) {
        const float e = fast_exp2(ps.s1[r]);
        if ((r & 1) == 0) {
          if (r < 8) e2_lo = e; else e3_lo = e;
        } else {
          const uint32_t w = pack_bf16(r < 8 ? e2_lo : e3_lo, e);
          l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), ones, l, false);
          dst[(r & 7) >> 1] = w;
        }
      };
      if (o < 8) {
        s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, c.qreg[o], o == 0 ? s_init : s0, 0, 0, 0);
        prev_exp(o, pp2);
        if (o < 4) prev_exp(8 + o, pp3);
      } else if (o < 12) {
        st.o[o - 8] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, as_bf16x8(pp2), st.o[o - 8], 0, 0, 0);
        prev_exp(12 + o - 8, pp3);
      } else if (o < 16) {
        st.o[o - 12] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, as_bf16x8(pp3), st.o[o - 12], 0, 0, 0);
        if (o == 12 && tail) mask_tail(s0, 0);
        exp_one(s0, o - 12, p0, (o - 12) >> 1);
      } else if (o < 24) {
        s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, c.qreg[o - 16], o == 16 ? s_init : s1, 0, 0, 0);
        const int r = 4 + o - 16;
        exp_one(s0, r, r < 8 ? p0 : p1, (r & 7) >> 1);
      } else if (o < 28) {
        st.o[o - 24] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, as_bf16x8(p0), st.o[o - 24], 0, 0, 0);
        const int r = 12 + o - 24;
        exp_one(s0, r, p1, (r & 7) >> 1);
      } else {
        st.o[o - 28] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, as_bf16x8(p1), st.o[o - 28], 0, 0, 0);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  st.l_run += l;
  if (tail) mask_tail(s1, 32);
  ps.s1 = s1;
  wait_dma_all_but_last_page();
}

// Finishes tile 1 of the range's last page (V^T in LDS stage `stage`).
__device__ __forceinline__ void video_flush(const VideoCtx& c, VideoState& st, const PipeState& ps,
                                            int stage) {
  const uint16_t* sv = stage_v_at(stage);
  const int half = c.half, l32 = c.l32;
  u32x4 pa, pb;
  st.l_run += exp_tile(ps.s1, pa, pb);
#pragma unroll
  for (int n = 0; n < 8; ++n) {
    const int t4 = n & 3, jc = 2 + (n >> 2);
    const int d = 32 * t4 + l32;
    const bf16x8 v =
        as_bf16x8(*reinterpret_cast<const u32x4*>(sv + d * kPageTokens + 8 * ((2 * jc + half) ^ ((l32 >> 1) & 7))));
    st.o[t4] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v, as_bf16x8(n < 4 ? pa : pb), st.o[t4], 0, 0, 0);
  }
}

// One segment of a video workgroup's work: the query tile of rows
// [q_lo, min(q_lo + 256, q_hi)) of head `head` against entries
// [p_begin, p_end) of the call's page list, which is key range `seg` of the
// n_seg ranges that split this head's pages (q_hi ends the tile's query
// class).  With one range the output is written in bf16; otherwise the
// softmax-normalised partial and its log-sum-exp go to the split-KV
// workspace for the combine kernel.
struct VideoSeg {
  int head, p_begin, p_end, seg, n_seg, q_lo, q_hi;
};

__device__ __forceinline__ void video_segment(const AttnArgs& a, const VideoSeg& sg, bool first_segment) {
  // Lane-derived values (LDS and load offsets) are recomputed per segment:
  // kept live across the segment loop they would push the page loop into
  // register spills.
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = lane >> 5, l32 = lane & 31;
  const int head = sg.head, p_begin = sg.p_begin, p_end = sg.p_end;

  VideoCtx c;
  c.pages = page_list(a);
  c.page_stride = static_cast<int64_t>(a.num_heads) * kPageHeadElems;
  c.kpool = a.kpool + head * kPageHeadElems;
  c.vpool = a.vpool + head * kPageHeadElems;
  // The wave's rows: video rows of q, and at and past rq_row0 (the end of
  // the video rows) rider rows, the prepared rows of rq that see the same
  // pages; a wave may hold both.
  const int wrow = sg.q_lo + wave * 32;
  c.active = wrow < sg.q_hi || (a.n_rq > 0 && wrow < a.rq_row0 + a.n_rq && wrow + 32 > a.rq_row0);
  c.wave = wave;
  c.half = half;
  c.l32 = l32;
  {
    const int r0 = 4 * wave + (lane >> 4);  // K row of block i = 0
    c.dma_k = 2 * k_tile_index(swap23(r0), 8 * ((lane & 15) ^ (r0 & 15)));
    const int d0 = 8 * wave + (lane >> 3);  // V^T row of block i = 0
    c.dma_v = 2 * v_tile_index(8 * ((lane & 7) ^ ((d0 >> 1) & 7)), d0);
  }

  // Prologue loads, issued so that no dependent load waits behind an
  // unrelated one (vector memory counters complete in order): the page-list
  // entries of the first three pages are scalar loads; then every
  // independent vector load (positions, the page-list entries of the
  // key-norm scan, Q, gamma); then the direct loads of the first three pages
  // (a later segment first waits for every wave to be done with the
  // previous segment's stages); then the loads that depend on the first
  // batch (key norms, rotary table entries).
  int pg_first[3] = {0, 0, 0};
  if (p_begin < p_end) {
#pragma unroll
    for (int k = 0; k < 3; ++k) pg_first[k] = c.pages[min(p_begin + k, p_end - 1)].x;
  }
  const bool rider = a.n_rq > 0 && wrow + l32 >= a.rq_row0;  // the same in both halves of a row
  const int q = wrow + l32 - (rider ? a.rq_row0 : 0);
  const bool q_ok = q < (rider ? a.n_rq : sg.q_hi);
  const bool norm_rope = !rider && a.mode == 1;
  int3 qpos = make_int3(0, 0, 0);
  if (norm_rope && q_ok) qpos = make_int3(a.positions[3 * q], a.positions[3 * q + 1], a.positions[3 * q + 2]);
  // the segment's page-list entries (two per lane in the first pass)
  int pgl[2];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int pi = p_begin + lane + 64 * k;
    pgl[k] = pi < p_end ? c.pages[pi].x : -1;
  }
  u32x4 qraw[8];
  const uint16_t* qp = rider ? a.rq + q * a.rq_tok_stride + head * a.rq_head_stride + 8 * half
                             : a.q + q * a.q_tok_stride + head * a.q_head_stride + 8 * half;
#pragma unroll
  for (int s = 0; s < 8; ++s)
    qraw[s] = q_ok ? *reinterpret_cast<const u32x4*>(qp + 16 * s) : (u32x4){0u, 0u, 0u, 0u};
  float gam[8][8];
  if (norm_rope) {
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const float4 g0 = *reinterpret_cast<const float4*>(a.gamma + 16 * s + 8 * half);
      const float4 g1 = *reinterpret_cast<const float4*>(a.gamma + 16 * s + 8 * half + 4);
      gam[s][0] = g0.x; gam[s][1] = g0.y; gam[s][2] = g0.z; gam[s][3] = g0.w;
      gam[s][4] = g1.x; gam[s][5] = g1.y; gam[s][6] = g1.z; gam[s][7] = g1.w;
    }
  }
  if (!first_segment) __syncthreads();
  if (p_begin < p_end) {
    stage_dma(c, pg_first[0], g_k0, g_v0);
    stage_dma(c, pg_first[1], g_k1, g_v1);
    stage_dma(c, pg_first[2], g_k2, g_v2);
  }
  // key norms of the segment's pages
  float kn2 = 0.f;
#pragma unroll
  for (int k = 0; k < 2; ++k)
    if (pgl[k] >= 0) kn2 = fmaxf(kn2, a.knorm2[static_cast<int64_t>(pgl[k]) * a.num_heads + head]);
  for (int pi = p_begin + lane + 128; pi < p_end; pi += 64)  // segments longer than 128 pages
    kn2 = fmaxf(kn2, a.knorm2[static_cast<int64_t>(c.pages[pi].x) * a.num_heads + head]);

  // ---- Q prologue: lane holds Q''[q][16s + 8h + j], s = 0..7, j = 0..7 ----
  if (norm_rope) {
    int pt = 0, ph = 0, pw = 0;
    if (q_ok) clamp_pos(a.rope, qpos.x, qpos.y, qpos.z, a.flags, pt, ph, pw);
    float ss = 0.f;
#pragma unroll
    for (int s = 0; s < 8; ++s)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float x0 = bf16_lo(qraw[s][i]), x1 = bf16_hi(qraw[s][i]);
        ss += x0 * x0 + x1 * x1;
      }
    ss += __shfl_xor(ss, 32);
    const float inv = rsqrtf(ss * (1.0f / kHeadDim) + a.eps);
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int d0 = 16 * s + 8 * half;
      u32x4 w;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float y0 = bf16_lo(qraw[s][i]) * inv * gam[s][2 * i];
        const float y1 = bf16_hi(qraw[s][i]) * inv * gam[s][2 * i + 1];
        const float2 cs = rope_cs(a.rope, (d0 >> 1) + i, pt, ph, pw);
        w[i] = pack_bf16((y0 * cs.x - y1 * cs.y) * a.scale_log2, (y0 * cs.y + y1 * cs.x) * a.scale_log2);
      }
      c.qreg[s] = as_bf16x8(q_ok ? w : (u32x4){0u, 0u, 0u, 0u});
    }
  } else if (a.mode == 2 || rider) {  // prepared: Q'' as given
#pragma unroll
    for (int s = 0; s < 8; ++s) c.qreg[s] = as_bf16x8(qraw[s]);
  } else {
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      u32x4 w;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        w[i] = pack_bf16(bf16_lo(qraw[s][i]) * a.scale_log2, bf16_hi(qraw[s][i]) * a.scale_log2);
      c.qreg[s] = as_bf16x8(w);
    }
  }

  // ---- softmax shift ----
  // Logits arrive in the log2 domain (the scale and log2(e) are folded into
  // Q'').  By Cauchy-Schwarz every logit of row q is at most
  // B_q = |Q''_q| * max |k| over the segment's pages (knorm2 holds the
  // squared norms of the stored keys).  Softmax is shift invariant, so B_q
  // serves as the exp2 shift as it stands: p = exp2(s - B_q) <= 1, with no
  // running maximum and no rescale of O.  The row's largest p is at least
  // 2^(-2 B_q), so for B_q <= kShiftBoundMax every weight above 2^-46 of the
  // row maximum stays a normal bf16/fp32 number.  Otherwise the running
  // maximum is raised lazily: only when a 32-key tile exceeds it by more than
  // kLazyTau (p then stays below 2^kLazyTau), which makes the O rescale rare.
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) kn2 = fmaxf(kn2, __shfl_xor(kn2, o));
  float qn2 = 0.f;
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    const u32x4 w = __builtin_bit_cast(u32x4, c.qreg[s]);
#pragma unroll
    for (int i = 0; i < 4; ++i) qn2 += bf16_lo(w[i]) * bf16_lo(w[i]) + bf16_hi(w[i]) * bf16_hi(w[i]);
  }
  qn2 += __shfl_xor(qn2, 32);
  const float bound = sqrtf(qn2 * kn2);
  const bool fixed_shift = a.fixed_shift != 0 && __all(bound <= kShiftBoundMax);

  // ---- main loop over this segment's pages ----
  VideoState st;
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) st.o[t][r] = 0.f;
  st.m_run = fixed_shift ? bound : 0.f;
  st.l_run = 0.f;
  st.first = true;

  if (p_begin < p_end) wait_dma_all_but_last_page();
  if (c.active && fixed_shift) {
    if (p_begin < p_end) {
      PipeState ps;
      f32x16 s_init;
#pragma unroll
      for (int r = 0; r < 16; ++r) s_init[r] = -st.m_run;
      video_iter<0, true>(c, st, ps, s_init, p_begin, p_end);
      for (int pi = p_begin + 1; pi < p_end; pi += 5) {
        video_iter<1, false>(c, st, ps, s_init, pi, p_end);
        if (pi + 1 < p_end) video_iter<2, false>(c, st, ps, s_init, pi + 1, p_end);
        if (pi + 2 < p_end) video_iter<3, false>(c, st, ps, s_init, pi + 2, p_end);
        if (pi + 3 < p_end) video_iter<4, false>(c, st, ps, s_init, pi + 3, p_end);
        if (pi + 4 < p_end) video_iter<0, false>(c, st, ps, s_init, pi + 4, p_end);
      }
      video_flush(c, st, ps, (p_end - 1 - p_begin) % kStages);
    }
  } else if (c.active) {
    for (int pi = p_begin; pi < p_end; pi += 5) {
      video_page<true, 0>(c, st, pi, p_end);
      if (pi + 1 < p_end) video_page<true, 1>(c, st, pi + 1, p_end);
      if (pi + 2 < p_end) video_page<true, 2>(c, st, pi + 2, p_end);
      if (pi + 3 < p_end) video_page<true, 3>(c, st, pi + 3, p_end);
      if (pi + 4 < p_end) video_page<true, 4>(c, st, pi + 4, p_end);
    }
  } else {
    for (int pi = p_begin; pi < p_end; pi += 5) {
      video_page_stage_only<0>(c, pi, p_end);
      if (pi + 1 < p_end) video_page_stage_only<1>(c, pi + 1, p_end);
      if (pi + 2 < p_end) video_page_stage_only<2>(c, pi + 2, p_end);
      if (pi + 3 < p_end) video_page_stage_only<3>(c, pi + 3, p_end);
      if (pi + 4 < p_end) video_page_stage_only<4>(c, pi + 4, p_end);
    }
  }
  // no direct load may still be writing this workgroup's LDS when it exits
  wait_dma_all();

  // ---- epilogue: lane holds O^T[32t + 8g + 4h + i][q], g = r/4, i = r%4 ----
  const float l_tot = st.l_run + __shfl_xor(st.l_run, 32);
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
  if (rider) {  // always a partial, fp32, for the rider rows' own merge
    if (!q_ok) return;
    const int64_t row = (static_cast<int64_t>(sg.seg) * a.num_heads + head) * a.n_rq + q;
    float* po = a.rpart_o + row * kHeadDim;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 w = {st.o[t][4 * g] * inv, st.o[t][4 * g + 1] * inv, st.o[t][4 * g + 2] * inv,
                         st.o[t][4 * g + 3] * inv};
        *reinterpret_cast<f32x4*>(po + 32 * t + 8 * g + 4 * half) = w;
      }
    if (half == 0) a.rpart_lse[row] = l_tot > 0.f ? st.m_run + __log2f(l_tot) : kNegInf;
    return;
  }
  if (sg.n_seg == 1) {
    if (!q_ok) return;
    uint16_t* op = a.out + q * a.out_tok_stride + head * a.out_head_stride;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d0 = 32 * t + 8 * g + 4 * half;
        u32x2 w;
        w[0] = pack_bf16(st.o[t][4 * g] * inv, st.o[t][4 * g + 1] * inv);
        w[1] = pack_bf16(st.o[t][4 * g + 2] * inv, st.o[t][4 * g + 3] * inv);
        *reinterpret_cast<u32x2*>(op + d0) = w;
      }
    return;
  }
  // Partial of a key range: the softmax-normalised O rounded to bf16 (a
  // convex combination of V rows, so bf16 keeps its range; the merge adds at
  // most one more bf16 rounding of the output's size) and its fp32
  // log-sum-exp.  Half the bytes of fp32 partials, written here and read by
  // the combine kernel.
  if (!q_ok) return;
  const int64_t row = (static_cast<int64_t>(sg.seg) * a.num_heads + head) * a.n_q + q;
  uint16_t* po = reinterpret_cast<uint16_t*>(a.part_o) + row * kHeadDim;
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int d0 = 32 * t + 8 * g + 4 * half;
      u32x2 w;
      w[0] = pack_bf16(st.o[t][4 * g] * inv, st.o[t][4 * g + 1] * inv);
      w[1] = pack_bf16(st.o[t][4 * g + 2] * inv, st.o[t][4 * g + 3] * inv);
      *reinterpret_cast<u32x2*>(po + d0) = w;
    }
  if (half == 0) a.part_lse[row] = l_tot > 0.f ? st.m_run + __log2f(l_tot) : kNegInf;
}

// The call's query classes, read in place from the kernel arguments (the
// kernel's only argument is the AttnArgs; indexing the by-value argument at a
// run-time class would make the compiler copy it to private memory).
typedef const __attribute__((address_space(4))) AttnClass* const_class_table;
__device__ __forceinline__ const_class_table class_table() {
  const __attribute__((address_space(4))) char* seg =
      (const __attribute__((address_space(4))) char*)__builtin_amdgcn_kernarg_segment_ptr();
  return (const_class_table)(seg + offsetof(AttnArgs, cls));
}

__device__ __forceinline__ void rider_pages_wave(const AttnArgs& a, int head, int range0, int k, int n);

__global__ __launch_bounds__(kVideoWaves * 64) void unit_attn_kernel(const AttnArgs a) {
  // Work decode.  Each query class (the rows of one unit's queries, with the
  // pages its mask leaves visible) owns a block of workgroups: n_groups
  // groups of n_qtiles workgroups; group g takes a contiguous share of the
  // class's (head, page) units in head-major order (VideoPartition: even
  // shares of pages plus a cost per head started), one workgroup per query
  // tile, so the work fits a single round, and a share that crosses a head
  // boundary is processed as two segments.  Workgroups are dispatched
  // round-robin over the 8 XCDs; renumber so that consecutive work items
  // (the query tiles of a group, which read the same pages at the same time,
  // and neighbouring groups) run on one XCD and share its L2.
  const int nblk = gridDim.x, bid = blockIdx.x;
  const int xcd = bid & 7, per = nblk >> 3, rem = nblk & 7;
  const int item = xcd * per + min(xcd, rem) + (bid >> 3);
  const const_class_table tab = class_table();
  int ci = 0;
  for (int k = 1; k < a.n_classes; ++k)
    if (item >= tab[k].wg0) ci = k;
  const int local = item - tab[ci].wg0;
  const int n_qtiles = tab[ci].n_qtiles;
  const int q0 = tab[ci].q0, q_hi = q0 + tab[ci].n_q;
  const int page0 = tab[ci].page0;
  const int q_lo = q0 + (local % n_qtiles) * kVideoQTile;
  const int64_t group = local / n_qtiles;
  const int64_t n_pages = tab[ci].n_pages;
  if (n_pages == 0) {  // nothing visible: one empty segment per head, output 0
    if (group < a.num_heads)
      video_segment(a, VideoSeg{static_cast<int>(group), 0, 0, 0, 1, q_lo, q_hi}, true);
    return;
  }
  const VideoPartition part{a.num_heads, n_pages, a.seg_cost, tab[ci].n_groups};
  const int64_t lo = video_group_lo(part, group), hi = video_group_lo(part, group + 1);
  // The rider rows' own pages: in the last query tile's workgroup of the
  // group that holds a head's last page, the waves without rows of their
  // own (the last rx_waves of the 8) attend them for that head before they
  // join the page loop (where such waves only stage pages), as key ranges
  // after the head's ranges of the shared pages.
  if (a.rx_pages > 0 && local % n_qtiles == n_qtiles - 1 && lo < hi) {
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
    const int k = wave - (kVideoWaves - a.rx_waves);
    if (k >= 0) {
      for (int64_t head = lo / n_pages; head <= (hi - 1) / n_pages; ++head) {
        const int64_t h0 = head * n_pages;
        if (video_group_of(part, h0 + n_pages - 1) != group) continue;
        rider_pages_wave(a, static_cast<int>(head), static_cast<int>(group - video_group_of(part, h0) + 1), k,
                         a.rx_waves);
      }
    }
  }
  bool first = true;
  for (int64_t x = lo; x < hi; first = false) {
    const int64_t head = x / n_pages, h0 = head * n_pages;
    const int64_t x_end = min(hi, h0 + n_pages);
    const int64_t g_first = video_group_of(part, h0);
    const int64_t g_last = video_group_of(part, h0 + n_pages - 1);
    const VideoSeg sg{static_cast<int>(head), page0 + static_cast<int>(x - h0), page0 + static_cast<int>(x_end - h0),
                      static_cast<int>(group - g_first), static_cast<int>(g_last - g_first + 1), q_lo, q_hi};
    video_segment(a, sg, first);
    x = x_end;
  }
}

// ------------------------------------------------------------------------- //
// audio_attn: the few audio queries, memory-bound.  A workgroup of 4 waves
// takes one (head, 16-query tile, key range); wave w streams pages w, w + 4,
// ... of the range on its own (no LDS staging, no barriers), loading each
// page's valid K rows and V^T columns straight into registers in MFMA
// operand layout, and the four waves merge through LDS at the end.  Two
// workgroups fit a CU, so 8 independent waves per CU keep enough bytes in
// flight to stream the cache from HBM.  Each workgroup writes the partial of
// its key range; the combine kernel merges them.
//
// With lane l = 16 g + i (i = query column, g = lane group), per page:
//   S^T (16 keys x 16 queries) = K Q''^T  4 key tiles x 4 v_mfma_f32_16x16x32_bf16
//   O^T (16 d x 16 queries) += V^T P^T    8 d tiles x 2 key chunks, same MFMA
// Row m = 4 g' + r of key tile t holds key 32 (t/2) + 8 g' + 4 (t%2) + r, so
// that accumulator registers r of tiles 2c and 2c + 1 in lane group g are
// keys 32 c + 8 g + 0..7: exactly the B operand of the P*V MFMA of key chunk c.
// ------------------------------------------------------------------------- //
// Row m (lane index i) of key tile t: the key it holds.
__device__ __forceinline__ int audio_key(int t, int m) {
  return 32 * (t >> 1) + 8 * (m >> 2) + 4 * (t & 1) + (m & 3);
}

// Loads of one page's K operands, k[t][s] = K[key(t, i)][32 s + 8 g .. + 8],
// and V^T operands, v[dt][c] = V^T[16 dt + i][32 c + 8 g .. + 8].  Rows and
// columns past n_valid are read from the 1 KB zero block instead (a cache
// hit), so partly filled pages cost only their valid tokens in HBM traffic
// and no load is predicated.
__device__ __forceinline__ void audio_load_k(u32x4 (&k)[4][4], const uint16_t* kt, const uint16_t* zeros,
                                             int n_valid, int g, int i, int lane) {
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int key = audio_key(t, i);
    const uint16_t* src = key < n_valid ? kt + k_tile_index(key, 8 * g) : zeros + 8 * lane;
    const int step = key < n_valid ? k_tile_index(0, 32) : 0;  // next 32 d
#pragma unroll
    for (int s = 0; s < 4; ++s) k[t][s] = *reinterpret_cast<const u32x4*>(src + step * s);
  }
}
__device__ __forceinline__ void audio_load_v(u32x4 (&v)[8][2], const uint16_t* vt, const uint16_t* zeros,
                                             int n_valid, int g, int i, int lane) {
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const bool ok = 32 * c + 8 * g < n_valid;
    const uint16_t* src = ok ? vt + v_tile_index(32 * c + 8 * g, i) : zeros + 8 * lane;
    const int step = ok ? v_tile_index(0, 16) : 0;  // next 16 d
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) v[dt][c] = *reinterpret_cast<const u32x4*>(src + step * dt);
  }
}

// The page loop of the audio path, one wave: pages p_begin, p_begin + step,
// ... (< p_end) of the list, whose first page's operands kreg and vreg hold
// on entry.  Accumulates O^T (o), the running maximum and the row sum of the
// wave's 16 query columns (m_run and l_run as set up by the caller: the
// fixed shift, or -inf for a running maximum).
//
// Each page's K registers are reloaded (for the wave's next page) as soon as
// its S products are issued, and its V^T registers as soon as the P*V
// products are, so both loads of a page are in flight while the wave waits on
// the one before it.
__device__ __forceinline__ void audio_page_loop(const_page_list pages, int p_begin, int p_end, int step,
                                                const uint16_t* kpool, const uint16_t* vpool, int64_t page_stride,
                                                const uint16_t* zeros, const bf16x8 (&qreg)[4], bool fixed_shift,
                                                u32x4 (&kreg)[4][4], u32x4 (&vreg)[8][2], int g, int i16, int lane,
                                                f32x4 (&o)[8], float& m_run, float& l_run) {
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) o[dt] = (f32x4){0.f, 0.f, 0.f, 0.f};
  const bf16x2 ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
  for (int pi = p_begin; pi < p_end; pi += step) {
    const int n_valid = pages[pi].y;
    int2 nxt = make_int2(0, 0);  // past the last page: zeros
    if (pi + step < p_end) nxt = make_int2(pages[pi + step].x, pages[pi + step].y);
    // S^T of the page's four key tiles
    f32x4 sacc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      sacc[t] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < 4; ++s)
        sacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kreg[t][s]), qreg[s], sacc[t], 0, 0, 0);
    }
    audio_load_k(kreg, kpool + nxt.x * page_stride, zeros, nxt.y, g, i16, lane);
    if (n_valid < kPageTokens) {
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (audio_key(t, 4 * g + r) >= n_valid) sacc[t][r] = kNegInf;
    }
    float alpha = 1.f;
    if (!fixed_shift) {
      float mx = kNegInf;
#pragma unroll
      for (int t = 0; t < 4; ++t) mx = fmaxf(mx, fmaxf(fmaxf(sacc[t][0], sacc[t][1]), fmaxf(sacc[t][2], sacc[t][3])));
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx);
      alpha = m_new == kNegInf ? 1.f : fast_exp2(m_run - m_new);
      m_run = m_new;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) o[dt] *= alpha;
    }
    const float m_use = m_run == kNegInf ? 0.f : m_run;
    // P in bf16 (word c of chunk c: keys 32 c + 8 g + 0..7); the row sum is
    // taken over the same bf16 values the MFMAs consume
    u32x4 pw[2];
    float psum = 0.f;
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const f32x4& sc = sacc[2 * c + h];
        const uint32_t w0 = pack_bf16(fast_exp2(sc[0] - m_use), fast_exp2(sc[1] - m_use));
        const uint32_t w1 = pack_bf16(fast_exp2(sc[2] - m_use), fast_exp2(sc[3] - m_use));
        pw[c][2 * h] = w0;
        pw[c][2 * h + 1] = w1;
        psum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w0), ones, psum, false);
        psum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w1), ones, psum, false);
      }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int dt = 0; dt < 8; ++dt)
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vreg[dt][c]), as_bf16x8(pw[c]), o[dt], 0, 0, 0);
    audio_load_v(vreg, vpool + nxt.x * page_stride, zeros, nxt.y, g, i16, lane);
  }
}

// The rider rows over their own pages (entries rx_page0 .. rx_page0 + rx_pages
// of the page list) for one head, inside the video kernel: the audio path's
// page loop on all 8 waves (wave w takes pages w, w + 8, ...), 16 rider rows
// at a time, merged across the waves through the (then idle) LDS stages and
// written as key range `range` of the rows' fp32 partials.
// The rider rows over their own pages (entries rx_page0 .. rx_page0 + rx_pages
// of the page list) for one head, by one wave of the video kernel that has no
// rows of its own: the audio path's page loop over pages k, k + n, ... of
// them (wave k of n such waves), 16 rider rows at a time, each written as a
// key range of its own (range0 + k) of the rows' fp32 partials.  No LDS and
// no barrier: the wave does this before its first page barrier, while the
// waves with rows run their first segment's prologue.
__device__ __forceinline__ void rider_pages_wave(const AttnArgs& a, int head, int range0, int k, int n) {
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, i16 = lane & 15;
  const_page_list pages = page_list(a);
  const int64_t page_stride = static_cast<int64_t>(a.num_heads) * kPageHeadElems;
  const uint16_t* kpool = a.kpool + head * kPageHeadElems;
  const uint16_t* vpool = a.vpool + head * kPageHeadElems;
  const int p_begin = a.rx_page0 + k, p_end = a.rx_page0 + a.rx_pages;
  const int64_t row0 = (static_cast<int64_t>(range0 + k) * a.num_heads + head) * a.n_rq;
  for (int q0 = 0; q0 < a.n_rq; q0 += kAudioQTile) {
    u32x4 kreg[4][4], vreg[8][2];
    {
      int2 pg = make_int2(0, 0);
      if (p_begin < p_end) pg = make_int2(pages[p_begin].x, pages[p_begin].y);
      audio_load_k(kreg, kpool + pg.x * page_stride, a.zeros, pg.y, g, i16, lane);
      audio_load_v(vreg, vpool + pg.x * page_stride, a.zeros, pg.y, g, i16, lane);
    }
    const int q = q0 + i16;
    const bool q_ok = q < a.n_rq;
    bf16x8 qreg[4];
    const uint16_t* qp = a.rq + q * a.rq_tok_stride + head * a.rq_head_stride + 8 * g;
#pragma unroll
    for (int s = 0; s < 4; ++s)
      qreg[s] = as_bf16x8(q_ok ? *reinterpret_cast<const u32x4*>(qp + 32 * s) : (u32x4){0u, 0u, 0u, 0u});
    // softmax shift as in the audio kernel, over the wave's pages
    float kn2 = 0.f;
    for (int pi = p_begin + n * lane; pi < p_end; pi += 64 * n)
      kn2 = fmaxf(kn2, a.knorm2[static_cast<int64_t>(pages[pi].x) * a.num_heads + head]);
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) kn2 = fmaxf(kn2, __shfl_xor(kn2, off));
    float qn2 = 0.f;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const u32x4 w = __builtin_bit_cast(u32x4, qreg[s]);
#pragma unroll
      for (int j = 0; j < 4; ++j) qn2 += bf16_lo(w[j]) * bf16_lo(w[j]) + bf16_hi(w[j]) * bf16_hi(w[j]);
    }
    qn2 += __shfl_xor(qn2, 16);
    qn2 += __shfl_xor(qn2, 32);
    const float bound = sqrtf(qn2 * kn2);
    const bool fixed_shift = a.fixed_shift != 0 && __all(bound <= kShiftBoundMax);
    float m_run = fixed_shift ? bound : kNegInf, l_run = 0.f;
    f32x4 o[8];
    audio_page_loop(pages, p_begin, p_end, n, kpool, vpool, page_stride, a.zeros, qreg, fixed_shift, kreg, vreg,
                    g, i16, lane, o, m_run, l_run);
    // lane holds O^T[16 dt + 4 g + r][q] of the wave's pages
    float l_w = l_run + __shfl_xor(l_run, 16);
    l_w += __shfl_xor(l_w, 32);
    if (q_ok) {
      const float inv = l_w > 0.f ? 1.0f / l_w : 0.f;
      float* po = a.rpart_o + (row0 + q) * kHeadDim;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt)
        *reinterpret_cast<f32x4*>(po + 16 * dt + 4 * g) = o[dt] * inv;
      if (g == 0) a.rpart_lse[row0 + q] = l_w > 0.f ? m_run + __log2f(l_w) : kNegInf;
    }
  }
}

__global__ __launch_bounds__(256, 2) void audio_attn_kernel(const AttnArgs a) {
  __shared__ float sm_o[4][kHeadDim][16];  // per wave O^T, merged at the end
  __shared__ float sm_ml[4][2][16];        // per wave (m, l) per query
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, i16 = lane & 15;
  const int bid = blockIdx.x;
  const int split = bid % a.n_splits;
  const int rest = bid / a.n_splits;
  const int qtile = rest % a.n_qtiles;
  const int head = rest / a.n_qtiles;
  const int p_begin = split * a.pages_per_split + wave;
  const int p_end = min(a.n_pages, (split + 1) * a.pages_per_split);
  const_page_list pages = page_list(a);
  const int64_t page_stride = static_cast<int64_t>(a.num_heads) * kPageHeadElems;
  const uint16_t* kpool = a.kpool + head * kPageHeadElems;
  const uint16_t* vpool = a.vpool + head * kPageHeadElems;

  // the wave's first page is requested before the query prologue
  u32x4 kreg[4][4], vreg[8][2];
  {
    int2 pg = make_int2(0, 0);  // no page: zeros
    if (p_begin < p_end) pg = make_int2(pages[p_begin].x, pages[p_begin].y);
    audio_load_k(kreg, kpool + pg.x * page_stride, a.zeros, pg.y, g, i16, lane);
    audio_load_v(vreg, vpool + pg.x * page_stride, a.zeros, pg.y, g, i16, lane);
  }

  // Q prologue: lane holds Q''[q][32 s + 8 g + j], s = 0..3, with the
  // softmax scale and log2(e) folded in
  const int q = qtile * kAudioQTile + i16;
  const bool q_ok = q < a.n_q;
  u32x4 qraw[4];
  const uint16_t* qp = a.q + q * a.q_tok_stride + head * a.q_head_stride + 8 * g;
#pragma unroll
  for (int s = 0; s < 4; ++s)
    qraw[s] = q_ok ? *reinterpret_cast<const u32x4*>(qp + 32 * s) : (u32x4){0u, 0u, 0u, 0u};
  bf16x8 qreg[4];
  if (a.mode == 1) {
    int pt = 0, ph = 0, pw = 0;
    if (q_ok) load_pos(a.rope, a.positions, q, a.flags, pt, ph, pw);
    float ss = 0.f;
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float x0 = bf16_lo(qraw[s][k]), x1 = bf16_hi(qraw[s][k]);
        ss += x0 * x0 + x1 * x1;
      }
    ss += __shfl_xor(ss, 16);
    ss += __shfl_xor(ss, 32);
    const float inv = rsqrtf(ss * (1.0f / kHeadDim) + a.eps);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int d0 = 32 * s + 8 * g;
      const float4 g0 = *reinterpret_cast<const float4*>(a.gamma + d0);
      const float4 g1 = *reinterpret_cast<const float4*>(a.gamma + d0 + 4);
      const float gg[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
      u32x4 w;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float y0 = bf16_lo(qraw[s][k]) * inv * gg[2 * k];
        const float y1 = bf16_hi(qraw[s][k]) * inv * gg[2 * k + 1];
        const float2 cs = rope_cs(a.rope, (d0 >> 1) + k, pt, ph, pw);
        w[k] = pack_bf16((y0 * cs.x - y1 * cs.y) * a.scale_log2, (y0 * cs.y + y1 * cs.x) * a.scale_log2);
      }
      qreg[s] = as_bf16x8(q_ok ? w : (u32x4){0u, 0u, 0u, 0u});
    }
  } else if (a.mode == 2) {  // prepared: Q'' as given
#pragma unroll
    for (int s = 0; s < 4; ++s) qreg[s] = as_bf16x8(qraw[s]);
  } else {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      u32x4 w;
#pragma unroll
      for (int k = 0; k < 4; ++k)
        w[k] = pack_bf16(bf16_lo(qraw[s][k]) * a.scale_log2, bf16_hi(qraw[s][k]) * a.scale_log2);
      qreg[s] = as_bf16x8(w);
    }
  }

  // Softmax shift, as in the video kernel: the logit bound |Q''_q| max |k|
  // (log2 units) over the wave's pages when it is at most kShiftBoundMax for
  // all 16 queries, else a running maximum.
  float kn2 = 0.f;
  for (int pi = p_begin + 4 * lane; pi < p_end; pi += 256)
    kn2 = fmaxf(kn2, a.knorm2[static_cast<int64_t>(pages[pi].x) * a.num_heads + head]);
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) kn2 = fmaxf(kn2, __shfl_xor(kn2, off));
  float qn2 = 0.f;
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const u32x4 w = __builtin_bit_cast(u32x4, qreg[s]);
#pragma unroll
    for (int k = 0; k < 4; ++k) qn2 += bf16_lo(w[k]) * bf16_lo(w[k]) + bf16_hi(w[k]) * bf16_hi(w[k]);
  }
  qn2 += __shfl_xor(qn2, 16);
  qn2 += __shfl_xor(qn2, 32);
  const float bound = sqrtf(qn2 * kn2);
  const bool fixed_shift = a.fixed_shift != 0 && __all(bound <= kShiftBoundMax);
  float m_run = fixed_shift ? bound : kNegInf, l_run = 0.f;

  f32x4 o[8];
  audio_page_loop(pages, p_begin, p_end, 4, kpool, vpool, page_stride, a.zeros, qreg, fixed_shift, kreg, vreg,
                  g, i16, lane, o, m_run, l_run);

  // merge the four waves: lane holds O^T[16 dt + 4 g + r][q] of its keys
  float l_w = l_run + __shfl_xor(l_run, 16);
  l_w += __shfl_xor(l_w, 32);
#pragma unroll
  for (int dt = 0; dt < 8; ++dt)
#pragma unroll
    for (int r = 0; r < 4; ++r) sm_o[wave][16 * dt + 4 * g + r][i16] = o[dt][r];
  if (g == 0) {
    sm_ml[wave][0][i16] = m_run;
    sm_ml[wave][1][i16] = l_w;
  }
  __syncthreads();
  // thread t: query t % 16, d = 8 (t / 16) .. + 8
  const int qi = tid & 15, d0 = 8 * (tid >> 4);
  float mw[4], big = kNegInf;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    mw[w] = sm_ml[w][0][qi];
    big = fmaxf(big, mw[w]);
  }
  float ew[4], l_tot = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    ew[w] = big == kNegInf ? 0.f : fast_exp2(mw[w] - big);
    l_tot += ew[w] * sm_ml[w][1][qi];
  }
  const int qq = qtile * kAudioQTile + qi;
  if (qq >= a.n_q) return;
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
  const int64_t row = (static_cast<int64_t>(split) * a.num_heads + head) * a.n_q + qq;
  float* po = a.part_o + row * kHeadDim + d0;
  f32x4 out0, out1;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) v += ew[w] * sm_o[w][d0 + k][qi];
    if (k < 4) out0[k] = v * inv; else out1[k - 4] = v * inv;
  }
  *reinterpret_cast<f32x4*>(po) = out0;
  *reinterpret_cast<f32x4*>(po + 4) = out1;
  if (tid < 16) a.part_lse[row] = l_tot > 0.f ? big + __log2f(l_tot) : kNegInf;
}

// ------------------------------------------------------------------------- //
// combine (audio key ranges): 16 threads per (head, query) row, 8 d each, 16
// rows per block.  A thread reads the row's log-sum-exps, then requests the
// 8 values of kMergeBatch ranges before using any (one memory round trip per
// batch) and folds them against the largest.  The batch sets the registers a
// thread holds: the audio call's own merge takes 16 ranges at once; inside
// the merge launch of a step, whose video rows need few registers, 3 (more
// would cap the occupancy of the video rows' blocks).
// ------------------------------------------------------------------------- //
template <int kMergeBatch>
__device__ __forceinline__ void combine_block(const CombineArgs& a, int bid) {
  const int lane = threadIdx.x & 15;
  const int row = bid * 16 + (threadIdx.x >> 4);
  if (row >= a.num_heads * a.n_q) return;
  const int head = row / a.n_q, q = row % a.n_q;
  int n_splits = a.n_splits;
  if (a.r_groups > 0) {  // the ranges the video kernel wrote for rider rows
    const VideoPartition part{a.num_heads, a.r_pages, a.seg_cost, a.r_groups};
    const int64_t h0 = static_cast<int64_t>(head) * a.r_pages;
    n_splits += static_cast<int>(video_group_of(part, h0 + a.r_pages - 1) - video_group_of(part, h0) + 1) +
                a.r_extra;  // and those of the rows' own pages
  }
  const int d0 = 8 * lane;
  const int64_t split_stride = static_cast<int64_t>(a.num_heads) * a.n_q;
  // The largest log-sum-exp first: every range is then weighted the same way
  // whatever the batch, so the step's merge launch and the audio call's own
  // give the same bits.  (With all ranges in one batch it comes from that
  // batch's loads.)
  float mx = kNegInf;
  for (int sp0 = 0; n_splits > kMergeBatch && sp0 < n_splits; sp0 += 16) {
    float lb[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) lb[i] = sp0 + i < n_splits ? a.part_lse[(sp0 + i) * split_stride + row] : kNegInf;
#pragma unroll
    for (int i = 0; i < 16; ++i) mx = fmaxf(mx, lb[i]);
  }
  float wsum = 0.f;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int sp0 = 0; sp0 < n_splits; sp0 += kMergeBatch) {
    float lb[kMergeBatch];
    f32x4 o0[kMergeBatch], o1[kMergeBatch];
#pragma unroll
    for (int i = 0; i < kMergeBatch; ++i) {
      const int sp = sp0 + i;
      const bool ok = sp < n_splits;
      const float* po = a.part_o + (sp * split_stride + row) * kHeadDim + d0;
      lb[i] = ok ? a.part_lse[sp * split_stride + row] : kNegInf;
      o0[i] = ok ? *reinterpret_cast<const f32x4*>(po) : (f32x4){0.f, 0.f, 0.f, 0.f};
      o1[i] = ok ? *reinterpret_cast<const f32x4*>(po + 4) : (f32x4){0.f, 0.f, 0.f, 0.f};
    }
    if (n_splits <= kMergeBatch) {
#pragma unroll
      for (int i = 0; i < kMergeBatch; ++i) mx = fmaxf(mx, lb[i]);
    }
    if (mx == kNegInf) break;
#pragma unroll
    for (int i = 0; i < kMergeBatch; ++i) {
      const float w = lb[i] == kNegInf ? 0.f : fast_exp2(lb[i] - mx);
      wsum += w;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        acc[k] += w * o0[i][k];
        acc[4 + k] += w * o1[i][k];
      }
    }
  }
  const float inv = mx != kNegInf ? 1.0f / wsum : 0.f;
  u32x4 w;
#pragma unroll
  for (int k = 0; k < 4; ++k) w[k] = pack_bf16(acc[2 * k] * inv, acc[2 * k + 1] * inv);
  *reinterpret_cast<u32x4*>(a.out + q * a.out_tok_stride + head * a.out_head_stride + d0) = w;
}

__global__ __launch_bounds__(256) void combine_kernel(const CombineArgs a) { combine_block<16>(a, blockIdx.x); }

// ------------------------------------------------------------------------- //
// video_combine: merges the key ranges of the video schedule.  A head's
// range count follows from the groups' shares (VideoPartition; a head
// in one range was written in bf16 by the attention kernel: nothing to
// merge).  16 threads per (head, query) row, 8 d each (16-byte loads), 16
// rows per block; all of a row's (at most kMaxVideoSplits) partials are
// requested before any is used.
// ------------------------------------------------------------------------- //
__device__ __forceinline__ void video_combine_block(const CombineArgs& a, const_class_table tab, int bid) {
  const int lane = threadIdx.x & 15;
  const int row = bid * 16 + (threadIdx.x >> 4);
  if (row >= a.num_heads * a.n_q) return;
  const int head = row / a.n_q, q = row % a.n_q;
  // the row's query class: every table entry is read with uniform (scalar)
  // loads and the row's fields are selected per lane
  int32_t cls_pages = tab[0].n_pages, cls_groups = tab[0].n_groups;
  for (int k = 1; k < a.n_classes; ++k) {
    const bool in = q >= tab[k].q0;
    cls_pages = in ? tab[k].n_pages : cls_pages;
    cls_groups = in ? tab[k].n_groups : cls_groups;
  }
  const int64_t n_pages = cls_pages;
  if (n_pages == 0) return;
  const VideoPartition part{a.num_heads, n_pages, a.seg_cost, cls_groups};
  const int64_t h0 = static_cast<int64_t>(head) * n_pages;
  const int n_ranges = static_cast<int>(video_group_of(part, h0 + n_pages - 1) - video_group_of(part, h0) + 1);
  if (n_ranges < 2) return;
  const int d0 = 8 * lane;
  const int64_t split_stride = static_cast<int64_t>(a.num_heads) * a.n_q;
  const uint16_t* po = reinterpret_cast<const uint16_t*>(a.part_o);
  float l[kMaxVideoSplits];
  u32x4 w[kMaxVideoSplits];
#pragma unroll
  for (int sp = 0; sp < kMaxVideoSplits; ++sp) {
    if (sp < n_ranges) {
      l[sp] = a.part_lse[sp * split_stride + row];
      w[sp] = *reinterpret_cast<const u32x4*>(po + (sp * split_stride + row) * kHeadDim + d0);
    } else {
      l[sp] = kNegInf;
      w[sp] = (u32x4){0u, 0u, 0u, 0u};
    }
  }
  float mx = kNegInf;
#pragma unroll
  for (int sp = 0; sp < kMaxVideoSplits; ++sp) mx = fmaxf(mx, l[sp]);
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (mx != kNegInf) {
    float wsum = 0.f;
#pragma unroll
    for (int sp = 0; sp < kMaxVideoSplits; ++sp) {
      if (l[sp] == kNegInf) continue;
      const float e = fast_exp2(l[sp] - mx);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[2 * i] += e * bf16_lo(w[sp][i]);
        acc[2 * i + 1] += e * bf16_hi(w[sp][i]);
      }
      wsum += e;
    }
    const float inv = 1.0f / wsum;
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] *= inv;
  }
  u32x4 o;
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = pack_bf16(acc[2 * i], acc[2 * i + 1]);
  *reinterpret_cast<u32x4*>(a.out + q * a.out_tok_stride + head * a.out_head_stride + d0) = o;
}

// The class table of the video CombineArgs, which is the first kernel
// argument of both merge kernels below, read in place.
__device__ __forceinline__ const_class_table combine_class_table() {
  const __attribute__((address_space(4))) char* seg =
      (const __attribute__((address_space(4))) char*)__builtin_amdgcn_kernarg_segment_ptr();
  return (const_class_table)(seg + offsetof(CombineArgs, cls));
}

__global__ __launch_bounds__(256) void video_combine_kernel(const CombineArgs a) {
  video_combine_block(a, combine_class_table(), blockIdx.x);
}

// The merges of one step's video and audio calls in one launch: blocks below
// n_audio merge audio rows (they start first: their rows fold more ranges),
// the rest video rows.
__global__ __launch_bounds__(256) void step_combine_kernel(const CombineArgs v, const CombineArgs au,
                                                           int n_audio) {
  if (static_cast<int>(blockIdx.x) < n_audio)
    combine_block<3>(au, blockIdx.x);
  else
    video_combine_block(v, combine_class_table(), blockIdx.x - n_audio);
}

}  // namespace

// The no-allocation entry point's split-KV workspace.  Host code never
// passes this name to a kernel or a copy (in host code it is only a stand-in
// for the symbol): it uses the device address static_scratch() looks up.
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

hipError_t static_scratch(void** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

// With start or stop events, a launch goes through hipExtLaunchKernelGGL,
// whose events take the dispatch's own start and end timestamps (the
// kernel's execution, without the queue's event processing around it).
hipError_t launch_kv_append(const AppendArgs& a, hipStream_t stream, hipEvent_t start, hipEvent_t stop) {
  const int tiles = a.n_blocks * a.num_heads;
  const int grid = std::min(tiles, std::max(1, a.grid_blocks));
  if (start || stop)
    hipExtLaunchKernelGGL(kv_append_kernel, dim3(grid), dim3(256), 0, stream, start, stop, 0, a);
  else
    hipLaunchKernelGGL(kv_append_kernel, dim3(grid), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_unit_attention(const AttnArgs& a, hipStream_t stream, hipEvent_t start, hipEvent_t stop) {
  const dim3 grid(a.n_wg), block(kVideoWaves * 64);
  if (start || stop)
    hipExtLaunchKernelGGL(unit_attn_kernel, grid, block, 0, stream, start, stop, 0, a);
  else
    hipLaunchKernelGGL(unit_attn_kernel, grid, block, 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_audio_attention(const AttnArgs& a, hipStream_t stream, hipEvent_t start, hipEvent_t stop) {
  const dim3 grid(a.num_heads * a.n_qtiles * a.n_splits);
  if (start || stop)
    hipExtLaunchKernelGGL(audio_attn_kernel, grid, dim3(256), 0, stream, start, stop, 0, a);
  else
    hipLaunchKernelGGL(audio_attn_kernel, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_step_combine(const CombineArgs& v, const CombineArgs& au, hipStream_t stream) {
  const int n_video = v.n_groups > 0 ? (v.num_heads * v.n_q + 15) / 16 : 0;
  const int n_audio = au.num_heads > 0 ? (au.num_heads * au.n_q + 15) / 16 : 0;
  if (n_video + n_audio == 0) return hipSuccess;
  hipLaunchKernelGGL(step_combine_kernel, dim3(n_video + n_audio), dim3(256), 0, stream, v, au, n_audio);
  return hipGetLastError();
}

hipError_t launch_combine(const CombineArgs& a, hipStream_t stream) {
  const int rows = a.num_heads * a.n_q;
  if (a.n_groups > 0)
    hipLaunchKernelGGL(video_combine_kernel, dim3((rows + 15) / 16), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(combine_kernel, dim3((rows + 15) / 16), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ws
