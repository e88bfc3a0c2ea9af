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
#include "ws_kernels.hpp"

namespace ws {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kNegInf = -__builtin_inff();

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

// ------------------------------------------------------------------------- //
// kv_append: grid (pages of this launch, heads), 256 threads.
// ------------------------------------------------------------------------- //
template <int kMode>
__global__ __launch_bounds__(256) void kv_append_kernel(const AppendArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t vt[kPageTokens][kHeadDim + 8];
  const int head = blockIdx.y;
  const int page = a.pages[blockIdx.x];
  const int tok0 = (a.first_page + blockIdx.x) * kPageTokens;
  const int64_t tile = (static_cast<int64_t>(page) * a.num_heads + head) * kPageHeadElems;
  uint16_t* kdst = a.kpool + tile;
  uint16_t* vdst = a.vpool + tile;
  const int t = threadIdx.x;

  // K: 16 threads per token row, 8 consecutive d each; 16 rows per pass.
  const int c = t & 15;
  const int rr = t >> 4;
  float g[8];
  if (kMode == 1) {
    const float4 g0 = *reinterpret_cast<const float4*>(a.gamma + 8 * c);
    const float4 g1 = *reinterpret_cast<const float4*>(a.gamma + 8 * c + 4);
    g[0] = g0.x; g[1] = g0.y; g[2] = g0.z; g[3] = g0.w;
    g[4] = g1.x; g[5] = g1.y; g[6] = g1.z; g[7] = g1.w;
  }
#pragma unroll
  for (int pass = 0; pass < 4; ++pass) {
    const int slot = pass * 16 + rr;
    const int tok = tok0 + slot;
    const bool valid = tok < a.n_tokens;
    u32x4 x = {0u, 0u, 0u, 0u};
    if (valid)
      x = *reinterpret_cast<const u32x4*>(a.k + tok * a.tok_stride + head * a.head_stride + 8 * c);
    u32x4 y = x;
    if (kMode == 1) {
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
      const float inv = rsqrtf(ss * (1.0f / kHeadDim) + a.eps);
      int pt = 0, ph = 0, pw = 0;
      if (valid) load_pos(a.rope, a.positions, tok, a.flags, pt, ph, pw);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float y0 = f[2 * i] * inv * g[2 * i];
        const float y1 = f[2 * i + 1] * inv * g[2 * i + 1];
        const float2 cs = rope_cs(a.rope, 4 * c + i, pt, ph, pw);
        y[i] = pack_bf16(y0 * cs.x - y1 * cs.y, y0 * cs.y + y1 * cs.x);
      }
      if (!valid) y = (u32x4){0u, 0u, 0u, 0u};
    }
    *reinterpret_cast<u32x4*>(kdst + slot * kHeadDim + 8 * c) = y;
  }

  // V: stage [slot][d] in LDS, write [d][slot].
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ch = t + 256 * i;
    const int slot = ch >> 4, dc = ch & 15;
    const int tok = tok0 + slot;
    u32x4 x = {0u, 0u, 0u, 0u};
    if (tok < a.n_tokens)
      x = *reinterpret_cast<const u32x4*>(a.v + tok * a.tok_stride + head * a.head_stride + 8 * dc);
    *reinterpret_cast<u32x4*>(&vt[slot][8 * dc]) = x;
  }
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
    *reinterpret_cast<u32x4*>(vdst + d * kPageTokens + 8 * tc) = y;
  }
}

// ------------------------------------------------------------------------- //
// unit_attn (video): 4 waves x 32 queries, 64-key pages through LDS.
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
// LDS chunk swizzles (16-byte chunks): conflict-free MFMA operand reads.
__device__ __forceinline__ int swz_k(int row, int chunk) { return chunk ^ swap23(row & 15); }
__device__ __forceinline__ int swz_v(int d, int chunk) { return chunk ^ ((d ^ (d >> 3)) & 7); }

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

struct VideoSmem {
  uint16_t k[2][kPageTokens * kHeadDim];
  uint16_t v[2][kHeadDim * kPageTokens];
};

__global__ __launch_bounds__(256, 2) void unit_attn_kernel(const AttnArgs a) {
  __shared__ __attribute__((aligned(16))) VideoSmem sm;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;

  // Work decode.  Workgroups are dispatched round-robin over the 8 XCDs;
  // renumber so that each XCD owns a contiguous run of (head, q-tile, split)
  // items, i.e. whole heads, whose K/V pages then stay in that XCD's L2.
  const int nblk = gridDim.x, bid = blockIdx.x;
  const int xcd = bid & 7, per = nblk >> 3, rem = nblk & 7;
  const int item = xcd * per + min(xcd, rem) + (bid >> 3);
  const int split = item % a.n_splits;
  const int rest = item / a.n_splits;
  const int qtile = rest % a.n_qtiles;
  const int head = rest / a.n_qtiles;
  const int p_begin = split * a.pages_per_split;
  const int p_end = min(a.n_pages, p_begin + a.pages_per_split);

  // ---- Q prologue: lane holds Q'[q][16s + 8h + j], s = 0..7, j = 0..7 ----
  const int q = qtile * kVideoQTile + wave * 32 + l32;
  const bool q_ok = q < a.n_q;
  u32x4 qraw[8];
  const uint16_t* qp = a.q + q * a.q_tok_stride + head * a.q_head_stride + 8 * half;
#pragma unroll
  for (int s = 0; s < 8; ++s)
    qraw[s] = q_ok ? *reinterpret_cast<const u32x4*>(qp + 16 * s) : (u32x4){0u, 0u, 0u, 0u};
  bf16x8 qreg[8];
  if (a.mode == 1) {
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
    int pt = 0, ph = 0, pw = 0;
    if (q_ok) load_pos(a.rope, a.positions, q, a.flags, pt, ph, pw);
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int d0 = 16 * s + 8 * half;
      const float4 g0 = *reinterpret_cast<const float4*>(a.gamma + d0);
      const float4 g1 = *reinterpret_cast<const float4*>(a.gamma + d0 + 4);
      const float g[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
      u32x4 w;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float y0 = bf16_lo(qraw[s][i]) * inv * g[2 * i];
        const float y1 = bf16_hi(qraw[s][i]) * inv * g[2 * i + 1];
        const float2 cs = rope_cs(a.rope, (d0 >> 1) + i, pt, ph, pw);
        w[i] = pack_bf16(y0 * cs.x - y1 * cs.y, y0 * cs.y + y1 * cs.x);
      }
      qreg[s] = as_bf16x8(q_ok ? w : (u32x4){0u, 0u, 0u, 0u});
    }
  } else {
#pragma unroll
    for (int s = 0; s < 8; ++s) qreg[s] = as_bf16x8(qraw[s]);
  }

  // ---- main loop over this split's pages ----
  f32x16 o[4];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[t][r] = 0.f;
  float m_run = kNegInf, l_run = 0.f;
  const float c = a.scale_log2;
  const int krow = swap23(l32);

  u32x4 kst[4], vst[4];
  auto gload = [&](int pi) {
    const int page = a.pages[pi].x;
    const int64_t tileo = (static_cast<int64_t>(page) * a.num_heads + head) * kPageHeadElems;
    const u32x4* kb = reinterpret_cast<const u32x4*>(a.kpool + tileo);
    const u32x4* vb = reinterpret_cast<const u32x4*>(a.vpool + tileo);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      kst[i] = kb[tid + 256 * i];
      vst[i] = vb[tid + 256 * i];
    }
  };
  if (p_begin < p_end) gload(p_begin);

  for (int pi = p_begin; pi < p_end; ++pi) {
    const int buf = (pi - p_begin) & 1;
    uint16_t* sk = sm.k[buf];
    uint16_t* sv = sm.v[buf];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int ch = tid + 256 * i;
      const int kr = ch >> 4, kc = ch & 15;
      *reinterpret_cast<u32x4*>(sk + kr * kHeadDim + 8 * swz_k(kr, kc)) = kst[i];
      const int vd = ch >> 3, vc = ch & 7;
      *reinterpret_cast<u32x4*>(sv + vd * kPageTokens + 8 * swz_v(vd, vc)) = vst[i];
    }
    __syncthreads();
    const int n_valid = a.pages[pi].y;
    if (pi + 1 < p_end) gload(pi + 1);

    // S^T = K Q'^T
    f32x16 s0, s1;
#pragma unroll
    for (int r = 0; r < 16; ++r) { s0[r] = 0.f; s1[r] = 0.f; }
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int ck = 2 * s + half;
      const bf16x8 ka = as_bf16x8(
          *reinterpret_cast<const u32x4*>(sk + krow * kHeadDim + 8 * swz_k(krow, ck)));
      const bf16x8 kb = as_bf16x8(
          *reinterpret_cast<const u32x4*>(sk + (32 + krow) * kHeadDim + 8 * swz_k(krow, ck)));
      s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qreg[s], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kb, qreg[s], s1, 0, 0, 0);
    }

    // page tail: register r of half h holds key 16*(r/8) + 8*h + r%8 (+32 in s1)
    if (n_valid < kPageTokens) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 16 * (r >> 3) + 8 * half + (r & 7);
        if (key >= n_valid) s0[r] = kNegInf;
        if (key + 32 >= n_valid) s1[r] = kNegInf;
      }
    }

    // online softmax (exp2 domain, scale folded into c)
    float mx = kNegInf;
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, fmaxf(s0[r], s1[r]));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == kNegInf) ? 0.f : m_new;
    const float alpha = fast_exp2((m_run - m_use) * c);
    const float mc = m_use * c;
    float psum = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      s0[r] = fast_exp2(__builtin_fmaf(s0[r], c, -mc));
      s1[r] = fast_exp2(__builtin_fmaf(s1[r], c, -mc));
      psum += s0[r] + s1[r];
    }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[t][r] *= alpha;

    bf16x8 pb[4];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      u32x4 w0, w1;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        w0[i] = pack_bf16(s0[8 * j + 2 * i], s0[8 * j + 2 * i + 1]);
        w1[i] = pack_bf16(s1[8 * j + 2 * i], s1[8 * j + 2 * i + 1]);
      }
      pb[j] = as_bf16x8(w0);
      pb[2 + j] = as_bf16x8(w1);
    }

    // O^T += V^T P^T
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int d = 32 * t + l32;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bf16x8 va = as_bf16x8(*reinterpret_cast<const u32x4*>(
            sv + d * kPageTokens + 8 * swz_v(d, 2 * j + half)));
        o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[j], o[t], 0, 0, 0);
      }
    }
  }

  // ---- epilogue: lane holds O^T[32t + 8g + 4h + i][q], g = r/4, i = r%4 ----
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!q_ok) return;
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
  if (a.n_splits == 1) {
    uint16_t* op = a.out + q * a.out_tok_stride + head * a.out_head_stride;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d0 = 32 * t + 8 * g + 4 * half;
        u32x2 w;
        w[0] = pack_bf16(o[t][4 * g] * inv, o[t][4 * g + 1] * inv);
        w[1] = pack_bf16(o[t][4 * g + 2] * inv, o[t][4 * g + 3] * inv);
        *reinterpret_cast<u32x2*>(op + d0) = w;
      }
  } else {
    const int64_t row = (static_cast<int64_t>(split) * a.num_heads + head) * a.n_q + q;
    float* po = a.part_o + row * kHeadDim;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d0 = 32 * t + 8 * g + 4 * half;
        *reinterpret_cast<f32x4*>(po + d0) =
            (f32x4){o[t][4 * g] * inv, o[t][4 * g + 1] * inv, o[t][4 * g + 2] * inv,
                    o[t][4 * g + 3] * inv};
      }
    if (half == 0) a.part_lse[row] = l_tot > 0.f ? m_run * c + __log2f(l_tot) : kNegInf;
  }
}

// ------------------------------------------------------------------------- //
// audio_attn: one wave per (head, q-tile of 16, key range); 4 waves per block.
//
// Lane l = 16*g + i (g = 0..3, i = query column).  16x16x32 MFMAs:
//   S^T tile t (16 keys) = K Q'^T, 4 d-steps of 32;
//   O^T d-tile u' (16 d) += V^T P^T, 2 key-steps of 32 per page.
// A-row m of S-tile t reads key 32*(t/2) + 8*(m/4) + 4*(t%2) + m%4, so that
// register r of lane group g in S-tiles 2u and 2u+1 holds keys 32u + 8g + r and
// 32u + 8g + 4 + r: exactly the eight consecutive keys the P*V B operand of
// key-step u needs from that lane.  Rows and chunks past the page's valid
// tokens are not loaded (no HBM traffic for the partly filled pages).
// ------------------------------------------------------------------------- //
__global__ __launch_bounds__(256) void audio_attn_kernel(const AttnArgs a) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, i16 = lane & 15;
  const int wid = blockIdx.x * 4 + wave;
  const int n_work = a.num_heads * a.n_qtiles * a.n_splits;
  if (wid >= n_work) return;
  const int split = wid % a.n_splits;
  const int rest = wid / a.n_splits;
  const int qtile = rest % a.n_qtiles;
  const int head = rest / a.n_qtiles;
  const int p_begin = split * a.pages_per_split;
  const int p_end = min(a.n_pages, p_begin + a.pages_per_split);

  // Q prologue: lane holds Q'[q][32s + 8g + j], s = 0..3
  const int q = qtile * kAudioQTile + i16;
  const bool q_ok = q < a.n_q;
  u32x4 qraw[4];
  const uint16_t* qp = a.q + q * a.q_tok_stride + head * a.q_head_stride + 8 * g;
#pragma unroll
  for (int s = 0; s < 4; ++s)
    qraw[s] = q_ok ? *reinterpret_cast<const u32x4*>(qp + 32 * s) : (u32x4){0u, 0u, 0u, 0u};
  bf16x8 qreg[4];
  if (a.mode == 1) {
    float ss = 0.f;
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float x0 = bf16_lo(qraw[s][i]), x1 = bf16_hi(qraw[s][i]);
        ss += x0 * x0 + x1 * x1;
      }
    ss += __shfl_xor(ss, 16);
    ss += __shfl_xor(ss, 32);
    const float inv = rsqrtf(ss * (1.0f / kHeadDim) + a.eps);
    int pt = 0, ph = 0, pw = 0;
    if (q_ok) load_pos(a.rope, a.positions, q, a.flags, pt, ph, pw);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int d0 = 32 * s + 8 * g;
      const float4 g0 = *reinterpret_cast<const float4*>(a.gamma + d0);
      const float4 g1 = *reinterpret_cast<const float4*>(a.gamma + d0 + 4);
      const float gg[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
      u32x4 w;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float y0 = bf16_lo(qraw[s][i]) * inv * gg[2 * i];
        const float y1 = bf16_hi(qraw[s][i]) * inv * gg[2 * i + 1];
        const float2 cs = rope_cs(a.rope, (d0 >> 1) + i, pt, ph, pw);
        w[i] = pack_bf16(y0 * cs.x - y1 * cs.y, y0 * cs.y + y1 * cs.x);
      }
      qreg[s] = as_bf16x8(q_ok ? w : (u32x4){0u, 0u, 0u, 0u});
    }
  } else {
#pragma unroll
    for (int s = 0; s < 4; ++s) qreg[s] = as_bf16x8(qraw[s]);
  }

  f32x4 o[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) o[u] = (f32x4){0.f, 0.f, 0.f, 0.f};
  float m_run = kNegInf, l_run = 0.f;
  const float c = a.scale_log2;
  const u32x4 zero4 = {0u, 0u, 0u, 0u};

  for (int pi = p_begin; pi < p_end; ++pi) {
    const int2 pr = a.pages[pi];
    const int n_valid = pr.y;
    const int64_t tileo = (static_cast<int64_t>(pr.x) * a.num_heads + head) * kPageHeadElems;
    const uint16_t* kb = a.kpool + tileo;
    const uint16_t* vb = a.vpool + tileo;
    u32x4 kr[4][4], vr[2][8];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int key = 32 * (t >> 1) + 8 * (i16 >> 2) + 4 * (t & 1) + (i16 & 3);
#pragma unroll
      for (int s = 0; s < 4; ++s)
        kr[t][s] = key < n_valid
                       ? *reinterpret_cast<const u32x4*>(kb + key * kHeadDim + 32 * s + 8 * g)
                       : zero4;
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const bool chunk_ok = 32 * u + 8 * g < n_valid;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt)
        vr[u][dt] = chunk_ok ? *reinterpret_cast<const u32x4*>(
                                   vb + (16 * dt + i16) * kPageTokens + 32 * u + 8 * g)
                             : zero4;
    }
    f32x4 st[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      st[t] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < 4; ++s)
        st[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kr[t][s]), qreg[s], st[t], 0, 0,
                                                        0);
    }
    // register r of group g in tile t holds key 32*(t/2) + 8*g + 4*(t%2) + r
    float mx = kNegInf;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = 32 * (t >> 1) + 8 * g + 4 * (t & 1) + r;
        if (key >= n_valid) st[t][r] = kNegInf;
        mx = fmaxf(mx, st[t][r]);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == kNegInf) ? 0.f : m_new;
    const float alpha = fast_exp2((m_run - m_use) * c);
    const float mc = m_use * c;
    float psum = 0.f;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        st[t][r] = fast_exp2(__builtin_fmaf(st[t][r], c, -mc));
        psum += st[t][r];
      }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int u = 0; u < 8; ++u) o[u] *= alpha;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      u32x4 w;
      w[0] = pack_bf16(st[2 * u][0], st[2 * u][1]);
      w[1] = pack_bf16(st[2 * u][2], st[2 * u][3]);
      w[2] = pack_bf16(st[2 * u + 1][0], st[2 * u + 1][1]);
      w[3] = pack_bf16(st[2 * u + 1][2], st[2 * u + 1][3]);
      const bf16x8 pbv = as_bf16x8(w);
#pragma unroll
      for (int dt = 0; dt < 8; ++dt)
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vr[u][dt]), pbv, o[dt], 0, 0, 0);
    }
  }

  // lane holds O^T[16*dt + 4*g + r][q]; row sums are spread over the 4 groups
  float l_tot = l_run + __shfl_xor(l_run, 16);
  l_tot += __shfl_xor(l_tot, 32);
  if (!q_ok) return;
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
  const int64_t row = (static_cast<int64_t>(split) * a.num_heads + head) * a.n_q + q;
  float* po = a.part_o + row * kHeadDim;
#pragma unroll
  for (int dt = 0; dt < 8; ++dt)
    *reinterpret_cast<f32x4*>(po + 16 * dt + 4 * g) = o[dt] * inv;
  if (g == 0) a.part_lse[row] = l_tot > 0.f ? m_run * c + __log2f(l_tot) : kNegInf;
}

// ------------------------------------------------------------------------- //
// combine: 32 threads per (head, query) row, 4 d each; 8 rows per block.
// ------------------------------------------------------------------------- //
__global__ __launch_bounds__(256) void combine_kernel(const CombineArgs a) {
  const int row = blockIdx.x * 8 + (threadIdx.x >> 5);
  if (row >= a.num_heads * a.n_q) return;
  const int head = row / a.n_q, q = row % a.n_q;
  const int d0 = 4 * (threadIdx.x & 31);
  const int64_t split_stride = static_cast<int64_t>(a.num_heads) * a.n_q;
  float mx = kNegInf;
  for (int s = 0; s < a.n_splits; ++s) mx = fmaxf(mx, a.part_lse[s * split_stride + row]);
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  float wsum = 0.f;
  if (mx != kNegInf) {
    for (int s = 0; s < a.n_splits; ++s) {
      const float l = a.part_lse[s * split_stride + row];
      if (l == kNegInf) continue;
      const float w = fast_exp2(l - mx);
      wsum += w;
      acc += w * *reinterpret_cast<const f32x4*>(a.part_o + (s * split_stride + row) * kHeadDim + d0);
    }
    acc *= 1.0f / wsum;
  }
  u32x2 w;
  w[0] = pack_bf16(acc[0], acc[1]);
  w[1] = pack_bf16(acc[2], acc[3]);
  *reinterpret_cast<u32x2*>(a.out + q * a.out_tok_stride + head * a.out_head_stride + d0) = w;
}

}  // namespace

hipError_t launch_kv_append(const AppendArgs& a, hipStream_t stream) {
  dim3 grid(a.n_pages, a.num_heads);
  if (a.mode == 1)
    hipLaunchKernelGGL(kv_append_kernel<1>, grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(kv_append_kernel<0>, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_unit_attention(const AttnArgs& a, hipStream_t stream) {
  dim3 grid(a.n_qtiles * a.num_heads * a.n_splits);
  hipLaunchKernelGGL(unit_attn_kernel, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_audio_attention(const AttnArgs& a, hipStream_t stream) {
  const int waves = a.num_heads * a.n_qtiles * a.n_splits;
  dim3 grid((waves + 3) / 4);
  hipLaunchKernelGGL(audio_attn_kernel, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_combine(const CombineArgs& a, hipStream_t stream) {
  const int rows = a.num_heads * a.n_q;
  dim3 grid((rows + 7) / 8);
  hipLaunchKernelGGL(combine_kernel, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ws
