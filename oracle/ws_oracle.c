/*
 * Plain fp64 CPU oracle for the Wan-Streamer v0.2 performer unit attention.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  The product path (the
 * HIP library and its Python binding) never calls it and shares no code with
 * it: no headers, helpers, tables or constants.
 *
 * What it computes (Wan-Streamer v0.2, arXiv 2607.04443):
 *   - the performer's per-denoising-step attention of the next unit's latent
 *     queries over the K/V cache that conditions generation (Abstract; Sec. 3,
 *     "Performer" and the unit-k schedule paragraph);
 *   - the cache holds the thinker's K/V slice plus committed history units
 *     (Sec. 2.1, latents committed back into history after each unit; Sec. 3);
 *   - visibility is block-causal on one timeline (Fig. 1 caption).
 * The paper prints no equations for the attention, normalisation or rotary
 * positions; the readings used here are the textbook definitions:
 *   RMS-norm:  n(x)_c = x_c / sqrt(mean_c' x_c'^2 + eps) * gamma_c
 *   RoPE:      pair p = (2p, 2p+1) rotated by angle pos_band(p) * theta^(-p_b/n_b)
 *   attention: O_i = sum_j softmax_j(s_ij) V_j,  s_ij = scale * <Q_i, K_j>
 * computed in double precision with a two-pass softmax and no blocking.
 *
 * Parity status: every function below is pinned by CPU tests against closed
 * forms, invariants and library routines (see tests/test_oracle_*.py).
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <string.h>

#define WS_ORACLE_API __attribute__((visibility("default")))

/* Threads the parallel loops below run on (for reporting CPU timings). */
WS_ORACLE_API int ws_oracle_num_threads(void) { return omp_get_max_threads(); }

/* bf16 is the upper half of an IEEE binary32; widening is exact. */
WS_ORACLE_API void ws_oracle_bf16_decode(const uint16_t* src, int64_t n, double* dst) {
  for (int64_t i = 0; i < n; ++i) {
    uint32_t bits = ((uint32_t)src[i]) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    dst[i] = (double)f;
  }
}

/* Per-row RMS normalisation over the last axis (length d), then an
 * elementwise weight gamma[d].  Rows are independent. */
WS_ORACLE_API void ws_oracle_rmsnorm(const double* x, int64_t n, int64_t d,
                                     const double* gamma, double eps, double* out) {
  for (int64_t i = 0; i < n; ++i) {
    const double* row = x + i * d;
    double ss = 0.0;
    for (int64_t c = 0; c < d; ++c) ss += row[c] * row[c];
    double inv = 1.0 / sqrt(ss / (double)d + eps);
    for (int64_t c = 0; c < d; ++c) out[i * d + c] = row[c] * inv * gamma[c];
  }
}

/* Band of a rotary pair: pairs [0, P_t) use t, [P_t, P_t+P_h) use h, the
 * rest use w.  Returns the band and writes the pair's index inside it. */
static int rope_band(int64_t p, const int32_t* band_pairs, int64_t* p_in_band) {
  if (p < band_pairs[0]) { *p_in_band = p; return 0; }
  if (p < band_pairs[0] + band_pairs[1]) { *p_in_band = p - band_pairs[0]; return 1; }
  *p_in_band = p - band_pairs[0] - band_pairs[1];
  return 2;
}

/* The rotation angle of pair p for a token at integer position pos[3]. */
WS_ORACLE_API double ws_oracle_rope_angle(int64_t p, const int32_t* pos, const int32_t* band_pairs,
                                          double theta) {
  int64_t pb;
  int b = rope_band(p, band_pairs, &pb);
  double omega = pow(theta, -(double)pb / (double)band_pairs[b]);
  return (double)pos[b] * omega;
}

/* Rotary positions over (t, h, w): x is [n][d], pos is [n][3], d = 2 * sum(band_pairs).
 * Each pair (x_2p, x_2p+1) is rotated counter-clockwise by its angle:
 *   x'_2p   = x_2p cos(phi) - x_2p+1 sin(phi)
 *   x'_2p+1 = x_2p sin(phi) + x_2p+1 cos(phi)                                  */
WS_ORACLE_API void ws_oracle_rope(const double* x, const int32_t* pos, int64_t n, int64_t d,
                                  const int32_t* band_pairs, double theta, double* out) {
  for (int64_t i = 0; i < n; ++i) {
    for (int64_t p = 0; p < d / 2; ++p) {
      double phi = ws_oracle_rope_angle(p, pos + 3 * i, band_pairs, theta);
      double c = cos(phi), s = sin(phi);
      double a = x[i * d + 2 * p], b = x[i * d + 2 * p + 1];
      out[i * d + 2 * p] = a * c - b * s;
      out[i * d + 2 * p + 1] = a * s + b * c;
    }
  }
}

/* Dense scaled-dot-product attention of nq queries over nk keys (one head).
 * q [nq][d], k [nk][d], v [nk][d]; visible [nq][nk] (1 = key visible to the
 * query) or NULL for all visible.  out [nq][d]; lse [nq] (natural log of the
 * softmax denominator plus the row maximum) or NULL.
 * A row with no visible key gets out = 0 and lse = -inf. */
WS_ORACLE_API void ws_oracle_attention(const double* q, const double* k, const double* v,
                                       int64_t nq, int64_t nk, int64_t d,
                                       const uint8_t* visible, double scale,
                                       double* out, double* lse) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t i = 0; i < nq; ++i) {
    double m = -INFINITY;
    int any = 0;
    /* pass 1: logits' maximum over the visible keys */
    for (int64_t j = 0; j < nk; ++j) {
      if (visible && !visible[i * nk + j]) continue;
      double s = 0.0;
      for (int64_t c = 0; c < d; ++c) s += q[i * d + c] * k[j * d + c];
      s *= scale;
      if (!any || s > m) m = s;
      any = 1;
    }
    double* o = out + i * d;
    for (int64_t c = 0; c < d; ++c) o[c] = 0.0;
    if (!any) {
      if (lse) lse[i] = -INFINITY;
      continue;
    }
    /* pass 2: exponentials, their sum, and the weighted sum of values */
    double l = 0.0;
    for (int64_t j = 0; j < nk; ++j) {
      if (visible && !visible[i * nk + j]) continue;
      double s = 0.0;
      for (int64_t c = 0; c < d; ++c) s += q[i * d + c] * k[j * d + c];
      double p = exp(s * scale - m);
      l += p;
      for (int64_t c = 0; c < d; ++c) o[c] += p * v[j * d + c];
    }
    for (int64_t c = 0; c < d; ++c) o[c] /= l;
    if (lse) lse[i] = m + log(l);
  }
}

/* Merge of attention results computed over disjoint key subsets:
 * parts[s] = (o_s [nq][d] normalised, lse_s [nq]).  With M = max_s lse_s,
 *   O = sum_s exp(lse_s - M) o_s / sum_s exp(lse_s - M),  lse = M + log(sum).
 * A query whose every part is empty (lse = -inf) gets O = 0, lse = -inf. */
WS_ORACLE_API void ws_oracle_lse_merge(const double* o_parts, const double* lse_parts,
                                       int64_t n_parts, int64_t nq, int64_t d,
                                       double* out, double* lse) {
  for (int64_t i = 0; i < nq; ++i) {
    double M = -INFINITY;
    for (int64_t s = 0; s < n_parts; ++s) {
      double x = lse_parts[s * nq + i];
      if (x > M) M = x;
    }
    for (int64_t c = 0; c < d; ++c) out[i * d + c] = 0.0;
    if (M == -INFINITY) {
      if (lse) lse[i] = -INFINITY;
      continue;
    }
    double wsum = 0.0;
    for (int64_t s = 0; s < n_parts; ++s) {
      double x = lse_parts[s * nq + i];
      if (x == -INFINITY) continue;
      double w = exp(x - M);
      wsum += w;
      for (int64_t c = 0; c < d; ++c) out[i * d + c] += w * o_parts[(s * nq + i) * d + c];
    }
    for (int64_t c = 0; c < d; ++c) out[i * d + c] /= wsum;
    if (lse) lse[i] = M + log(wsum);
  }
}

/* Round n doubles to the nearest bfloat16 (8 significant bits, ties to
 * even), returned as bf16 bit patterns (the upper half of the binary32 with
 * the same value).  The rounding is taken once, from the double itself:
 * x = m * 2^e with m in [0.5, 1), m * 2^8 rounded to the nearest integer
 * (ties to even, the default rounding mode of rint), scaled back.  Finite
 * values inside the normal binary32 range only (the block step's products). */
WS_ORACLE_API void ws_oracle_bf16_round(const double* x, int64_t n, uint16_t* out) {
  for (int64_t i = 0; i < n; ++i) {
    double r = 0.0;
    if (x[i] != 0.0) {
      int e;
      double m = frexp(x[i], &e);
      r = ldexp(rint(ldexp(m, 8)), e - 8);
    }
    float f = (float)r; /* exact: r has 8 significant bits */
    uint32_t bits;
    memcpy(&bits, &f, sizeof bits);
    out[i] = (uint16_t)(bits >> 16);
  }
}
