// The attention sub-block of one performer layer at one denoising step
// (Wan-Streamer v0.2, Sec. 3: the performer generates the next unit
// conditioned on its K/V cache and writes the unit's own K/V into it): the
// QKV projection, the append of the unit's K/V with the query preparation,
// the video and audio attention, and the output projection.  The two
// projections are plain GEMMs and run on hipBLASLt; everything between them
// is this library's own kernels (ws_step_append, ws_step_attention).
//
// All device memory the step uses is allocated by ws_block_create.
#include <hip/hip_runtime.h>
#include <hipblaslt/hipblaslt.h>

#include <cmath>
#include <cstring>

#include "ws.h"
#include "ws_internal.hpp"

namespace {

constexpr int kMaxPlans = 8;           // projection shapes kept per block (row counts)
constexpr size_t kGemmWorkspace = size_t(64) << 20;
constexpr int kTuneCandidates = 16;    // heuristic algorithms timed per new projection shape
constexpr int kTuneRuns = 5;           // timed launches per candidate (after one untimed)

struct GemmPlan {
  int64_t rows = -1;                  // M (tokens)
  hipblasLtMatrixLayout_t a = nullptr, b = nullptr, c = nullptr;
  hipblasLtMatmulAlgo_t algo{};
  size_t workspace = 0;
};

}  // namespace

struct ws_block {
  ws_cache* cache = nullptr;
  int32_t hidden = 0;
  int32_t max_rows = 0;
  const uint16_t* w_qkv = nullptr;
  const uint16_t* w_out = nullptr;
  hipblasLtHandle_t lt = nullptr;
  hipblasLtMatmulDesc_t desc = nullptr;
  hipblasLtMatmulPreference_t pref = nullptr;
  void* workspace = nullptr;
  uint16_t* qkv = nullptr;    // [max_rows][3 hidden]
  uint16_t* qprep = nullptr;  // [max_rows][hidden] prepared queries
  uint16_t* attn = nullptr;   // [max_rows][hidden] attention output
  GemmPlan plans[2][kMaxPlans];  // [0]: QKV projection, [1]: output projection
  int next_plan[2] = {0, 0};
};

namespace {

const char* lt_status_name(hipblasStatus_t s) {
  switch (s) {
    case HIPBLAS_STATUS_SUCCESS: return "success";
    case HIPBLAS_STATUS_NOT_INITIALIZED: return "not initialized";
    case HIPBLAS_STATUS_ALLOC_FAILED: return "allocation failed";
    case HIPBLAS_STATUS_INVALID_VALUE: return "invalid value";
    case HIPBLAS_STATUS_ARCH_MISMATCH: return "arch mismatch";
    case HIPBLAS_STATUS_EXECUTION_FAILED: return "execution failed";
    case HIPBLAS_STATUS_NOT_SUPPORTED: return "not supported";
    default: return "error";
  }
}

ws_status lt_fail(hipblasStatus_t s, const char* what) {
  return ws_internal::fail(WS_ERR_HIP, "%s: hipBLASLt %s (%d)", what, lt_status_name(s), static_cast<int>(s));
}

#define WS_LT(call)                                      \
  do {                                                   \
    hipblasStatus_t s_ = (call);                         \
    if (s_ != HIPBLAS_STATUS_SUCCESS) return lt_fail(s_, #call); \
  } while (0)

void free_plan(GemmPlan& p) {
  if (p.a) (void)hipblasLtMatrixLayoutDestroy(p.a);
  if (p.b) (void)hipblasLtMatrixLayoutDestroy(p.b);
  if (p.c) (void)hipblasLtMatrixLayoutDestroy(p.c);
  p = GemmPlan{};
}

void free_block(ws_block* b) {
  for (auto& row : b->plans)
    for (auto& p : row) free_plan(p);
  if (b->pref) (void)hipblasLtMatmulPreferenceDestroy(b->pref);
  if (b->desc) (void)hipblasLtMatmulDescDestroy(b->desc);
  if (b->lt) (void)hipblasLtDestroy(b->lt);
  if (b->workspace) (void)hipFree(b->workspace);
  if (b->qkv) (void)hipFree(b->qkv);
  if (b->qprep) (void)hipFree(b->qprep);
  if (b->attn) (void)hipFree(b->attn);
}

// Times each heuristic candidate on the operands it will run on (kTuneRuns
// launches after an untimed one, HIP events on the stream) and returns the
// index of the fastest; candidates that fail to launch or need more
// workspace than the block holds are skipped.  Waits for the stream.
int fastest_candidate(ws_block* b, const GemmPlan& p, const hipblasLtMatmulHeuristicResult_t* res, int found,
                      const uint16_t* x, const uint16_t* w, uint16_t* y, hipStream_t stream) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (hipEventCreate(&e0) != hipSuccess) return 0;
  if (hipEventCreate(&e1) != hipSuccess) {
    (void)hipEventDestroy(e0);
    return 0;
  }
  const float alpha = 1.0f, beta = 0.0f;
  int best = 0;
  float best_ms = -1.0f;
  for (int i = 0; i < found; ++i) {
    if (res[i].state != HIPBLAS_STATUS_SUCCESS || res[i].workspaceSize > kGemmWorkspace) continue;
    auto run = [&]() {
      return hipblasLtMatmul(b->lt, b->desc, &alpha, w, p.a, x, p.b, &beta, y, p.c, y, p.c, &res[i].algo,
                             b->workspace, res[i].workspaceSize, stream);
    };
    if (run() != HIPBLAS_STATUS_SUCCESS) continue;
    bool ok = hipEventRecord(e0, stream) == hipSuccess;
    for (int r = 0; ok && r < kTuneRuns; ++r) ok = run() == HIPBLAS_STATUS_SUCCESS;
    ok = ok && hipEventRecord(e1, stream) == hipSuccess && hipEventSynchronize(e1) == hipSuccess;
    float ms = 0.0f;
    if (!ok || hipEventElapsedTime(&ms, e0, e1) != hipSuccess) continue;
    if (best_ms < 0.0f || ms < best_ms) {
      best_ms = ms;
      best = i;
    }
  }
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  return best;
}

// Row-major Y[M][N] = X[M][K] W[K][N] in hipBLASLt's column-major terms:
// Y^T (N x M, ld N) = W^T (N x K, ld N) X^T (K x M, ld K), no transposes.
// The layouts and the algorithm are kept per (projection, M): a new M asks
// the heuristic for up to kTuneCandidates algorithms and keeps the one that
// runs fastest on this step's operands (x, w -> y).
ws_status gemm_plan(ws_block* b, int which, int64_t m, const uint16_t* x, const uint16_t* w, uint16_t* y,
                    hipStream_t stream, const GemmPlan** out) {
  const int64_t k = b->hidden, n = which == 0 ? 3 * int64_t(b->hidden) : b->hidden;
  for (const GemmPlan& p : b->plans[which])
    if (p.rows == m) {
      *out = &p;
      return WS_OK;
    }
  GemmPlan& p = b->plans[which][b->next_plan[which]];
  b->next_plan[which] = (b->next_plan[which] + 1) % kMaxPlans;
  free_plan(p);
  WS_LT(hipblasLtMatrixLayoutCreate(&p.a, HIP_R_16BF, n, k, n));
  WS_LT(hipblasLtMatrixLayoutCreate(&p.b, HIP_R_16BF, k, m, k));
  WS_LT(hipblasLtMatrixLayoutCreate(&p.c, HIP_R_16BF, n, m, n));
  hipblasLtMatmulHeuristicResult_t res[kTuneCandidates];
  int found = 0;
  WS_LT(hipblasLtMatmulAlgoGetHeuristic(b->lt, b->desc, p.a, p.b, p.c, p.c, b->pref, kTuneCandidates, res,
                                        &found));
  if (found < 1) return ws_internal::fail(WS_ERR_UNSUPPORTED, "hipBLASLt found no algorithm for %lld x %lld x %lld",
                                          static_cast<long long>(m), static_cast<long long>(n),
                                          static_cast<long long>(k));
  const int best = found > 1 ? fastest_candidate(b, p, res, found, x, w, y, stream) : 0;
  p.algo = res[best].algo;
  p.workspace = res[best].workspaceSize;
  p.rows = m;
  *out = &p;
  return WS_OK;
}

ws_status gemm(ws_block* b, const GemmPlan* p, const uint16_t* x, const uint16_t* w, uint16_t* y,
               hipStream_t stream) {
  const float alpha = 1.0f, beta = 0.0f;
  WS_LT(hipblasLtMatmul(b->lt, b->desc, &alpha, w, p->a, x, p->b, &beta, y, p->c, y, p->c, &p->algo,
                        b->workspace, p->workspace, stream));
  return WS_OK;
}

ws_status create_impl(ws_cache* cache, const void* w_qkv, const void* w_out, int32_t max_rows, ws_block** out) {
  using ws_internal::fail;
  if (!cache || !w_qkv || !w_out || !out) return fail(WS_ERR_INVALID_ARG, "NULL argument");
  *out = nullptr;
  if ((reinterpret_cast<uintptr_t>(w_qkv) | reinterpret_cast<uintptr_t>(w_out)) & 15u)
    return fail(WS_ERR_INVALID_ARG, "weights must be 16-byte aligned");
  const int32_t H = ws_internal::cache_heads(cache);
  if (max_rows < 1 || max_rows > ws_internal::cache_max_q(cache))
    return fail(WS_ERR_SHAPE, "max_rows %d outside [1, max_q_tokens = %d]", max_rows,
                ws_internal::cache_max_q(cache));
  ws_block* b = new ws_block;
  b->cache = cache;
  b->hidden = H * 128;
  b->max_rows = max_rows;
  b->w_qkv = static_cast<const uint16_t*>(w_qkv);
  b->w_out = static_cast<const uint16_t*>(w_out);
  auto bail = [&](ws_status st) {
    free_block(b);
    delete b;
    return st;
  };
  auto lt_bail = [&](hipblasStatus_t s, const char* what) { return bail(lt_fail(s, what)); };
  hipblasStatus_t s;
  if ((s = hipblasLtCreate(&b->lt)) != HIPBLAS_STATUS_SUCCESS) return lt_bail(s, "hipblasLtCreate");
  if ((s = hipblasLtMatmulDescCreate(&b->desc, HIPBLAS_COMPUTE_32F, HIP_R_32F)) != HIPBLAS_STATUS_SUCCESS)
    return lt_bail(s, "hipblasLtMatmulDescCreate");
  if ((s = hipblasLtMatmulPreferenceCreate(&b->pref)) != HIPBLAS_STATUS_SUCCESS)
    return lt_bail(s, "hipblasLtMatmulPreferenceCreate");
  const uint64_t ws_bytes = kGemmWorkspace;
  if ((s = hipblasLtMatmulPreferenceSetAttribute(b->pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &ws_bytes,
                                                 sizeof ws_bytes)) != HIPBLAS_STATUS_SUCCESS)
    return lt_bail(s, "hipblasLtMatmulPreferenceSetAttribute");
  hipError_t e;
  if ((e = hipMalloc(&b->workspace, kGemmWorkspace)) != hipSuccess)
    return bail(ws_internal::hip_fail(e, "hipMalloc(GEMM workspace)"));
  const size_t rows = static_cast<size_t>(max_rows), hid = static_cast<size_t>(b->hidden);
  if ((e = hipMalloc(&b->qkv, rows * 3 * hid * 2)) != hipSuccess) return bail(ws_internal::hip_fail(e, "hipMalloc(qkv)"));
  if ((e = hipMalloc(&b->qprep, rows * hid * 2)) != hipSuccess) return bail(ws_internal::hip_fail(e, "hipMalloc(queries)"));
  if ((e = hipMalloc(&b->attn, rows * hid * 2)) != hipSuccess) return bail(ws_internal::hip_fail(e, "hipMalloc(attn)"));
  *out = b;
  return WS_OK;
}

}  // namespace

extern "C" {

ws_status ws_block_create(ws_cache* cache, const void* w_qkv, const void* w_out, int32_t max_rows,
                          ws_block** out) {
  try {
    return create_impl(cache, w_qkv, w_out, max_rows, out);
  } catch (...) {
    return ws_internal::fail(WS_ERR_INVALID_ARG, "host allocation failed");
  }
}

ws_status ws_block_destroy(ws_block* b) {
  if (!b) return WS_OK;
  const hipError_t e = hipDeviceSynchronize();
  free_block(b);
  delete b;
  if (e != hipSuccess) return ws_internal::hip_fail(e, "hipDeviceSynchronize");
  return WS_OK;
}

ws_status ws_block_step(ws_block* b, const ws_block_step_args* s, void* hip_stream) {
  using ws_internal::fail;
  if (!b || !s) return fail(WS_ERR_INVALID_ARG, "NULL argument");
  if (!s->x || !s->y) return fail(WS_ERR_INVALID_ARG, "x and y are required");
  if ((reinterpret_cast<uintptr_t>(s->x) | reinterpret_cast<uintptr_t>(s->y)) & 15u)
    return fail(WS_ERR_INVALID_ARG, "x and y must be 16-byte aligned");
  const int32_t n = s->n_video + s->n_audio;
  if (s->n_video < 1 || s->n_audio < 0 || s->n_audio > 64 || n > b->max_rows)
    return fail(WS_ERR_SHAPE, "n_video %d / n_audio %d outside [1, ..] / [0, 64], or more than %d rows",
                s->n_video, s->n_audio, b->max_rows);
  if (!s->video_positions || (s->n_audio > 0 && !s->audio_positions) || !s->gamma_q || !s->gamma_k)
    return fail(WS_ERR_INVALID_ARG, "positions and gamma are required");
  if ((reinterpret_cast<uintptr_t>(s->gamma_q) | reinterpret_cast<uintptr_t>(s->gamma_k)) & 15u)
    return fail(WS_ERR_INVALID_ARG, "gamma must be 16-byte aligned");
  if (!(s->eps >= 0.f) || !std::isfinite(s->eps) || !(s->softmax_scale >= 0.f) || !std::isfinite(s->softmax_scale))
    return fail(WS_ERR_INVALID_ARG, "bad eps or softmax_scale");
  if (s->attn_out && (reinterpret_cast<uintptr_t>(s->attn_out) & 15u))
    return fail(WS_ERR_INVALID_ARG, "attn_out must be 16-byte aligned");
  {
    int32_t need = 0;
    if (ws_status st = ws_internal::precheck_append(b->cache, s->unit, WS_KIND_VIDEO, s->n_video, &need);
        st != WS_OK)
      return st;
    if (s->n_audio > 0)
      if (ws_status st = ws_internal::precheck_append(b->cache, s->unit, WS_KIND_AUDIO, s->n_audio, &need);
          st != WS_OK)
        return st;
  }
  // both projections' layouts and algorithms are resolved before the step
  // is enqueued (a new row count times the candidates on the step's own
  // operands: the output projection's input is the attention buffer as it
  // stands, its output y, which the step then overwrites)
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  uint16_t* attn = s->attn_out ? static_cast<uint16_t*>(s->attn_out) : b->attn;
  const GemmPlan *p_qkv = nullptr, *p_out = nullptr;
  if (ws_status st = gemm_plan(b, 0, n, static_cast<const uint16_t*>(s->x), b->w_qkv, b->qkv, stream, &p_qkv);
      st != WS_OK)
    return st;
  if (ws_status st = gemm_plan(b, 1, n, attn, b->w_out, static_cast<uint16_t*>(s->y), stream, &p_out);
      st != WS_OK)
    return st;
  ws_cache* c = b->cache;
  const int64_t hid = b->hidden, row3 = 3 * hid;
  // Every argument of the two library calls is checked by them before they
  // enqueue anything; the projections are checked here.  Order on the
  // stream: QKV GEMM, append + query preparation, attention, output GEMM.
  int slot = -1;
  if (ws_status st = ws_internal::timing_begin_path(c, 3, n, stream, &slot); st != WS_OK) return st;
  if (ws_status st = gemm(b, p_qkv, static_cast<const uint16_t*>(s->x), b->w_qkv, b->qkv, stream); st != WS_OK)
    return st;
  if (ws_status st = ws_internal::timing_mark(c, slot, 1, stream); st != WS_OK) return st;
  if (ws_status st = ws_internal::timing_mark(c, slot, 2, stream); st != WS_OK) return st;
  // Q, K, V of token t, head h: qkv[t][{0, 1, 2} hid + 128 h + d]
  ws_append_item kv[2];
  ws_query_item qs[2];
  int n_kv = 0, n_qs = 0;
  auto add = [&](int32_t row0, int32_t rows, ws_kind kind, const int32_t* pos) {
    ws_append_item& it = kv[n_kv++];
    it = ws_append_item{};
    it.k = b->qkv + row0 * row3 + hid;
    it.v = b->qkv + row0 * row3 + 2 * hid;
    it.tok_stride = row3;
    it.head_stride = 128;
    it.desc.unit = s->unit;
    it.desc.kind = kind;
    it.desc.n_tokens = rows;
    it.desc.mode = WS_APPEND_NORM_ROPE;
    it.desc.positions = pos;
    it.desc.gamma = s->gamma_k;
    it.desc.eps = s->eps;
    ws_query_item& q = qs[n_qs++];
    q = ws_query_item{};
    q.q = b->qkv + row0 * row3;
    q.tok_stride = row3;
    q.head_stride = 128;
    q.n_q = rows;
    q.desc.mode = WS_APPEND_NORM_ROPE;
    q.desc.positions = pos;
    q.desc.gamma = s->gamma_q;
    q.desc.eps = s->eps;
    q.desc.softmax_scale = s->softmax_scale;
    q.q_out = b->qprep + row0 * hid;
    q.out_tok_stride = hid;
    q.out_head_stride = 128;
  };
  add(0, s->n_video, WS_KIND_VIDEO, s->video_positions);
  if (s->n_audio > 0) add(s->n_video, s->n_audio, WS_KIND_AUDIO, s->audio_positions);
  if (ws_status st = ws_step_append(c, n_kv, kv, n_qs, qs, hip_stream); st != WS_OK) return st;
  auto call = [&](int32_t row0, int32_t rows, const ws_mask_spec& m) {
    ws_attn_call a{};
    a.q = b->qprep + row0 * hid;
    a.q_tok_stride = hid;
    a.q_head_stride = 128;
    a.n_q = rows;
    a.desc.mode = WS_QUERY_PREPARED;
    a.mask = m;
    a.out = attn + row0 * hid;
    a.out_tok_stride = hid;
    a.out_head_stride = 128;
    return a;
  };
  const ws_attn_call cv = call(0, s->n_video, s->video_mask);
  if (s->n_audio > 0) {
    const ws_attn_call ca = call(s->n_video, s->n_audio, s->audio_mask);
    if (ws_status st = ws_step_attention(c, &cv, &ca, hip_stream); st != WS_OK) return st;
  } else if (ws_status st = ws_unit_attention(cv.q, cv.q_tok_stride, cv.q_head_stride, cv.n_q, &cv.desc, c,
                                              &cv.mask, cv.out, cv.out_tok_stride, cv.out_head_stride,
                                              hip_stream);
             st != WS_OK) {
    return st;
  }
  if (ws_status st = ws_internal::timing_begin_path(c, 4, n, stream, &slot); st != WS_OK) return st;
  if (ws_status st = gemm(b, p_out, attn, b->w_out, static_cast<uint16_t*>(s->y), stream); st != WS_OK)
    return st;
  if (ws_status st = ws_internal::timing_mark(c, slot, 1, stream); st != WS_OK) return st;
  return ws_internal::timing_mark(c, slot, 2, stream);
}

}  // extern "C"
