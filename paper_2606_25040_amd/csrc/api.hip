// Host side of the C ABI: argument validation, workspace carving, dispatch.
// Nothing here allocates device memory or synchronises; all work is enqueued
// on the caller's stream.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "chorus_internal.h"

namespace chorus {

static thread_local char g_last_error[512] = "";

chorus_status fail(chorus_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return st;
}

chorus_status check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(CHORUS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return CHORUS_OK;
}

static chorus_status from_hip(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(CHORUS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return check_launch(what);
}

static size_t elem_size(chorus_dtype dt) { return dt == CHORUS_FP8_E4M3 ? 1 : 2; }

static chorus_status check_shape(const chorus_shape* s) {
  if (!s) return fail(CHORUS_ERR_INVALID_ARG, "shape is NULL");
  if (s->B < 1 || s->S < 1 || s->H < 1)
    return fail(CHORUS_ERR_INVALID_ARG, "shape B=%d S=%d H=%d must be >= 1", s->B, s->S, s->H);
  if (s->D != kHeadDim)
    return fail(CHORUS_ERR_UNSUPPORTED, "head dim D=%d unsupported (only 128)", s->D);
  return CHORUS_OK;
}

static chorus_status check_tensor(const chorus_tensor* t, const char* name, size_t esize) {
  if (!t) return fail(CHORUS_ERR_INVALID_ARG, "%s descriptor is NULL", name);
  if (!t->data) return fail(CHORUS_ERR_INVALID_ARG, "%s data pointer is NULL", name);
  if (reinterpret_cast<uintptr_t>(t->data) % 16)
    return fail(CHORUS_ERR_INVALID_ARG, "%s data pointer is not 16-byte aligned", name);
  const int64_t st[3] = {t->stride_b, t->stride_s, t->stride_h};
  for (int i = 0; i < 3; ++i) {
    if (st[i] < 0) return fail(CHORUS_ERR_INVALID_ARG, "%s has a negative stride", name);
    if ((st[i] * (int64_t)esize) % 16)
      return fail(CHORUS_ERR_INVALID_ARG, "%s stride %lld elements breaks 16-byte row alignment",
                  name, (long long)st[i]);
  }
  return CHORUS_OK;
}

static TensorArg targ(const chorus_tensor* t) { return {t->data, t->stride_b, t->stride_s, t->stride_h}; }

// Tile loads address a token row of one (request, head) with a 32-bit byte
// offset from the head's base: (S - 1) * stride_s * element size + 256 must fit.
static bool offsets_fit(int32_t S, int64_t stride_s, size_t es) {
  return (int64_t)(S - 1) * stride_s * (int64_t)es + 256 <= (int64_t)UINT32_MAX;
}

// kv block sizes a mask may list: 64 (square blocks) or 128 (the paper's
// kernel geometry, q-blocks of 64 with kv blocks of 128).
static bool kv_block_ok(int32_t kvb) { return kvb == kBlock || kvb == 2 * kBlock; }

// Columns of a mask: kv blocks per row.
static int32_t mask_columns(const chorus_block_mask* m) {
  return (int32_t)(((int64_t)m->n_blocks * kBlock + m->block - 1) / m->block);
}

static chorus_status check_mask(const chorus_shape* s, const chorus_block_mask* m) {
  if (!m) return fail(CHORUS_ERR_INVALID_ARG, "mask is NULL");
  if (!kv_block_ok(m->block))
    return fail(CHORUS_ERR_UNSUPPORTED, "mask kv block %d unsupported (64 or 128)", m->block);
  if (m->mask_batch != 1 && m->mask_batch != s->B)
    return fail(CHORUS_ERR_INVALID_ARG, "mask_batch %d must be 1 or B=%d", m->mask_batch, s->B);
  if (m->H != s->H) return fail(CHORUS_ERR_INVALID_ARG, "mask H=%d != shape H=%d", m->H, s->H);
  if (m->n_blocks != blocks_of(s->S))
    return fail(CHORUS_ERR_INVALID_ARG, "mask n_blocks=%d != ceil(S/64)=%d", m->n_blocks, blocks_of(s->S));
  if (!m->row_ptr || !m->col_idx) return fail(CHORUS_ERR_INVALID_ARG, "mask row_ptr/col_idx is NULL");
  return CHORUS_OK;
}

// Copies an optional key scale; NULL, n_first == 0 or beta == 1 turn it off.
static chorus_status check_key_scale(const chorus_key_scale* ks, int S, KeyScale* out) {
  out->n_first = 0;
  out->beta = 1.f;
  if (!ks) return CHORUS_OK;
  if (ks->n_first < 0 || ks->n_first > S)
    return fail(CHORUS_ERR_INVALID_ARG, "key_scale n_first=%d outside [0, S=%d]", ks->n_first, S);
  if (!std::isfinite(ks->beta)) return fail(CHORUS_ERR_INVALID_ARG, "key_scale beta must be finite");
  if (ks->n_first > 0 && ks->beta != 1.f) {
    out->n_first = ks->n_first;
    out->beta = ks->beta;
  }
  return CHORUS_OK;
}

static chorus_status check_workspace(void* ws, size_t have, size_t need) {
  if (need == 0) return CHORUS_OK;
  if (!ws) return fail(CHORUS_ERR_WORKSPACE, "workspace is NULL (need %zu bytes)", need);
  if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(CHORUS_ERR_WORKSPACE, "workspace not 256-byte aligned");
  if (have < need) return fail(CHORUS_ERR_WORKSPACE, "workspace %zu bytes < required %zu", have, need);
  return CHORUS_OK;
}

BuilderWorkspace carve_builder(void* ws, int B, int H, int n, size_t* bytes) {
  Carver c(ws);
  BuilderWorkspace w;
  const size_t rows = (size_t)B * H * n;
  w.words = (n + 31) / 32;
  w.qbar = c.take<double>(rows * kHeadDim);
  w.kbar = c.take<double>(rows * kHeadDim);
  w.counts = c.take<int32_t>(rows);
  w.bitmap = c.take<uint32_t>(rows * w.words);
  w.scores = c.take<double>(rows * n);
  if (bytes) *bytes = align_up(c.used, 256);
  return w;
}

}  // namespace chorus

using namespace chorus;

extern "C" {

const char* chorus_status_string(chorus_status s) {
  switch (s) {
    case CHORUS_OK: return "CHORUS_OK";
    case CHORUS_ERR_INVALID_ARG: return "CHORUS_ERR_INVALID_ARG";
    case CHORUS_ERR_UNSUPPORTED: return "CHORUS_ERR_UNSUPPORTED";
    case CHORUS_ERR_CAPACITY: return "CHORUS_ERR_CAPACITY";
    case CHORUS_ERR_HIP: return "CHORUS_ERR_HIP";
    case CHORUS_ERR_WORKSPACE: return "CHORUS_ERR_WORKSPACE";
  }
  return "CHORUS_ERR_UNKNOWN";
}

const char* chorus_last_error(void) { return g_last_error; }

int32_t chorus_version(void) { return 100; }

size_t chorus_build_block_mask_workspace_size(const chorus_shape* shape) {
  if (!shape || shape->B < 1 || shape->S < 1 || shape->H < 1) return 0;
  size_t bytes = 0;
  carve_builder(nullptr, shape->B, shape->H, blocks_of(shape->S), &bytes);
  return bytes;
}

// Host checks of the selection arguments and outputs, shared by every builder
// entry point (shape already checked); on success fills the ids per row (nk)
// and the floor k_min.
static chorus_status check_selection(const chorus_shape* shape, double sm_scale, double top_p, double min_top_k,
                                     int32_t kv_block, int32_t* row_ptr, int32_t* col_idx, int64_t col_capacity,
                                     int* nk_out, int* k_min_out) {
  const int n = blocks_of(shape->S);
  if (n > kMaxBuilderBlocks)
    return fail(CHORUS_ERR_UNSUPPORTED, "n_blocks=%d exceeds builder limit %d", n, kMaxBuilderBlocks);
  if (!(top_p >= 0.0 && top_p <= 1.0)) return fail(CHORUS_ERR_INVALID_ARG, "top_p must be in [0, 1]");
  if (!(min_top_k >= 0.0 && min_top_k <= 1.0))
    return fail(CHORUS_ERR_INVALID_ARG, "min_top_k must be in [0, 1]");
  if (!std::isfinite(sm_scale)) return fail(CHORUS_ERR_INVALID_ARG, "sm_scale must be finite");
  if (!kv_block_ok(kv_block)) return fail(CHORUS_ERR_UNSUPPORTED, "kv_block %d unsupported (64 or 128)", kv_block);
  if (!row_ptr || !col_idx) return fail(CHORUS_ERR_INVALID_ARG, "row_ptr/col_idx is NULL");
  const int nk = (shape->S + kv_block - 1) / kv_block;
  const int64_t rows = (int64_t)shape->B * shape->H * n;
  if (rows * nk > INT32_MAX)
    return fail(CHORUS_ERR_UNSUPPORTED, "rows*kv blocks = %lld exceeds int32 CSR offsets", (long long)(rows * nk));
  if (col_capacity < rows * nk)
    return fail(CHORUS_ERR_CAPACITY, "col_capacity %lld < worst case %lld", (long long)col_capacity,
                (long long)(rows * nk));
  *nk_out = nk;
  *k_min_out = (int)std::ceil(min_top_k * (double)nk - 1e-9);
  return CHORUS_OK;
}

// Host checks of the builder entry points that read Q and K; on success fills
// nk, k_min and the key scale.
static chorus_status check_build(chorus_dtype dtype, const chorus_shape* shape, const chorus_tensor* q,
                                 const float* q_scale, const chorus_tensor* k, const float* k_scale,
                                 double sm_scale, double top_p, double min_top_k, int32_t kv_block,
                                 const chorus_key_scale* key_scale, int32_t* row_ptr, int32_t* col_idx,
                                 int64_t col_capacity, int* nk_out, int* k_min_out, KeyScale* ks_out) {
  chorus_status st;
  if ((st = check_shape(shape))) return st;
  const bool fp8 = dtype == CHORUS_FP8_E4M3;
  if (dtype != CHORUS_F16 && dtype != CHORUS_BF16 && !fp8)
    return fail(CHORUS_ERR_UNSUPPORTED, "builder input dtype %d unsupported (f16/bf16/fp8)", (int)dtype);
  if ((st = check_tensor(q, "q", fp8 ? 1 : 2))) return st;
  if ((st = check_tensor(k, "k", fp8 ? 1 : 2))) return st;
  if (fp8 && (!q_scale || !k_scale)) return fail(CHORUS_ERR_INVALID_ARG, "fp8 input needs q_scale and k_scale");
  if ((st = check_selection(shape, sm_scale, top_p, min_top_k, kv_block, row_ptr, col_idx, col_capacity, nk_out,
                            k_min_out)))
    return st;
  return check_key_scale(key_scale, shape->S, ks_out);
}

// Block scores, selection, CSR: steps 2-7 of the builder on the pooled means
// already in the workspace.
static chorus_status select_and_emit(const chorus_shape* shape, const BuilderWorkspace& w, int nk, double sm_scale,
                                     double top_p, int k_min, int32_t* row_ptr, int32_t* col_idx,
                                     float* block_scores, hipStream_t s) {
  chorus_status st;
  const int n = blocks_of(shape->S);
  const int64_t rows = (int64_t)shape->B * shape->H * n;
  const int words = (nk + 31) / 32;
  if ((st = from_hip(launch_score_select(w.qbar, w.kbar, shape->B, shape->H, n, nk, sm_scale, top_p, k_min,
                                         w.scores, w.counts, w.bitmap, words, block_scores, s),
                     "score_select")))
    return st;
  if ((st = from_hip(launch_scan_counts(w.counts, rows, row_ptr, s), "scan"))) return st;
  return from_hip(launch_compact(w.bitmap, words, row_ptr, rows, col_idx, s), "compact");
}

static chorus_status build_mask_impl(chorus_dtype dtype, const chorus_shape* shape, const chorus_tensor* q,
                                     const float* q_scale, const chorus_tensor* k, const float* k_scale,
                                     double sm_scale, double top_p, double min_top_k, int32_t kv_block,
                                     const chorus_key_scale* key_scale, int32_t* row_ptr, int32_t* col_idx,
                                     int64_t col_capacity, float* block_scores, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  g_last_error[0] = 0;
  chorus_status st;
  int nk = 0, k_min = 0;
  KeyScale ks;
  if ((st = check_build(dtype, shape, q, q_scale, k, k_scale, sm_scale, top_p, min_top_k, kv_block, key_scale,
                        row_ptr, col_idx, col_capacity, &nk, &k_min, &ks)))
    return st;
  const bool fp8 = dtype == CHORUS_FP8_E4M3;
  const int n = blocks_of(shape->S);
  size_t need = 0;
  BuilderWorkspace w = carve_builder(workspace, shape->B, shape->H, n, &need);   // sized for nk <= n
  if ((st = check_workspace(workspace, workspace_bytes, need))) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const hipError_t pe = fp8 ? launch_pool_fp8(targ(q), q_scale, targ(k), k_scale, shape->B, shape->S, shape->H,
                                              kv_block, ks, w.qbar, w.kbar, s)
                            : launch_pool(dtype, targ(q), targ(k), shape->B, shape->S, shape->H, kv_block, ks,
                                          w.qbar, w.kbar, s);
  if ((st = from_hip(pe, "pool"))) return st;
  return select_and_emit(shape, w, nk, sm_scale, top_p, k_min, row_ptr, col_idx, block_scores, s);
}

chorus_status chorus_build_block_mask(chorus_dtype dtype, const chorus_shape* shape,
                                      const chorus_tensor* q, const chorus_tensor* k,
                                      double sm_scale, double top_p, double min_top_k,
                                      int32_t kv_block, const chorus_key_scale* key_scale,
                                      int32_t* row_ptr, int32_t* col_idx, int64_t col_capacity,
                                      float* block_scores, void* workspace,
                                      size_t workspace_bytes, void* stream) {
  if (dtype == CHORUS_FP8_E4M3) {
    g_last_error[0] = 0;
    return fail(CHORUS_ERR_UNSUPPORTED, "fp8 input goes through chorus_build_block_mask_fp8 (it needs scales)");
  }
  return build_mask_impl(dtype, shape, q, nullptr, k, nullptr, sm_scale, top_p, min_top_k, kv_block, key_scale,
                         row_ptr, col_idx, col_capacity, block_scores, workspace, workspace_bytes, stream);
}

chorus_status chorus_build_block_mask_fp8(const chorus_shape* shape, const chorus_tensor* q, const float* q_scale,
                                          const chorus_tensor* k, const float* k_scale, double sm_scale,
                                          double top_p, double min_top_k, int32_t kv_block,
                                          const chorus_key_scale* key_scale,
                                          int32_t* row_ptr, int32_t* col_idx, int64_t col_capacity,
                                          float* block_scores, void* workspace, size_t workspace_bytes,
                                          void* stream) {
  return build_mask_impl(CHORUS_FP8_E4M3, shape, q, q_scale, k, k_scale, sm_scale, top_p, min_top_k, kv_block,
                         key_scale, row_ptr, col_idx, col_capacity, block_scores, workspace, workspace_bytes,
                         stream);
}

chorus_status chorus_build_block_mask_from_sums(const chorus_shape* shape, const double* q_sums,
                                                const double* k_sums, double sm_scale, double top_p,
                                                double min_top_k, int32_t kv_block, int32_t* row_ptr,
                                                int32_t* col_idx, int64_t col_capacity, float* block_scores,
                                                void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error[0] = 0;
  chorus_status st;
  if ((st = check_shape(shape))) return st;
  if (!q_sums || !k_sums) return fail(CHORUS_ERR_INVALID_ARG, "q_sums/k_sums is NULL");
  if (reinterpret_cast<uintptr_t>(q_sums) % 8 || reinterpret_cast<uintptr_t>(k_sums) % 8)
    return fail(CHORUS_ERR_INVALID_ARG, "q_sums/k_sums is not 8-byte aligned");
  int nk = 0, k_min = 0;
  if ((st = check_selection(shape, sm_scale, top_p, min_top_k, kv_block, row_ptr, col_idx, col_capacity, &nk,
                            &k_min)))
    return st;
  size_t need = 0;
  BuilderWorkspace w = carve_builder(workspace, shape->B, shape->H, blocks_of(shape->S), &need);
  if ((st = check_workspace(workspace, workspace_bytes, need))) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = from_hip(launch_means_from_sums(q_sums, k_sums, shape->B, shape->S, shape->H, kv_block, w.qbar, w.kbar,
                                            s),
                     "means")))
    return st;
  return select_and_emit(shape, w, nk, sm_scale, top_p, k_min, row_ptr, col_idx, block_scores, s);
}

chorus_status chorus_build_block_mask_noalloc(chorus_dtype dtype, const chorus_shape* shape,
                                              const chorus_tensor* q, const chorus_tensor* k, double sm_scale,
                                              double top_p, double min_top_k, int32_t kv_block,
                                              const chorus_key_scale* key_scale, int32_t* row_ptr,
                                              int32_t* col_idx, int64_t col_capacity, float* block_scores,
                                              void* stream) {
  g_last_error[0] = 0;
  if (dtype != CHORUS_F16 && dtype != CHORUS_BF16)
    return fail(CHORUS_ERR_UNSUPPORTED, "builder without allocation takes f16 or bf16 input (dtype %d)", (int)dtype);
  chorus_status st;
  int nk = 0, k_min = 0;
  KeyScale ks;
  if ((st = check_build(dtype, shape, q, nullptr, k, nullptr, sm_scale, top_p, min_top_k, kv_block, key_scale,
                        row_ptr, col_idx, col_capacity, &nk, &k_min, &ks)))
    return st;
  const int n = blocks_of(shape->S);
  const int64_t rows = (int64_t)shape->B * shape->H * n;
  if (noalloc_heads_per_chunk(rows, (nk + 31) / 32, n, nk, shape->H) < 1)
    return fail(CHORUS_ERR_CAPACITY,
                "B*H*n_blocks=%lld rows with %d kv blocks need more than the %zu-byte builder scratch "
                "(counts and bitmaps of every row plus one head's pooled means and scores)",
                (long long)rows, nk, builder_noalloc_scratch_bytes());
  return build_mask_noalloc(dtype, shape->B, shape->S, shape->H, targ(q), targ(k), sm_scale, top_p, k_min, kv_block,
                            ks, row_ptr, col_idx, block_scores, static_cast<hipStream_t>(stream));
}

size_t chorus_plan_workspace_size(const chorus_shape* shape, const chorus_block_mask* mask) {
  (void)shape;
  (void)mask;
  return 0;   // the plan runs in LDS
}

chorus_status chorus_plan_block_mask(const chorus_shape* shape, const chorus_block_mask* mask,
                                     int32_t* order, void* workspace, size_t workspace_bytes,
                                     void* stream) {
  g_last_error[0] = 0;
  chorus_status st;
  if ((st = check_shape(shape))) return st;
  if ((st = check_mask(shape, mask))) return st;
  if (!order) return fail(CHORUS_ERR_INVALID_ARG, "order is NULL");
  if ((st = check_workspace(workspace, workspace_bytes, chorus_plan_workspace_size(shape, mask)))) return st;
  return from_hip(launch_plan(mask->row_ptr, mask->mask_batch, shape->B, shape->H, mask->n_blocks,
                              mask->block / kBlock, order, static_cast<hipStream_t>(stream)),
                  "plan");
}

chorus_status chorus_validate_block_mask(const chorus_block_mask* mask, int64_t col_capacity,
                                         int32_t* d_flags, void* stream) {
  g_last_error[0] = 0;
  if (!mask || !mask->row_ptr || !mask->col_idx || !d_flags)
    return fail(CHORUS_ERR_INVALID_ARG, "mask, its arrays and d_flags must be non-NULL");
  if (mask->mask_batch < 1 || mask->H < 1 || mask->n_blocks < 1)
    return fail(CHORUS_ERR_INVALID_ARG, "mask dimensions must be >= 1");
  if (!kv_block_ok(mask->block))
    return fail(CHORUS_ERR_UNSUPPORTED, "mask kv block %d unsupported (64 or 128)", mask->block);
  const int64_t rows = (int64_t)mask->mask_batch * mask->H * mask->n_blocks;
  return from_hip(launch_validate(mask->row_ptr, mask->col_idx, rows, mask_columns(mask), col_capacity, d_flags,
                                  static_cast<hipStream_t>(stream)),
                  "validate");
}

chorus_status chorus_quantize_fp8_blockwise(chorus_dtype in_dtype, const chorus_shape* shape,
                                            const chorus_tensor* x, const chorus_tensor* codes,
                                            float* scales, void* stream) {
  g_last_error[0] = 0;
  chorus_status st;
  if ((st = check_shape(shape))) return st;
  if (in_dtype != CHORUS_F16 && in_dtype != CHORUS_BF16)
    return fail(CHORUS_ERR_UNSUPPORTED, "quantiser input dtype %d unsupported (f16/bf16)", (int)in_dtype);
  if ((st = check_tensor(x, "x", 2))) return st;
  if ((st = check_tensor(codes, "codes", 1))) return st;
  if (!scales) return fail(CHORUS_ERR_INVALID_ARG, "scales is NULL");
  return from_hip(launch_quant_fp8(in_dtype, targ(x), targ(codes), shape->B, shape->S, shape->H, scales,
                                   KeyScale{0, 1.f}, nullptr, static_cast<hipStream_t>(stream)),
                  "quant_fp8");
}

chorus_status chorus_quantize_fp8_blockwise_sums(chorus_dtype in_dtype, const chorus_shape* shape,
                                                 const chorus_tensor* x, const chorus_tensor* codes,
                                                 float* scales, const chorus_key_scale* key_scale,
                                                 double* block_sums, void* stream) {
  g_last_error[0] = 0;
  chorus_status st;
  if ((st = check_shape(shape))) return st;
  if (in_dtype != CHORUS_F16 && in_dtype != CHORUS_BF16)
    return fail(CHORUS_ERR_UNSUPPORTED, "quantiser input dtype %d unsupported (f16/bf16)", (int)in_dtype);
  if ((st = check_tensor(x, "x", 2))) return st;
  if ((st = check_tensor(codes, "codes", 1))) return st;
  if (!scales || !block_sums) return fail(CHORUS_ERR_INVALID_ARG, "scales/block_sums is NULL");
  if (reinterpret_cast<uintptr_t>(block_sums) % 8)
    return fail(CHORUS_ERR_INVALID_ARG, "block_sums is not 8-byte aligned");
  KeyScale ks;
  if ((st = check_key_scale(key_scale, shape->S, &ks))) return st;
  return from_hip(launch_quant_fp8(in_dtype, targ(x), targ(codes), shape->B, shape->S, shape->H, scales, ks,
                                   block_sums, static_cast<hipStream_t>(stream)),
                  "quant_fp8_sums");
}

size_t chorus_attn_workspace_size(chorus_dtype dtype, const chorus_shape* shape, const chorus_block_mask* mask) {
  (void)dtype;
  (void)shape;
  (void)mask;
  return 0;
}

chorus_status chorus_block_sparse_attn_fwd(chorus_dtype dtype, const chorus_shape* shape,
                                           const chorus_tensor* q, const chorus_tensor* k,
                                           const chorus_tensor* v, const float* q_scale,
                                           const float* k_scale, const float* v_scale,
                                           const chorus_block_mask* mask,
                                           const chorus_schedule* schedule, float sm_scale,
                                           const chorus_key_scale* key_scale,
                                           const chorus_tensor* out, float* lse, void* workspace,
                                           size_t workspace_bytes, void* stream) {
  g_last_error[0] = 0;
  chorus_status st;
  if ((st = check_shape(shape))) return st;
  if (dtype != CHORUS_F16 && dtype != CHORUS_BF16 && dtype != CHORUS_FP8_E4M3)
    return fail(CHORUS_ERR_UNSUPPORTED, "attention dtype %d unsupported", (int)dtype);
  const size_t es = elem_size(dtype);
  if ((st = check_tensor(q, "q", es))) return st;
  if ((st = check_tensor(k, "k", es))) return st;
  if ((st = check_tensor(v, "v", es))) return st;
  if ((st = check_tensor(out, "out", 2))) return st;
  if (mask && (st = check_mask(shape, mask))) return st;
  if (dtype == CHORUS_FP8_E4M3) {
    if (!q_scale || !k_scale || !v_scale)
      return fail(CHORUS_ERR_INVALID_ARG, "fp8 attention needs q_scale, k_scale and v_scale");
  } else if (q_scale || k_scale || v_scale) {
    return fail(CHORUS_ERR_INVALID_ARG, "scales are only accepted for fp8 attention");
  }
  if (!std::isfinite(sm_scale) || !(sm_scale > 0.f))
    return fail(CHORUS_ERR_INVALID_ARG, "sm_scale must be finite and > 0");
  KeyScale ks;
  if ((st = check_key_scale(key_scale, shape->S, &ks))) return st;
  const int n = blocks_of(shape->S);
  const int64_t items = (int64_t)shape->B * shape->H * n;
  if (items > INT32_MAX) return fail(CHORUS_ERR_UNSUPPORTED, "too many work items");
  // kv blocks of 128 are walked as 64-token halves: doubled CSR positions must fit int32
  if (mask && mask->block != kBlock && (int64_t)mask->mask_batch * shape->H * n * mask_columns(mask) * 2 > INT32_MAX)
    return fail(CHORUS_ERR_UNSUPPORTED, "mask too large for kv blocks of 128");
  if (!offsets_fit(shape->S, std::max(std::max(q->stride_s, k->stride_s), v->stride_s), es))
    return fail(CHORUS_ERR_UNSUPPORTED, "token stride too large for 32-bit in-head offsets");
  if (schedule) {
    if (!schedule->order) return fail(CHORUS_ERR_INVALID_ARG, "schedule order is NULL");
    if (schedule->n_units != shape->B * shape->H)
      return fail(CHORUS_ERR_INVALID_ARG, "schedule has %d units, expected B*H = %d", schedule->n_units,
                  shape->B * shape->H);
  }
  if ((st = check_workspace(workspace, workspace_bytes, chorus_attn_workspace_size(dtype, shape, mask))))
    return st;
  AttnArgs a;
  a.q = targ(q);
  a.k = targ(k);
  a.v = targ(v);
  a.o = targ(out);
  a.q_scale = q_scale;
  a.k_scale = k_scale;
  a.v_scale = v_scale;
  a.row_ptr = mask ? mask->row_ptr : nullptr;   // NULL row_ptr selects the dense kernel
  a.col_idx = mask ? mask->col_idx : nullptr;
  a.mask_batch = mask ? mask->mask_batch : 1;
  a.kv_block = mask ? mask->block : kBlock;
  a.order = schedule ? schedule->order : nullptr;
  a.lse = lse;
  a.B = shape->B;
  a.S = shape->S;
  a.H = shape->H;
  a.n = n;
  a.sm_scale = sm_scale;
  a.ks = ks;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == CHORUS_FP8_E4M3) return from_hip(launch_attn_fwd_fp8(a, s), "attn_fwd_fp8");
  return from_hip(launch_attn_fwd_16(dtype, a, s), "attn_fwd");
}

chorus_status chorus_block_sparse_attn_fwd_f16(const chorus_shape* shape, const chorus_tensor* q,
                                               const chorus_tensor* k, const chorus_tensor* v,
                                               const chorus_block_mask* mask,
                                               const chorus_schedule* schedule, float sm_scale,
                                               const chorus_key_scale* key_scale,
                                               const chorus_tensor* out, float* lse, void* workspace,
                                               size_t workspace_bytes, void* stream) {
  return chorus_block_sparse_attn_fwd(CHORUS_F16, shape, q, k, v, nullptr, nullptr, nullptr, mask, schedule,
                                      sm_scale, key_scale, out, lse, workspace, workspace_bytes, stream);
}

chorus_status chorus_block_sparse_attn_fwd_bf16(const chorus_shape* shape, const chorus_tensor* q,
                                                const chorus_tensor* k, const chorus_tensor* v,
                                                const chorus_block_mask* mask,
                                                const chorus_schedule* schedule, float sm_scale,
                                                const chorus_key_scale* key_scale,
                                                const chorus_tensor* out, float* lse, void* workspace,
                                                size_t workspace_bytes, void* stream) {
  return chorus_block_sparse_attn_fwd(CHORUS_BF16, shape, q, k, v, nullptr, nullptr, nullptr, mask, schedule,
                                      sm_scale, key_scale, out, lse, workspace, workspace_bytes, stream);
}

chorus_status chorus_block_sparse_attn_fwd_fp8(const chorus_shape* shape, const chorus_tensor* q,
                                               const chorus_tensor* k, const chorus_tensor* v,
                                               const float* q_scale, const float* k_scale,
                                               const float* v_scale, const chorus_block_mask* mask,
                                               const chorus_schedule* schedule, float sm_scale,
                                               const chorus_key_scale* key_scale,
                                               const chorus_tensor* out, float* lse, void* workspace,
                                               size_t workspace_bytes, void* stream) {
  return chorus_block_sparse_attn_fwd(CHORUS_FP8_E4M3, shape, q, k, v, q_scale, k_scale, v_scale, mask,
                                      schedule, sm_scale, key_scale, out, lse, workspace, workspace_bytes,
                                      stream);
}

chorus_status chorus_attn_block_mass(chorus_dtype dtype, const chorus_shape* shape,
                                     const chorus_tensor* q, const chorus_tensor* k, const float* lse,
                                     float sm_scale, int32_t kv_block, const chorus_key_scale* key_scale,
                                     float* mass, void* stream) {
  g_last_error[0] = 0;
  chorus_status st;
  if ((st = check_shape(shape))) return st;
  if (dtype != CHORUS_F16 && dtype != CHORUS_BF16)
    return fail(CHORUS_ERR_UNSUPPORTED, "block mass dtype %d unsupported (f16/bf16)", (int)dtype);
  if ((st = check_tensor(q, "q", 2))) return st;
  if ((st = check_tensor(k, "k", 2))) return st;
  if (!lse || !mass) return fail(CHORUS_ERR_INVALID_ARG, "lse/mass is NULL");
  if (!std::isfinite(sm_scale) || !(sm_scale > 0.f))
    return fail(CHORUS_ERR_INVALID_ARG, "sm_scale must be finite and > 0");
  if (!offsets_fit(shape->S, k->stride_s, 2))
    return fail(CHORUS_ERR_UNSUPPORTED, "token stride too large for 32-bit in-head offsets");
  if (shape->H > 65535 || shape->B > 65535) return fail(CHORUS_ERR_UNSUPPORTED, "B or H above 65535");
  if (!kv_block_ok(kv_block)) return fail(CHORUS_ERR_UNSUPPORTED, "kv_block %d unsupported (64 or 128)", kv_block);
  KeyScale ks;
  if ((st = check_key_scale(key_scale, shape->S, &ks))) return st;
  return from_hip(launch_block_mass(dtype, targ(q), targ(k), lse, shape->B, shape->S, shape->H, sm_scale, ks,
                                    kv_block, mass,
                                    static_cast<hipStream_t>(stream)),
                  "block_mass");
}

size_t chorus_select_block_mask_workspace_size(const chorus_shape* shape) {
  if (!shape || shape->B < 1 || shape->H < 1 || shape->S < 1) return 0;
  const int n = blocks_of(shape->S);
  const size_t rows = (size_t)shape->B * shape->H * n;
  Carver c(nullptr);
  c.take<int32_t>(rows);
  c.take<uint32_t>(rows * ((n + 31) / 32));
  return align_up(c.used, 256);
}

chorus_status chorus_select_block_mask(const chorus_shape* shape, const float* mass, int32_t kv_block,
                                       double top_p, double min_top_k, int32_t* row_ptr, int32_t* col_idx,
                                       int64_t col_capacity, void* workspace, size_t workspace_bytes,
                                       void* stream) {
  g_last_error[0] = 0;
  chorus_status st;
  if ((st = check_shape(shape))) return st;
  if (!mass) return fail(CHORUS_ERR_INVALID_ARG, "mass is NULL");
  if (!kv_block_ok(kv_block)) return fail(CHORUS_ERR_UNSUPPORTED, "kv_block %d unsupported (64 or 128)", kv_block);
  const int n = blocks_of(shape->S);
  const int nk = (shape->S + kv_block - 1) / kv_block;
  if (n > kMaxBuilderBlocks)
    return fail(CHORUS_ERR_UNSUPPORTED, "n_blocks=%d exceeds selection limit %d", n, kMaxBuilderBlocks);
  if (!(top_p >= 0.0 && top_p <= 1.0)) return fail(CHORUS_ERR_INVALID_ARG, "top_p must be in [0, 1]");
  if (!(min_top_k >= 0.0 && min_top_k <= 1.0))
    return fail(CHORUS_ERR_INVALID_ARG, "min_top_k must be in [0, 1]");
  if (!row_ptr || !col_idx) return fail(CHORUS_ERR_INVALID_ARG, "row_ptr/col_idx is NULL");
  const int64_t rows = (int64_t)shape->B * shape->H * n;
  if (rows * nk > INT32_MAX)
    return fail(CHORUS_ERR_UNSUPPORTED, "rows*kv blocks = %lld exceeds int32 CSR offsets", (long long)(rows * nk));
  if (col_capacity < rows * nk)
    return fail(CHORUS_ERR_CAPACITY, "col_capacity %lld < worst case %lld", (long long)col_capacity,
                (long long)(rows * nk));
  if ((st = check_workspace(workspace, workspace_bytes, chorus_select_block_mask_workspace_size(shape)))) return st;
  Carver c(workspace);
  int32_t* counts = c.take<int32_t>(rows);
  const int words = (nk + 31) / 32;
  uint32_t* bitmap = c.take<uint32_t>(rows * words);   // the workspace is sized for nk <= n
  const int k_min = (int)std::ceil(min_top_k * (double)nk - 1e-9);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = from_hip(launch_select_from_mass(mass, rows, nk, top_p, k_min, counts, bitmap, words, s), "select")))
    return st;
  if ((st = from_hip(launch_scan_counts(counts, rows, row_ptr, s), "scan"))) return st;
  return from_hip(launch_compact(bitmap, words, row_ptr, rows, col_idx, s), "compact");
}

chorus_status chorus_mask_coverage(const chorus_shape* shape, const chorus_block_mask* mask,
                                   const float* mass, double* coverage, void* stream) {
  g_last_error[0] = 0;
  chorus_status st;
  if ((st = check_shape(shape))) return st;
  if ((st = check_mask(shape, mask))) return st;
  if (!mass || !coverage) return fail(CHORUS_ERR_INVALID_ARG, "mass/coverage is NULL");
  if (shape->H > 65535 || shape->B > 65535) return fail(CHORUS_ERR_UNSUPPORTED, "B or H above 65535");
  return from_hip(launch_coverage(mask->row_ptr, mask->col_idx, mask->mask_batch, mass, shape->B, shape->S,
                                  shape->H, mask->block, coverage, static_cast<hipStream_t>(stream)),
                  "coverage");
}

static chorus_status check_mask_alone(const chorus_block_mask* m) {
  if (!m) return fail(CHORUS_ERR_INVALID_ARG, "mask is NULL");
  if (!kv_block_ok(m->block))
    return fail(CHORUS_ERR_UNSUPPORTED, "mask kv block %d unsupported (64 or 128)", m->block);
  if (m->mask_batch < 1 || m->H < 1 || m->n_blocks < 1)
    return fail(CHORUS_ERR_INVALID_ARG, "mask_batch/H/n_blocks must be >= 1");
  if (m->n_blocks > kMaxBuilderBlocks)
    return fail(CHORUS_ERR_UNSUPPORTED, "n_blocks=%d exceeds limit %d", m->n_blocks, kMaxBuilderBlocks);
  if (!m->row_ptr || !m->col_idx) return fail(CHORUS_ERR_INVALID_ARG, "mask row_ptr/col_idx is NULL");
  return CHORUS_OK;
}

// Words of one row of a visited map: one bit per column of the mask.
static int64_t visit_words(const chorus_block_mask* m) { return (mask_columns(m) + 31) / 32; }

size_t chorus_visit_map_bytes(const chorus_block_mask* mask) {
  if (!mask || mask->mask_batch < 1 || mask->H < 1 || mask->n_blocks < 1 || !kv_block_ok(mask->block)) return 0;
  return (size_t)mask->mask_batch * mask->H * mask->n_blocks * visit_words(mask) * sizeof(uint32_t);
}

chorus_status chorus_visit_reset(const chorus_block_mask* mask, uint32_t* visited, void* stream) {
  g_last_error[0] = 0;
  chorus_status st;
  if ((st = check_mask_alone(mask))) return st;
  if (!visited) return fail(CHORUS_ERR_INVALID_ARG, "visited is NULL");
  const int64_t words = (int64_t)mask->mask_batch * mask->H * mask->n_blocks * visit_words(mask);
  return from_hip(launch_fill_u32(visited, 0u, words, static_cast<hipStream_t>(stream)), "visit_reset");
}

chorus_status chorus_visit_update(const chorus_block_mask* mask, uint32_t* visited, void* stream) {
  g_last_error[0] = 0;
  chorus_status st;
  if ((st = check_mask_alone(mask))) return st;
  if (!visited) return fail(CHORUS_ERR_INVALID_ARG, "visited is NULL");
  const int64_t rows = (int64_t)mask->mask_batch * mask->H * mask->n_blocks;
  return from_hip(launch_visit_update(mask->row_ptr, mask->col_idx, rows, mask_columns(mask), visited,
                                      static_cast<hipStream_t>(stream)),
                  "visit_update");
}

size_t chorus_visit_refresh_workspace_size(const chorus_block_mask* mask) {
  if (!mask || mask->mask_batch < 1 || mask->H < 1 || mask->n_blocks < 1 || !kv_block_ok(mask->block)) return 0;
  const size_t rows = (size_t)mask->mask_batch * mask->H * mask->n_blocks;
  Carver c(nullptr);
  c.take<int32_t>(rows);
  c.take<uint32_t>(rows * visit_words(mask));
  return align_up(c.used, 256);
}

chorus_status chorus_visit_refresh(const chorus_block_mask* mask, const uint32_t* visited,
                                   int32_t* row_ptr, int32_t* col_idx, int64_t col_capacity,
                                   void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error[0] = 0;
  chorus_status st;
  if ((st = check_mask_alone(mask))) return st;
  if (!visited) return fail(CHORUS_ERR_INVALID_ARG, "visited is NULL");
  if (!row_ptr || !col_idx) return fail(CHORUS_ERR_INVALID_ARG, "row_ptr/col_idx is NULL");
  const int nk = mask_columns(mask);
  const int64_t rows = (int64_t)mask->mask_batch * mask->H * mask->n_blocks;
  if (rows * nk > INT32_MAX)
    return fail(CHORUS_ERR_UNSUPPORTED, "rows*columns = %lld exceeds int32 CSR offsets", (long long)(rows * nk));
  if (col_capacity < rows * nk)
    return fail(CHORUS_ERR_CAPACITY, "col_capacity %lld < worst case %lld", (long long)col_capacity,
                (long long)(rows * nk));
  if ((st = check_workspace(workspace, workspace_bytes, chorus_visit_refresh_workspace_size(mask)))) return st;
  Carver c(workspace);
  int32_t* counts = c.take<int32_t>(rows);
  const int words = (int)visit_words(mask);
  uint32_t* bitmap = c.take<uint32_t>(rows * words);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = from_hip(launch_visit_refresh(mask->row_ptr, mask->col_idx, rows, nk, visited, counts, bitmap, s),
                     "visit_refresh")))
    return st;
  if ((st = from_hip(launch_scan_counts(counts, rows, row_ptr, s), "scan"))) return st;
  return from_hip(launch_compact(bitmap, words, row_ptr, rows, col_idx, s), "compact");
}

}  // extern "C"
