// Internal declarations shared by the host API and the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "chorus.h"

namespace chorus {

constexpr int kBlock = 64;            // tokens per mask block
constexpr int kHeadDim = 128;         // supported head dim
constexpr int kMaxBuilderBlocks = 4096;
constexpr int kNumXcd = 8;            // MI355X: 8 XCDs x 32 CUs

// Record a formatted error for chorus_last_error(); returns `st` for chaining.
chorus_status fail(chorus_status st, const char* fmt, ...);
chorus_status check_launch(const char* what);

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
inline int32_t blocks_of(int32_t S) { return (S + kBlock - 1) / kBlock; }

// Carves a workspace into 256-byte aligned segments.
struct Carver {
  char* base;
  size_t used = 0;
  explicit Carver(void* p) : base(static_cast<char*>(p)) {}
  template <class T>
  T* take(size_t count) {
    used = align_up(used, 256);
    T* p = base ? reinterpret_cast<T*>(base + used) : nullptr;
    used += count * sizeof(T);
    return p;
  }
};

// Plain-old-data view of one [B, S, H, D] tensor for kernels.
struct TensorArg {
  const void* data;
  int64_t sb, ss, sh;
};

// First-frame key enhancement: keys of tokens < n_first count beta times
// (n_first == 0: off).
struct KeyScale {
  int n_first;
  float beta;
};

// ---- mask builder (mask_builder.hip) ----
struct BuilderWorkspace {
  double* qbar;      // [B*H*n, D]
  double* kbar;      // [B*H*n, D]
  int32_t* counts;   // [B*H*n]
  uint32_t* bitmap;  // [B*H*n, words]
  double* scores;    // [B*H*n, n]
  int32_t words;
};
BuilderWorkspace carve_builder(void* ws, int B, int H, int n, size_t* bytes);
hipError_t launch_pool(chorus_dtype dt, TensorArg q, TensorArg k, int B, int S, int H, int kvb, KeyScale ks,
                       double* qbar, double* kbar, hipStream_t st);
hipError_t launch_pool_fp8(TensorArg q, const float* q_scale, TensorArg k, const float* k_scale, int B, int S,
                           int H, int kvb, KeyScale ks, double* qbar, double* kbar, hipStream_t st);
// block means from the fp8 quantiser's 64-token column sums [B, H, n, 128]
hipError_t launch_means_from_sums(const double* q_sums, const double* k_sums, int B, int S, int H, int kvb,
                                  double* qbar, double* kbar, hipStream_t st);
hipError_t launch_score_select(const double* qbar, const double* kbar, int B, int H, int n, int nk,
                               double sm_scale, double top_p, int k_min, double* scores,
                               int32_t* counts, uint32_t* bitmap, int words, float* block_scores,
                               hipStream_t st);
hipError_t launch_select_from_mass(const float* mass, int64_t rows, int n, double top_p, int k_min,
                                   int32_t* counts, uint32_t* bitmap, int words, hipStream_t st);
hipError_t launch_scan_counts(const int32_t* counts, int64_t rows, int32_t* row_ptr, hipStream_t st);
hipError_t launch_compact(const uint32_t* bitmap, int words, const int32_t* row_ptr, int64_t rows,
                          int32_t* col_idx, hipStream_t st);
hipError_t launch_plan(const int32_t* row_ptr, int mask_batch, int B, int H, int n, int per_id, int32_t* order,
                       hipStream_t st);
hipError_t launch_validate(const int32_t* row_ptr, const int32_t* col_idx, int64_t rows, int n,
                           int64_t capacity, int32_t* flags, hipStream_t st);

// ---- mask builder with its scratch in a fixed device array (builder_noalloc.hip) ----
size_t builder_noalloc_scratch_bytes();
int noalloc_heads_per_chunk(int64_t rows, int words, int n, int nk, int H);
chorus_status build_mask_noalloc(chorus_dtype dtype, int B, int S, int H, const TensorArg& q, const TensorArg& k,
                                 double sm_scale, double top_p, int k_min, int kv_block, KeyScale ks,
                                 int32_t* row_ptr, int32_t* col_idx, float* block_scores, hipStream_t st);

// ---- block mass and coverage (block_mass.hip) ----
hipError_t launch_block_mass(chorus_dtype dt, TensorArg q, TensorArg k, const float* lse, int B, int S, int H,
                             float sm_scale, KeyScale ks, int kvb, float* mass, hipStream_t st);
hipError_t launch_coverage(const int32_t* row_ptr, const int32_t* col_idx, int mask_batch, const float* mass, int B,
                           int S, int H, int kvb, double* coverage, hipStream_t st);

// ---- visit refreshing (fallback.hip) ----
hipError_t launch_visit_update(const int32_t* row_ptr, const int32_t* col_idx, int64_t rows, int n,
                               uint32_t* visited, hipStream_t st);
hipError_t launch_visit_refresh(const int32_t* row_ptr, const int32_t* col_idx, int64_t rows, int n,
                                const uint32_t* visited, int32_t* counts, uint32_t* bitmap, hipStream_t st);
hipError_t launch_fill_u32(uint32_t* p, uint32_t v, int64_t count, hipStream_t st);

// ---- fp8 quantiser (quant_fp8.hip) ----
// sums == nullptr: codes and scales only; otherwise also the float64 block
// column sums [B, H, n, 128] (first-frame tokens weighted by ks.beta)
hipError_t launch_quant_fp8(chorus_dtype in_dt, TensorArg x, TensorArg codes, int B, int S, int H,
                            float* scales, KeyScale ks, double* sums, hipStream_t st);

// ---- attention (attn_fwd.hip, attn_fwd_fp8.hip) ----
struct AttnArgs {
  TensorArg q, k, v, o;
  const float* q_scale;
  const float* k_scale;
  const float* v_scale;
  const int32_t* row_ptr;
  const int32_t* col_idx;
  const int32_t* order;   // nullable
  float* lse;             // nullable
  int B, S, H, n;
  int mask_batch;
  int kv_block;           // tokens per listed kv block: 64, or 128 (two 64-token halves)
  float sm_scale;
  KeyScale ks;
};
hipError_t launch_attn_fwd_16(chorus_dtype dt, const AttnArgs& a, hipStream_t st);
hipError_t launch_attn_fwd_fp8(const AttnArgs& a, hipStream_t st);

}  // namespace chorus
