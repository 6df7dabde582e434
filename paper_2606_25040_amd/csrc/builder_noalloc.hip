// Mask builder that allocates nothing: the same pool -> score -> select ->
// CSR pipeline as chorus_build_block_mask (Chorus II Sec. 3.2 Obs. 2 and
// "Mask Caching and Retrieval"), with its scratch in a fixed device array of
// this library instead of a caller workspace.
//
// The scratch holds the per-row counts and selection bitmaps of the whole
// mask (they feed the final scan and compaction) and, for one chunk of heads
// at a time, the float64 pooled means and block scores.  The heads of each
// request are processed in chunks as large as the scratch allows, so any
// shape the builder supports works as long as one head fits; the kernels and
// their arithmetic are the builder's own, so the mask is bitwise the one
// chorus_build_block_mask writes.
#include <mutex>

#include "chorus_internal.h"

namespace chorus {
namespace {

constexpr size_t kScratchBytes = (size_t)64 << 20;
constexpr int kMaxDevices = 64;

// One copy per GPU, alive until the process ends.  In host code this name is
// a host-side stand-in: kernels get the device address from
// hipGetSymbolAddress (scratch_on_current_device), never the name itself.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

chorus_status scratch_on_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(CHORUS_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(CHORUS_ERR_UNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(CHORUS_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return CHORUS_OK;
}

TensorArg head_view(const TensorArg& t, int b, int h0, size_t elem) {
  TensorArg v = t;
  v.data = static_cast<const char*>(t.data) + ((int64_t)b * t.sb + (int64_t)h0 * t.sh) * (int64_t)elem;
  return v;
}

}  // namespace

size_t builder_noalloc_scratch_bytes() { return kScratchBytes; }

// Scratch layout: counts [rows] | bitmap [rows, words] | per chunk of c heads:
// qbar [c n, D], kbar [c nk, D], scores [c n, nk] (float64).  Returns the
// largest c that fits, 0 if not even one head does.
int noalloc_heads_per_chunk(int64_t rows, int words, int n, int nk, int H) {
  const size_t fixed = align_up((size_t)rows * 4, 256) + align_up((size_t)rows * words * 4, 256);
  const size_t per_head = align_up((size_t)n * kHeadDim * 8, 256) + align_up((size_t)nk * kHeadDim * 8, 256) +
                          align_up((size_t)n * nk * 8, 256);
  if (fixed + 3 * 256 > kScratchBytes) return 0;
  const size_t c = (kScratchBytes - fixed - 3 * 256) / per_head;
  return (int)(c < (size_t)H ? c : (size_t)H);
}

chorus_status build_mask_noalloc(chorus_dtype dtype, int B, int S, int H, const TensorArg& q, const TensorArg& k,
                                 double sm_scale, double top_p, int k_min, int kv_block, KeyScale ks,
                                 int32_t* row_ptr, int32_t* col_idx, float* block_scores, hipStream_t st) {
  void* base = nullptr;
  chorus_status status;
  if ((status = scratch_on_current_device(&base))) return status;
  const int n = blocks_of(S), nk = (S + kv_block - 1) / kv_block;
  const int64_t rows = (int64_t)B * H * n;
  const int words = (nk + 31) / 32;
  const int c = noalloc_heads_per_chunk(rows, words, n, nk, H);
  if (c < 1)
    return fail(CHORUS_ERR_CAPACITY, "one head needs more than the %zu-byte builder scratch", kScratchBytes);
  Carver cv(base);
  int32_t* counts = cv.take<int32_t>((size_t)rows);
  uint32_t* bitmap = cv.take<uint32_t>((size_t)rows * words);
  double* qbar = cv.take<double>((size_t)c * n * kHeadDim);
  double* kbar = cv.take<double>((size_t)c * nk * kHeadDim);
  double* scores = cv.take<double>((size_t)c * n * nk);
  if (align_up(cv.used, 256) > kScratchBytes) return fail(CHORUS_ERR_CAPACITY, "builder scratch layout overflow");
  for (int b = 0; b < B; ++b) {
    for (int h0 = 0; h0 < H; h0 += c) {
      const int hc = H - h0 < c ? H - h0 : c;
      const int64_t row0 = ((int64_t)b * H + h0) * n;
      hipError_t e = launch_pool(dtype, head_view(q, b, h0, 2), head_view(k, b, h0, 2), 1, S, hc, kv_block, ks,
                                 qbar, kbar, st);
      if (e != hipSuccess) return fail(CHORUS_ERR_HIP, "pool: %s", hipGetErrorString(e));
      e = launch_score_select(qbar, kbar, 1, hc, n, nk, sm_scale, top_p, k_min, scores, counts + row0,
                              bitmap + row0 * words, words, block_scores ? block_scores + row0 * nk : nullptr, st);
      if (e != hipSuccess) return fail(CHORUS_ERR_HIP, "score_select: %s", hipGetErrorString(e));
    }
  }
  hipError_t e = launch_scan_counts(counts, rows, row_ptr, st);
  if (e != hipSuccess) return fail(CHORUS_ERR_HIP, "scan: %s", hipGetErrorString(e));
  e = launch_compact(bitmap, words, row_ptr, rows, col_idx, st);
  if (e != hipSuccess) return fail(CHORUS_ERR_HIP, "compact: %s", hipGetErrorString(e));
  return CHORUS_OK;
}

}  // namespace chorus
