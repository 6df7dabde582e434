// Block-pair visit refreshing (Chorus II Sec. 3.2 "Safety fallback against
// information loss", safeguard (1)): a visited bitmap V records the block
// pairs the masks of the current layer group have activated; at the group's
// last layer every pair still unvisited is forced into that layer's mask.
//
// V holds one bit per (mask row, kv block): row r owns words
// [r * words, (r + 1) * words), words = ceil(n / 32), bit j % 32 of word j / 32.
#include "chorus_internal.h"

namespace chorus {
namespace {

// OR the pairs of a mask into V: one wave per row.  The wave first scatters
// the row's ids into its LDS copy of the row's bits (n <= 4096, so <= 128
// words), then ORs those words into V's row with plain loads and stores: the
// row belongs to this wave alone, so V needs no global atomics.
__global__ __launch_bounds__(256) void visit_update_kernel(const int32_t* __restrict__ row_ptr,
                                                           const int32_t* __restrict__ col_idx, int64_t rows, int n,
                                                           int words, uint32_t* __restrict__ visited) {
  __shared__ uint32_t mrow_all[4][kMaxBuilderBlocks / 32];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + wave;
  if (row >= rows) return;
  uint32_t* mrow = mrow_all[wave];
  for (int w = lane; w < words; w += 64) mrow[w] = 0u;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  for (int e = row_ptr[row] + lane; e < row_ptr[row + 1]; e += 64) {
    const int j = col_idx[e];
    if (j >= 0 && j < n) atomicOr(&mrow[j >> 5], 1u << (j & 31));
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  uint32_t* v = visited + row * words;
  for (int w = lane; w < words; w += 64) {
    const uint32_t m = mrow[w];
    if (m) v[w] |= m;
  }
}

// Row r of the refreshed mask = (row r of the mask) | ~(row r of V), as a
// bitmap plus its population count.  One wave per row: the mask row is
// first scattered into the wave's LDS words (n <= 4096, so <= 128 words,
// two per lane).
__global__ __launch_bounds__(256) void visit_refresh_kernel(const int32_t* __restrict__ row_ptr,
                                                            const int32_t* __restrict__ col_idx, int64_t rows,
                                                            int n, int words, const uint32_t* __restrict__ visited,
                                                            int32_t* __restrict__ counts,
                                                            uint32_t* __restrict__ bitmap) {
  __shared__ uint32_t mrow_all[4][kMaxBuilderBlocks / 32];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + wave;
  if (row >= rows) return;
  uint32_t* mrow = mrow_all[wave];
  for (int w = lane; w < words; w += 64) mrow[w] = 0u;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  for (int e = row_ptr[row] + lane; e < row_ptr[row + 1]; e += 64) {
    const int j = col_idx[e];
    if (j >= 0 && j < n) atomicOr(&mrow[j >> 5], 1u << (j & 31));
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const uint32_t* v = visited + row * words;
  uint32_t* dst = bitmap + row * words;
  int cnt = 0;
  for (int w = lane; w < words; w += 64) {
    const int valid = min(32, n - 32 * w);
    const uint32_t in_range = valid == 32 ? ~0u : ((1u << valid) - 1u);
    const uint32_t x = (mrow[w] | ~v[w]) & in_range;
    dst[w] = x;
    cnt += __popc(x);
  }
  for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o);
  if (lane == 0) counts[row] = cnt;
}

__global__ void fill_u32_kernel(uint32_t* p, uint32_t v, int64_t count) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) p[i] = v;
}

}  // namespace

hipError_t launch_visit_update(const int32_t* row_ptr, const int32_t* col_idx, int64_t rows, int n,
                               uint32_t* visited, hipStream_t st) {
  const int words = (n + 31) / 32;
  hipLaunchKernelGGL(visit_update_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, row_ptr, col_idx, rows,
                     n, words, visited);
  return hipGetLastError();
}

hipError_t launch_visit_refresh(const int32_t* row_ptr, const int32_t* col_idx, int64_t rows, int n,
                                const uint32_t* visited, int32_t* counts, uint32_t* bitmap, hipStream_t st) {
  const int words = (n + 31) / 32;
  hipLaunchKernelGGL(visit_refresh_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, row_ptr, col_idx,
                     rows, n, words, visited, counts, bitmap);
  return hipGetLastError();
}

hipError_t launch_fill_u32(uint32_t* p, uint32_t v, int64_t count, hipStream_t st) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_u32_kernel, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, st, p, v, count);
  return hipGetLastError();
}

}  // namespace chorus
