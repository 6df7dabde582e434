// Mask builder kernels: block mean-pool -> float64 block scores -> per-row
// joint top-p / top-k selection -> CSR, plus the work plan and a mask checker.
//
// Method: Chorus II Sec. 3.2 Obs. 2 (scores softmax(mean(Q) mean(K)^T)),
// Sec. 3.2 "Mask Caching and Retrieval" (top-p with a top-k floor), Sec. 3.2
// "Minimum top-k guarantee" and Sec. 4.1 (top_p, min_top_k); the plan is the
// one-GPU form of Sec. 3.2 "Head-level scheduling for load balancing".
//
// Everything on the selection path is float64 so that the ranking and the
// top-p boundary agree with a float64 reference up to summation order.
#include <cmath>

#include "chorus_internal.h"

namespace chorus {
namespace {

__device__ inline float to_f32(uint16_t bits, bool is_bf16) {
  if (is_bf16) return __uint_as_float(uint32_t(bits) << 16);
  return static_cast<float>(*reinterpret_cast<const _Float16*>(&bits));
}

// ---------------------------------------------------------------------------
// 1. Block mean-pool.  One wave per (tensor, request, head, block): lanes
// (g, c) with g = lane / 16 over token residues mod 4 and c = lane % 16 over
// 16-byte column chunks; float64 partial sums, reduced over g by shuffles.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void pool_kernel(TensorArg q, TensorArg k, int S, int H, int n, bool bf16,
                                                   double* __restrict__ qbar, double* __restrict__ kbar) {
  const int blk = blockIdx.x, h = blockIdx.y;
  const int b = blockIdx.z >> 1, which = blockIdx.z & 1;
  const TensorArg t = which ? k : q;
  double* out = which ? kbar : qbar;
  const int lane = threadIdx.x;
  const int g = lane >> 4, c = lane & 15;
  const int t0 = blk * kBlock;
  const int cnt = min(kBlock, S - t0);
  const uint16_t* base = static_cast<const uint16_t*>(t.data) + (int64_t)b * t.sb + (int64_t)h * t.sh + c * 8;
  double acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0;
  for (int tok = g; tok < cnt; tok += 4) {
    const uint4 raw = *reinterpret_cast<const uint4*>(base + (int64_t)(t0 + tok) * t.ss);
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[2 * e] += (double)to_f32(uint16_t(w[e] & 0xffff), bf16);
      acc[2 * e + 1] += (double)to_f32(uint16_t(w[e] >> 16), bf16);
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    acc[e] += __shfl_xor(acc[e], 16);
    acc[e] += __shfl_xor(acc[e], 32);
  }
  if (g == 0) {
    double* dst = out + ((int64_t)(b * H + h) * n + blk) * kHeadDim + c * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) dst[e] = acc[e] / (double)cnt;
  }
}

// ---------------------------------------------------------------------------
// 2a. Block scores s = sm_scale * qbar kbar^T per (request, head): a float64
// GEMM tile of 64 x 64 outputs per workgroup, k-dim staged through LDS.
// Writes float64 scores into the workspace and, optionally, fp32 copies.
// ---------------------------------------------------------------------------
constexpr int kST = 64;   // score tile
constexpr int kSK = 16;   // k-chunk

__global__ __launch_bounds__(256) void score_kernel(const double* __restrict__ qbar,
                                                    const double* __restrict__ kbar, int n, double sm_scale,
                                                    double* __restrict__ scores, float* __restrict__ scores32) {
  __shared__ double qs[kSK][kST + 1];
  __shared__ double ks[kSK][kST + 1];
  const int bh = blockIdx.z;
  const int i0 = blockIdx.y * kST, j0 = blockIdx.x * kST;
  const double* qb = qbar + (int64_t)bh * n * kHeadDim;
  const double* kb = kbar + (int64_t)bh * n * kHeadDim;
  const int tid = threadIdx.x;
  const int ti = tid / 16, tj = tid % 16;   // 16 x 16 threads, 4 x 4 outputs each
  double acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[a][c] = 0.0;
  for (int kk = 0; kk < kHeadDim; kk += kSK) {
    for (int e = tid; e < kST * kSK; e += 256) {
      const int r = e / kSK, d = e % kSK;
      qs[d][r] = (i0 + r < n) ? qb[(int64_t)(i0 + r) * kHeadDim + kk + d] : 0.0;
      ks[d][r] = (j0 + r < n) ? kb[(int64_t)(j0 + r) * kHeadDim + kk + d] : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int d = 0; d < kSK; ++d) {
      double qa[4], kc[4];
#pragma unroll
      for (int a = 0; a < 4; ++a) qa[a] = qs[d][ti + 16 * a];
#pragma unroll
      for (int c = 0; c < 4; ++c) kc[c] = ks[d][tj + 16 * c];
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[a][c] = fma(qa[a], kc[c], acc[a][c]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    const int i = i0 + ti + 16 * a;
    if (i >= n) continue;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int j = j0 + tj + 16 * c;
      if (j >= n) continue;
      const double s = sm_scale * acc[a][c];
      const int64_t o = ((int64_t)bh * n + i) * n + j;
      scores[o] = s;
      if (scores32) scores32[o] = (float)s;
    }
  }
}

// ---------------------------------------------------------------------------
// 2b. Per-row selection.  One workgroup per mask row:
//   load the row's n scores into LDS (padded to a power of two with -inf),
//   max and sum of exp in float64, bitonic sort by (score desc, index asc),
//   mass in sorted order, inclusive scan, k_p = 1 + first position whose
//   cumulative mass reaches top_p, k = min(n, max(k_p, k_min, 1)), and a
//   bitmap of the first k indices.
// ---------------------------------------------------------------------------
constexpr int kSelThreads = 256;

__device__ inline bool before(double ka, int ia, double kb, int ib) {
  // true if (ka, ia) comes first in (score desc, index asc) order
  return ka > kb || (ka == kb && ia < ib);
}

__device__ double block_reduce_max(double v, double* red) {
  for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o));
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  double r = red[0];
  for (int i = 1; i < kSelThreads / 64; ++i) r = fmax(r, red[i]);
  return r;
}

__device__ double block_reduce_sum(double v, double* red) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  double r = red[0];
  for (int i = 1; i < kSelThreads / 64; ++i) r += red[i];
  return r;
}

__global__ __launch_bounds__(kSelThreads) void select_kernel(const double* __restrict__ scores, int n, int N,
                                                             double top_p, int k_min,
                                                             int32_t* __restrict__ counts,
                                                             uint32_t* __restrict__ bitmap, int words) {
  extern __shared__ double smem[];
  double* key = smem;                                        // [N]
  int* idx = reinterpret_cast<int*>(key + N);                // [N]
  double* part = reinterpret_cast<double*>(idx + N);         // [kSelThreads]
  double* red = part + kSelThreads;                          // [4]
  uint32_t* bits = reinterpret_cast<uint32_t*>(red + 4);     // [N / 32]
  __shared__ int kp_min;
  const int64_t row = blockIdx.x;
  const double* s = scores + row * n;
  const int tid = threadIdx.x;
  for (int j = tid; j < N; j += kSelThreads) {
    key[j] = j < n ? s[j] : -INFINITY;
    idx[j] = j;
  }
  for (int w = tid; w < N / 32; w += kSelThreads) bits[w] = 0u;
  if (tid == 0) kp_min = n;
  double m = -INFINITY;
  for (int j = tid; j < n; j += kSelThreads) m = fmax(m, s[j]);
  m = block_reduce_max(m, red);
  double z = 0.0;
  for (int j = tid; j < n; j += kSelThreads) z += exp(s[j] - m);
  z = block_reduce_sum(z, red);
  __syncthreads();
  // bitonic sort: the final order is ascending in the `before` relation
  for (int size = 2; size <= N; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int t = tid; t < N / 2; t += kSelThreads) {
        const int lo = 2 * t - (t & (stride - 1));
        const int hi = lo + stride;
        const bool up = (lo & size) == 0;
        const double ka = key[lo], kb = key[hi];
        const int ia = idx[lo], ib = idx[hi];
        const bool swap = up ? before(kb, ib, ka, ia) : before(ka, ia, kb, ib);
        if (swap) {
          key[lo] = kb; key[hi] = ka;
          idx[lo] = ib; idx[hi] = ia;
        }
      }
      __syncthreads();
    }
  }
  // cumulative mass in sorted order: each thread scans a contiguous chunk
  const int per = N / kSelThreads > 0 ? N / kSelThreads : 1;
  const int c0 = tid * per;
  double local = 0.0;
  for (int r = c0; r < c0 + per && r < N; ++r) local += r < n ? exp(key[r] - m) / z : 0.0;
  part[tid] = local;
  __syncthreads();
  if (tid == 0) {
    double run = 0.0;
    for (int t = 0; t < kSelThreads; ++t) {
      const double v = part[t];
      part[t] = run;
      run += v;
    }
  }
  __syncthreads();
  int kp;
  if (top_p <= 0.0) {
    kp = 0;
  } else if (top_p >= 1.0) {
    kp = n;
  } else {
    double run = part[tid];
    for (int r = c0; r < c0 + per && r < n; ++r) {
      run += exp(key[r] - m) / z;
      if (run >= top_p) {
        atomicMin(&kp_min, r + 1);
        break;
      }
    }
    __syncthreads();
    kp = kp_min;
  }
  int k = kp > k_min ? kp : k_min;
  if (k < 1) k = 1;
  if (k > n) k = n;
  for (int r = tid; r < k; r += kSelThreads) atomicOr(&bits[idx[r] >> 5], 1u << (idx[r] & 31));
  __syncthreads();
  uint32_t* dst = bitmap + row * words;
  for (int w = tid; w < words; w += kSelThreads) dst[w] = bits[w];
  if (tid == 0) counts[row] = k;
}

// ---------------------------------------------------------------------------
// 3. Exclusive scan of the row counts into row_ptr (one workgroup).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void scan_kernel(const int32_t* __restrict__ counts, int64_t rows,
                                                    int32_t* __restrict__ row_ptr) {
  __shared__ int32_t part[1024];
  const int tid = threadIdx.x;
  const int64_t per = (rows + 1023) / 1024;
  const int64_t r0 = tid * per;
  int32_t sum = 0;
  for (int64_t r = r0; r < r0 + per && r < rows; ++r) sum += counts[r];
  part[tid] = sum;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    const int32_t v = tid >= off ? part[tid - off] : 0;
    __syncthreads();
    part[tid] += v;
    __syncthreads();
  }
  int32_t run = tid ? part[tid - 1] : 0;
  if (tid == 0) row_ptr[0] = 0;
  for (int64_t r = r0; r < r0 + per && r < rows; ++r) {
    run += counts[r];
    row_ptr[r + 1] = run;
  }
}

// ---------------------------------------------------------------------------
// 4. Compact each row's bitmap into ascending col_idx (one wave per row; each
// lane owns up to two consecutive 32-bit words, so n <= 4096).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void compact_kernel(const uint32_t* __restrict__ bitmap, int words,
                                                      const int32_t* __restrict__ row_ptr, int64_t rows,
                                                      int32_t* __restrict__ col_idx) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int lane = threadIdx.x & 63;
  const uint32_t* src = bitmap + row * words;
  const int w0 = 2 * lane, w1 = 2 * lane + 1;
  const uint32_t a = w0 < words ? src[w0] : 0u;
  const uint32_t c = w1 < words ? src[w1] : 0u;
  const int cnt = __popc(a) + __popc(c);
  int incl = cnt;
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(incl, o);
    if (lane >= o) incl += v;
  }
  int pos = row_ptr[row] + incl - cnt;
  uint32_t x = a;
  while (x) {
    const int bit = __ffs(x) - 1;
    col_idx[pos++] = w0 * 32 + bit;
    x &= x - 1;
  }
  x = c;
  while (x) {
    const int bit = __ffs(x) - 1;
    col_idx[pos++] = w1 * 32 + bit;
    x &= x - 1;
  }
}

// ---------------------------------------------------------------------------
// 5. Work plan: head units u = b * H + h with cost sum_i (blocks(b,h,i) + 1)
// are assigned to the 8 XCDs greedily, heaviest first, each to the
// least-loaded XCD that still has room (equal unit counts per XCD); the order
// lists the units XCD by XCD, ascending unit id inside an XCD.  One
// workgroup; beyond kPlanMaxUnits units the natural order is kept.
// ---------------------------------------------------------------------------
constexpr int kPlanMaxUnits = 4096;

__global__ __launch_bounds__(256) void plan_kernel(const int32_t* __restrict__ row_ptr, int mask_batch, int B,
                                                   int H, int n, int32_t* __restrict__ unit_cost,
                                                   int32_t* __restrict__ order) {
  __shared__ int32_t unit_order[kPlanMaxUnits];
  const int U = B * H;
  const int tid = threadIdx.x;
  for (int u = tid; u < U; u += 256) {
    const int b = u / H, h = u % H;
    const int64_t r0 = ((int64_t)(mask_batch > 1 ? b : 0) * H + h) * n;
    unit_cost[u] = row_ptr[r0 + n] - row_ptr[r0] + n;
  }
  __syncthreads();
  if (tid == 0 && U <= kPlanMaxUnits) {
    // unit ids by (cost desc, id asc): insertion sort
    for (int u = 0; u < U; ++u) {
      const int32_t cu = unit_cost[u];
      int p = u;
      while (p > 0) {
        const int prev = unit_order[p - 1];
        const int32_t cp = unit_cost[prev];
        if (cp > cu || (cp == cu && prev < u)) break;
        unit_order[p] = prev;
        --p;
      }
      unit_order[p] = u;
    }
    int64_t load[kNumXcd];
    int used[kNumXcd], cap[kNumXcd];
    for (int x = 0; x < kNumXcd; ++x) {
      load[x] = 0;
      used[x] = 0;
      cap[x] = U / kNumXcd + (x < U % kNumXcd ? 1 : 0);
    }
    // the assignment overwrites unit_cost (each cost is read before)
    for (int p = 0; p < U; ++p) {
      const int u = unit_order[p];
      int best = -1;
      for (int x = 0; x < kNumXcd; ++x) {
        if (used[x] >= cap[x]) continue;
        if (best < 0 || load[x] < load[best]) best = x;
      }
      load[best] += unit_cost[u];
      used[best] += 1;
      unit_cost[u] = -1 - best;
    }
    int p = 0;
    for (int x = 0; x < kNumXcd; ++x)
      for (int u = 0; u < U; ++u)
        if (unit_cost[u] == -1 - x) unit_order[p++] = u;
  }
  __syncthreads();
  for (int u = tid; u < U; u += 256) order[u] = U > kPlanMaxUnits ? u : unit_order[u];
}

// ---------------------------------------------------------------------------
// 6. Mask checker (see chorus_validate_block_mask for the flag bits).
// ---------------------------------------------------------------------------
__global__ void fill_i32_kernel(int32_t* p, int32_t v, int64_t count) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) p[i] = v;
}

__global__ __launch_bounds__(256) void validate_kernel(const int32_t* __restrict__ row_ptr,
                                                       const int32_t* __restrict__ col_idx, int64_t rows, int n,
                                                       int64_t capacity, int32_t* flags) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r == 0) {
    int f = 0;
    if (row_ptr[0] != 0) f |= 1;
    if ((int64_t)row_ptr[rows] > capacity) f |= 16;
    if (f) atomicOr(flags, f);
  }
  if (r >= rows) return;
  const int64_t a = row_ptr[r], e = row_ptr[r + 1];
  if (e < a) {
    atomicOr(flags, 2);
    return;
  }
  if (a < 0 || e > capacity || e - a > n) {
    atomicOr(flags, e > capacity ? 16 : 4);
    return;
  }
  int prev = -1, f = 0;
  for (int64_t p = a; p < e; ++p) {
    const int c = col_idx[p];
    if (c < 0 || c >= n) f |= 4;
    if (c <= prev) f |= 8;
    prev = c;
  }
  if (f) atomicOr(flags, f);
}

}  // namespace

hipError_t launch_pool(chorus_dtype dt, TensorArg q, TensorArg k, int B, int S, int H, double* qbar,
                       double* kbar, hipStream_t st) {
  const int n = blocks_of(S);
  hipLaunchKernelGGL(pool_kernel, dim3(n, H, 2 * B), dim3(64), 0, st, q, k, S, H, n, dt == CHORUS_BF16, qbar,
                     kbar);
  return hipGetLastError();
}

hipError_t launch_score_select(const double* qbar, const double* kbar, int B, int H, int n, double sm_scale,
                               double top_p, int k_min, double* scores, int32_t* counts, uint32_t* bitmap,
                               int words, float* block_scores, hipStream_t st) {
  const int tiles = (n + kST - 1) / kST;
  hipLaunchKernelGGL(score_kernel, dim3(tiles, tiles, B * H), dim3(256), 0, st, qbar, kbar, n, sm_scale, scores,
                     block_scores);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  int N = 1;
  while (N < n) N <<= 1;
  if (N < 64) N = 64;
  const size_t shmem = (size_t)N * sizeof(double) + (size_t)N * sizeof(int) + kSelThreads * sizeof(double) +
                       4 * sizeof(double) + (size_t)(N / 32) * sizeof(uint32_t);
  const int64_t rows = (int64_t)B * H * n;
  hipLaunchKernelGGL(select_kernel, dim3((unsigned)rows), dim3(kSelThreads), shmem, st, scores, n, N, top_p, k_min,
                     counts, bitmap, words);
  return hipGetLastError();
}

hipError_t launch_scan_counts(const int32_t* counts, int64_t rows, int32_t* row_ptr, hipStream_t st) {
  hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(1024), 0, st, counts, rows, row_ptr);
  return hipGetLastError();
}

hipError_t launch_compact(const uint32_t* bitmap, int words, const int32_t* row_ptr, int64_t rows, int32_t* col_idx,
                          hipStream_t st) {
  hipLaunchKernelGGL(compact_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, bitmap, words, row_ptr,
                     rows, col_idx);
  return hipGetLastError();
}

hipError_t launch_plan(const int32_t* row_ptr, int mask_batch, int B, int H, int n, int32_t* unit_cost_ws,
                       int32_t* order, hipStream_t st) {
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(256), 0, st, row_ptr, mask_batch, B, H, n, unit_cost_ws, order);
  return hipGetLastError();
}

hipError_t launch_validate(const int32_t* row_ptr, const int32_t* col_idx, int64_t rows, int n, int64_t capacity,
                           int32_t* flags, hipStream_t st) {
  hipLaunchKernelGGL(fill_i32_kernel, dim3(1), dim3(64), 0, st, flags, 0, (int64_t)1);
  hipLaunchKernelGGL(validate_kernel, dim3((unsigned)((rows + 255) / 256)), dim3(256), 0, st, row_ptr, col_idx,
                     rows, n, capacity, flags);
  return hipGetLastError();
}

}  // namespace chorus
