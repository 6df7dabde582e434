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
__global__ __launch_bounds__(64) void pool_kernel(TensorArg q, TensorArg k, int S, int H, int n, int kvb, int nk,
                                                   bool bf16, KeyScale ks, double* __restrict__ qbar,
                                                   double* __restrict__ kbar) {
  const int blk = blockIdx.x, h = blockIdx.y;
  const int b = blockIdx.z >> 1, which = blockIdx.z & 1;
  // queries pool over 64-token blocks, keys over kvb-token blocks (nk of them)
  const int bs = which ? kvb : kBlock;
  const int nb = which ? nk : n;
  if (blk >= nb) return;
  const TensorArg t = which ? k : q;
  double* out = which ? kbar : qbar;
  const int lane = threadIdx.x;
  const int g = lane >> 4, c = lane & 15;
  const int t0 = blk * bs;
  const int cnt = min(bs, S - t0);
  const uint16_t* base = static_cast<const uint16_t*>(t.data) + (int64_t)b * t.sb + (int64_t)h * t.sh + c * 8;
  double acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0;
  // first-frame keys (Eq. 1) enter the sum beta times; otherwise weight 1,
  // for which the fma is the plain sum
  const int n_scaled = which ? ks.n_first : 0;
  const double beta = (double)ks.beta;
  // 64 tokens at a time: the lane's 16 loads (tokens g, g + 4, ...) are all
  // issued before the first is summed, so a wave keeps 16 KB in flight; the
  // sums still run in token order
  for (int c0 = 0; c0 < cnt; c0 += 64) {
    uint4 raw[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int tok = c0 + g + 4 * u;
      raw[u] = tok < cnt ? *reinterpret_cast<const uint4*>(base + (int64_t)(t0 + tok) * t.ss) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int tok = c0 + g + 4 * u;
      if (tok >= cnt) break;
      const uint32_t w[4] = {raw[u].x, raw[u].y, raw[u].z, raw[u].w};
      const double wt = t0 + tok < n_scaled ? beta : 1.0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[2 * e] = __builtin_fma(wt, (double)to_f32(uint16_t(w[e] & 0xffff), bf16), acc[2 * e]);
        acc[2 * e + 1] = __builtin_fma(wt, (double)to_f32(uint16_t(w[e] >> 16), bf16), acc[2 * e + 1]);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    acc[e] += __shfl_xor(acc[e], 16);
    acc[e] += __shfl_xor(acc[e], 32);
  }
  if (g == 0) {
    double* dst = out + ((int64_t)(b * H + h) * nb + blk) * kHeadDim + c * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) dst[e] = acc[e] / (double)cnt;
  }
}

// 1b. Block mean-pool of fp8 e4m3 codes with per-(request, head, 64-token
// block) scales, as written by the fp8 quantiser: the mean of code * scale
// over the block's valid tokens, in float64.  Same lane layout as
// pool_kernel, eight codes (8 bytes) per lane and token.
__global__ __launch_bounds__(64) void pool_fp8_kernel(TensorArg q, const float* __restrict__ q_scale, TensorArg k,
                                                      const float* __restrict__ k_scale, int S, int H, int n,
                                                      int kvb, int nk, KeyScale ks, double* __restrict__ qbar,
                                                      double* __restrict__ kbar) {
  const int blk = blockIdx.x, h = blockIdx.y;
  const int b = blockIdx.z >> 1, which = blockIdx.z & 1;
  const int bs = which ? kvb : kBlock;
  const int nb = which ? nk : n;
  if (blk >= nb) return;
  const TensorArg t = which ? k : q;
  const float* sc = (which ? k_scale : q_scale) + ((int64_t)b * H + h) * n;   // per 64-token block
  double* out = which ? kbar : qbar;
  const int lane = threadIdx.x;
  const int g = lane >> 4, c = lane & 15;
  const int t0 = blk * bs;
  const int cnt = min(bs, S - t0);
  const uint8_t* base = static_cast<const uint8_t*>(t.data) + (int64_t)b * t.sb + (int64_t)h * t.sh + c * 8;
  double acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0;
  const int n_scaled = which ? ks.n_first : 0;
  const double beta = (double)ks.beta;
  // 64 tokens at a time, all 16 loads of a lane issued before the sums (as in
  // pool_kernel); the sums run in token order
  for (int c0 = 0; c0 < cnt; c0 += 64) {
    uint2 raw[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int tok = c0 + g + 4 * u;
      raw[u] = tok < cnt ? *reinterpret_cast<const uint2*>(base + (int64_t)(t0 + tok) * t.ss) : make_uint2(0, 0);
    }
    // the tokens' values are code * (scale of their 64-token block)
    const double sc_blk = (double)sc[(t0 + c0) / kBlock];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int tok = c0 + g + 4 * u;
      if (tok >= cnt) break;
      const double wt = (t0 + tok < n_scaled ? beta : 1.0) * sc_blk;
      // v_cvt_pk_f32_fp8 decodes OCP e4m3fn exactly: each of the 256 codes
      // gives the value of its fields (bias 7, three mantissa bits, subnormals
      // m * 2^-9, S.1111.111 NaN)
      const auto f01 = __builtin_amdgcn_cvt_pk_f32_fp8((int)raw[u].x, false);
      const auto f23 = __builtin_amdgcn_cvt_pk_f32_fp8((int)raw[u].x, true);
      const auto f45 = __builtin_amdgcn_cvt_pk_f32_fp8((int)raw[u].y, false);
      const auto f67 = __builtin_amdgcn_cvt_pk_f32_fp8((int)raw[u].y, true);
      const float f[8] = {f01[0], f01[1], f23[0], f23[1], f45[0], f45[1], f67[0], f67[1]};
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] = __builtin_fma(wt, (double)f[e], acc[e]);
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    acc[e] += __shfl_xor(acc[e], 16);
    acc[e] += __shfl_xor(acc[e], 32);
  }
  if (g == 0) {
    double* dst = out + ((int64_t)(b * H + h) * nb + blk) * kHeadDim + c * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) dst[e] = acc[e] / (double)cnt;
  }
}

// 1c. Block means from the column sums that the fp8 quantiser writes per
// 64-token block (same weights as pool_kernel): a kv block of 128 tokens
// adds the sums of its two halves.  One thread per (tensor, request, head,
// block, column).
__global__ __launch_bounds__(kHeadDim) void means_from_sums_kernel(const double* __restrict__ q_sums,
                                                                   const double* __restrict__ k_sums, int S, int H,
                                                                   int n, int kvb, int nk, double* __restrict__ qbar,
                                                                   double* __restrict__ kbar) {
  const int blk = blockIdx.x, h = blockIdx.y;
  const int b = blockIdx.z >> 1, which = blockIdx.z & 1;
  const int bs = which ? kvb : kBlock;
  const int nb = which ? nk : n;
  if (blk >= nb) return;
  const int d = threadIdx.x;
  const double* src = (which ? k_sums : q_sums) + (int64_t)(b * H + h) * n * kHeadDim + d;
  const int t0 = blk * bs;
  const int cnt = min(bs, S - t0);
  const int s1 = (t0 + cnt + kBlock - 1) / kBlock;   // 64-token blocks t0 / 64 .. s1 - 1
  double acc = 0.0;
  for (int s = t0 / kBlock; s < s1; ++s) acc += src[(int64_t)s * kHeadDim];
  (which ? kbar : qbar)[((int64_t)(b * H + h) * nb + blk) * kHeadDim + d] = acc / (double)cnt;
}

// ---------------------------------------------------------------------------
// 2a. Block scores s = sm_scale * qbar kbar^T per (request, head), n x nk
// (q-blocks x kv blocks): a float64 GEMM on the matrix cores
// (v_mfma_f64_16x16x4f64), one 128 x 128 output tile per workgroup of eight
// waves, each wave a 64 x 32 eighth as 4 x 2 MFMA tiles (112 registers, so a
// SIMD holds four such waves: two workgroups per CU).  The head dim is
// staged through LDS sixteen at a time (both operands k-major, so a lane's
// fragment is one float64 of a row); the next chunk is fetched into
// registers while the current one is multiplied.  Writes float64 scores
// into the workspace and, optionally, fp32 copies.
// ---------------------------------------------------------------------------
constexpr int kST = 128;  // score tile
constexpr int kSK = 16;   // k-chunk
typedef double f64x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(512) void score_kernel(const double* __restrict__ qbar,
                                                    const double* __restrict__ kbar, int n, int nk, double sm_scale,
                                                    double* __restrict__ scores, float* __restrict__ scores32) {
  __shared__ double qs[kSK][kST + 2];
  __shared__ double ks[kSK][kST + 2];
  const int bh = blockIdx.z;
  const int i0 = blockIdx.y * kST, j0 = blockIdx.x * kST;
  const double* qb = qbar + (int64_t)bh * n * kHeadDim;
  const double* kb = kbar + (int64_t)bh * nk * kHeadDim;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int wr = wave >> 2, wc = wave & 3;   // 64-row half, 32-column quarter
  const int li = lane & 15, lk = lane >> 4;
  const bool wave_live = i0 + wr * 64 < n && j0 + wc * 32 < nk;
  // staging: thread -> (row r, dims d0 .. d0 + 3) of each operand's chunk
  const int sr = tid >> 2, sd0 = (tid & 3) * 4;
  const bool qin = i0 + sr < n, kin = j0 + sr < nk;
  const double* qrow = qb + (int64_t)(qin ? i0 + sr : 0) * kHeadDim + sd0;
  const double* krow = kb + (int64_t)(kin ? j0 + sr : 0) * kHeadDim + sd0;
  double qv[4], kv[4];
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    qv[d] = qin ? qrow[d] : 0.0;
    kv[d] = kin ? krow[d] : 0.0;
  }
  f64x4 acc[4][2];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int c = 0; c < 2; ++c) acc[a][c] = (f64x4){0.0, 0.0, 0.0, 0.0};
  for (int kk = 0; kk < kHeadDim; kk += kSK) {
    __syncthreads();   // the previous chunk is no longer read
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      qs[sd0 + d][sr] = qv[d];
      ks[sd0 + d][sr] = kv[d];
    }
    __syncthreads();
    if (kk + kSK < kHeadDim) {
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        qv[d] = qin ? qrow[kk + kSK + d] : 0.0;
        kv[d] = kin ? krow[kk + kSK + d] : 0.0;
      }
    }
    // a wave whose 64 rows or 32 columns all lie past the matrix edge only
    // helps stage the operands.  A[i][k]: lane holds row i = li of the tile,
    // k = lk; B[k][j]: column j = li.  The fragments of the next k-step are
    // read while this step's 8 products run.
    if (wave_live) {
      double af[2][4], bf[2][2];
#pragma unroll
      for (int t = 0; t < 4; ++t) af[0][t] = qs[lk][wr * 64 + t * 16 + li];
#pragma unroll
      for (int t = 0; t < 2; ++t) bf[0][t] = ks[lk][wc * 32 + t * 16 + li];
#pragma unroll
      for (int k4 = 0; k4 < kSK; k4 += 4) {
        const int cur = (k4 / 4) & 1;
        if (k4 + 4 < kSK) {
#pragma unroll
          for (int t = 0; t < 4; ++t) af[cur ^ 1][t] = qs[k4 + 4 + lk][wr * 64 + t * 16 + li];
#pragma unroll
          for (int t = 0; t < 2; ++t) bf[cur ^ 1][t] = ks[k4 + 4 + lk][wc * 32 + t * 16 + li];
        }
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int c = 0; c < 2; ++c)
            acc[a][c] = __builtin_amdgcn_mfma_f64_16x16x4f64(af[cur][a], bf[cur][c], acc[a][c], 0, 0, 0);
      }
    }
  }
  // D tile element (4 r + lane / 16, lane % 16) sits in register r of the lane
  if (i0 + kST <= n && j0 + kST <= nk && !scores32) {
    // interior tile, float64 scores only: no per-element checks
    double* out = scores + ((int64_t)bh * n + i0 + wr * 64 + lk) * nk + j0 + wc * 32 + li;
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 2; ++c) out[(int64_t)(a * 16 + 4 * r) * nk + c * 16] = sm_scale * acc[a][c][r];
    return;
  }
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = i0 + wr * 64 + a * 16 + 4 * r + lk;
      if (i >= n) continue;
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int j = j0 + wc * 32 + c * 16 + li;
        if (j >= nk) continue;
        const double v = sm_scale * acc[a][c][r];
        const int64_t o = ((int64_t)bh * n + i) * nk + j;
        scores[o] = v;
        if (scores32) scores32[o] = (float)v;
      }
    }
}

// ---------------------------------------------------------------------------
// 2b. Per-row selection.  One workgroup per mask row; thread t owns blocks
// j = t + 256 e.  The kept set is the first k blocks of the order (score
// descending, index ascending), k = min(n, max(k_p, k_min, 1)).  It is found
// without sorting the row: the position k is the first one at which both
// conditions hold -- cumulative mass >= top_p (dropped when top_p <= 0) and
// position >= max(k_min, 1) -- and both are monotone along the order, so a
// radix descent over an order-preserving 64-bit image of the float64 scores
// finds the block at that position: per 8-bit digit, a histogram of block
// counts and masses over the candidates, then the digit whose cumulative
// (count, mass), counted from the top, first meets both conditions becomes
// the new candidate range.  The descent stops when that digit holds a single
// block; blocks with bit-identical scores left after all 64 bits are ordered
// by index.  Masses enter the histograms as 62-bit fixed-point integers so
// every sum is exact and independent of the order of the atomic adds: the
// selection is deterministic.
// ---------------------------------------------------------------------------
constexpr int kSelThreads = 256;
constexpr int kTopScan = 3;   // distinct first-digit values walked before the histogram
constexpr double kMassOne = 4611686018427387904.0;          // 2^62
static_assert(kSelThreads == 256, "one histogram bin per thread");

// Order-preserving image of a float64 (larger score -> larger key); -0 is
// folded onto +0 so equal scores give equal keys.
__device__ inline uint64_t order_key(double s) {
  const uint64_t u = (uint64_t)__double_as_longlong(s == 0.0 ? 0.0 : s);
  return (u >> 63) ? ~u : (u | (1ull << 63));
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

__device__ uint64_t block_reduce_sum_u64(uint64_t v, uint64_t* red) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  uint64_t r = red[0];
  for (int i = 1; i < kSelThreads / 64; ++i) r += red[i];
  return r;
}

struct SelCond {
  uint64_t target;   // ceil(top_p * 2^62)
  uint32_t kk;       // max(k_min, 1)
  bool any_mass;     // top_p <= 0: the mass condition always holds
  __device__ bool operator()(uint32_t cnt, uint64_t mass) const {
    return cnt >= kk && (any_mass || mass >= target);
  }
};

__device__ uint64_t block_reduce_min_u64(uint64_t v, uint64_t* red) {
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t w = __shfl_xor(v, o);
    v = w < v ? w : v;
  }
  const int wv = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[wv] = v;
  __syncthreads();
  uint64_t r = red[0];
  for (int i = 1; i < kSelThreads / 64; ++i) r = red[i] < r ? red[i] : r;
  return r;
}

__device__ uint64_t block_reduce_max_u64(uint64_t v, uint64_t* red) {
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t w = __shfl_xor(v, o);
    v = w > v ? w : v;
  }
  const int wv = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[wv] = v;
  __syncthreads();
  uint64_t r = red[0];
  for (int i = 1; i < kSelThreads / 64; ++i) r = red[i] > r ? red[i] : r;
  return r;
}

// Dynamic LDS: key[n] and mass[n] (uint64 each).
// FROM_MASS: the row holds non-negative block masses (fp32) instead of
// float64 scores; the ranking key is the mass itself and each block's share
// is mass / row total instead of the softmax of the scores.
template <bool FROM_MASS>
__global__ __launch_bounds__(kSelThreads) void select_kernel(const void* __restrict__ in, int n,
                                                             double top_p, int k_min,
                                                             int32_t* __restrict__ counts,
                                                             uint32_t* __restrict__ bitmap, int words) {
  extern __shared__ uint64_t sel_smem[];
  uint64_t* key = sel_smem;
  uint64_t* mass = sel_smem + n;
  __shared__ uint32_t hist_cnt[256];
  __shared__ uint64_t hist_mass[256];
  __shared__ uint32_t bits[kMaxBuilderBlocks / 32];
  __shared__ uint32_t ties[kMaxBuilderBlocks / 32];
  __shared__ double red[kSelThreads / 64];
  __shared__ uint64_t red64[kSelThreads / 64];
  __shared__ uint64_t sel_mass_above, tie_mass, bound_key;
  __shared__ uint32_t sel_cnt_above, sel_bin, sel_bin_cnt;
  __shared__ int bound_j;

  const int64_t row = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  auto value = [&](int j) -> double {
    return FROM_MASS ? (double)(static_cast<const float*>(in) + row * n)[j]
                     : (static_cast<const double*>(in) + row * n)[j];
  };

  for (int w = tid; w < words; w += kSelThreads) {
    bits[w] = 0u;
    ties[w] = 0u;
  }
  // scores -> row max -> exp -> row sum -> fixed-point masses and keys
  // (masses: the values themselves and their row sum)
  double m = -INFINITY;
  for (int j = tid; j < n; j += kSelThreads) {
    const double v = value(j);
    key[j] = order_key(v);
    m = fmax(m, v);
  }
  if (!FROM_MASS) m = block_reduce_max(m, red);
  double z = 0.0;
  for (int j = tid; j < n; j += kSelThreads) {
    const double x = FROM_MASS ? value(j) : exp(value(j) - m);
    mass[j] = (uint64_t)__double_as_longlong(x);
    z += x;
  }
  z = block_reduce_sum(z, red);
  uint64_t total = 0, kmin = ~0ull, kmax = 0;
  for (int j = tid; j < n; j += kSelThreads) {
    const double share = z > 0.0 ? __longlong_as_double((long long)mass[j]) / z : 0.0;
    const uint64_t q = __double2ull_rn(share * kMassOne);
    mass[j] = q;
    total += q;
    const uint64_t kj = key[j];
    kmin = kj < kmin ? kj : kmin;
    kmax = kj > kmax ? kj : kmax;
  }
  total = block_reduce_sum_u64(total, red64);
  kmin = block_reduce_min_u64(kmin, red64);
  kmax = block_reduce_max_u64(kmax, red64);

  SelCond cond;
  cond.any_mass = !(top_p > 0.0);
  cond.target = cond.any_mass ? 0 : (uint64_t)ceil(fmin(top_p, 1.0) * kMassOne);
  cond.kk = (uint32_t)(k_min > 1 ? k_min : 1);
  // k = n when top_p >= 1, when the floor reaches n, or when rounding keeps
  // the whole row's mass below top_p
  const bool keep_all = top_p >= 1.0 || cond.kk >= (uint32_t)n || !cond((uint32_t)n, total);

  uint64_t kb = 0;   // keep blocks with key > kb, and key == kb with index <= jb
  int jb = n;
  uint32_t k = (uint32_t)n;
  if (!keep_all) {
    // Descent state: every candidate agrees with `prefix` on bits >= lo; the
    // bits above the highest one in which the row's keys differ are common
    // to all blocks, so the descent starts below them.
    const uint64_t diff = kmin ^ kmax;
    int lo = diff ? 64 - __clzll((long long)diff) : 0;
    uint64_t prefix = lo == 64 ? 0 : (kmin >> lo) << lo;
    uint64_t mass_above = 0;
    uint32_t cnt_above = 0, bin_cnt = (uint32_t)n;
    // first digit: its few distinct values walked from the top with block
    // reductions (as in the wave kernel below), the histogram after that
    int dig_limit = 256;
    if (lo > 0) {
      const int shift = lo > 8 ? lo - 8 : 0;
      for (int it = 0; it < kTopScan; ++it) {
        uint64_t dm = 0;   // 1 + the largest digit below dig_limit, 0 if none
        for (int j = tid; j < n; j += kSelThreads) {
          const uint64_t kj = key[j];
          const uint64_t d = (kj >> shift) & 255;
          if ((lo == 64 || ((kj ^ prefix) >> lo) == 0) && (int)d < dig_limit && d + 1 > dm) dm = d + 1;
        }
        dm = block_reduce_max_u64(dm, red64);
        if (dm == 0) break;
        const uint64_t dmax = dm - 1;
        uint64_t c = 0, m = 0;
        for (int j = tid; j < n; j += kSelThreads) {
          const uint64_t kj = key[j];
          if ((lo == 64 || ((kj ^ prefix) >> lo) == 0) && ((kj >> shift) & 255) == dmax) {
            ++c;
            m += mass[j];
          }
        }
        c = block_reduce_sum_u64(c, red64);
        m = block_reduce_sum_u64(m, red64);
        if (cond(cnt_above + (uint32_t)c, mass_above + m)) {
          prefix = (prefix & ~(255ull << shift)) | (dmax << shift);
          lo = shift;
          bin_cnt = (uint32_t)c;
          dig_limit = 256;
          break;
        }
        cnt_above += (uint32_t)c;
        mass_above += m;
        dig_limit = (int)dmax;
      }
    }
    while (lo > 0 && bin_cnt > 1) {
      const int shift = lo > 8 ? lo - 8 : 0;
      hist_cnt[tid] = 0u;
      hist_mass[tid] = 0ull;
      __syncthreads();
      for (int j = tid; j < n; j += kSelThreads) {
        const uint64_t kj = key[j];
        if ((lo == 64 || ((kj ^ prefix) >> lo) == 0) && (int)((kj >> shift) & 255) < dig_limit) {
          const int bin = (int)((kj >> shift) & 255);
          atomicAdd(&hist_cnt[bin], 1u);
          atomicAdd((unsigned long long*)&hist_mass[bin], (unsigned long long)mass[j]);
        }
      }
      __syncthreads();
      if (wave == 0) {
        // lane l owns bins 4l .. 4l+3; the bins above them are lanes > l
        uint32_t c[4], c4 = 0;
        uint64_t ms[4], m4 = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          c[q] = hist_cnt[4 * lane + q];
          ms[q] = hist_mass[4 * lane + q];
          c4 += c[q];
          m4 += ms[q];
        }
        uint32_t cs = c4;
        uint64_t msum = m4;
        for (int o = 1; o < 64; o <<= 1) {
          const uint32_t vc = __shfl_down(cs, o);
          const uint64_t vm = __shfl_down(msum, o);
          if (lane + o < 64) {
            cs += vc;
            msum += vm;
          }
        }
        uint32_t cc = cnt_above + (cs - c4);
        uint64_t mm = mass_above + (msum - m4);
        bool before = cond(cc, mm);
#pragma unroll
        for (int q = 3; q >= 0; --q) {
          const uint32_t c2 = cc + c[q];
          const uint64_t m2 = mm + ms[q];
          const bool now = cond(c2, m2);
          if (now && !before) {
            sel_bin = (uint32_t)(4 * lane + q);
            sel_cnt_above = cc;
            sel_mass_above = mm;
            sel_bin_cnt = c[q];
          }
          before = now;
          cc = c2;
          mm = m2;
        }
      }
      __syncthreads();
      prefix = (prefix & ~(255ull << shift)) | ((uint64_t)sel_bin << shift);
      cnt_above = sel_cnt_above;
      mass_above = sel_mass_above;
      bin_cnt = sel_bin_cnt;
      lo = shift;
      dig_limit = 256;
      if (bin_cnt == 1) break;
    }
    if (bin_cnt == 1) {
      // the boundary block is the only candidate left
      for (int j = tid; j < n; j += kSelThreads) {
        const uint64_t kj = key[j];
        if (lo == 64 || ((kj ^ prefix) >> lo) == 0) {
          bound_key = kj;
          bound_j = j;
        }
      }
      __syncthreads();
      kb = bound_key;
      jb = bound_j;
      k = cnt_above + 1;
    } else {
      // bin_cnt blocks share the score `prefix` (and so one mass): the
      // boundary is the t-th of them in index order
      for (int j = tid; j < n; j += kSelThreads) {
        if (key[j] == prefix) {
          atomicOr(&ties[j >> 5], 1u << (j & 31));
          tie_mass = mass[j];   // identical for every tied block
        }
      }
      __syncthreads();
      uint32_t t = 1;
      if (!cond.any_mass && mass_above < cond.target && tie_mass > 0)
        t = (uint32_t)((cond.target - mass_above + tie_mass - 1) / tie_mass);
      if (cond.kk > cnt_above && cond.kk - cnt_above > t) t = cond.kk - cnt_above;
      if (t > bin_cnt) t = bin_cnt;
      if (wave == 0) {
        // lane l owns tie words 2l, 2l+1 (words <= 128)
        const uint32_t w0 = 2 * lane < words ? ties[2 * lane] : 0u;
        const uint32_t w1 = 2 * lane + 1 < words ? ties[2 * lane + 1] : 0u;
        const uint32_t cnt = __popc(w0) + __popc(w1);
        uint32_t incl = cnt;
        for (int o = 1; o < 64; o <<= 1) {
          const uint32_t v = __shfl_up(incl, o);
          if (lane >= o) incl += v;
        }
        const uint32_t excl = incl - cnt;
        if (excl < t && t <= incl) {
          uint32_t r = t - excl;   // r-th set bit of (w0, w1), 1-based
          int j = -1;
          for (int b = 0; b < 64; ++b) {
            const uint32_t wv = b < 32 ? w0 : w1;
            if ((wv >> (b & 31)) & 1u) {
              if (--r == 0) {
                j = 64 * lane + b;
                break;
              }
            }
          }
          bound_j = j;
        }
      }
      __syncthreads();
      kb = prefix;
      jb = bound_j;
      k = cnt_above + t;
    }
  }
  for (int j = tid; j < n; j += kSelThreads) {
    const uint64_t kj = key[j];
    if (keep_all || kj > kb || (kj == kb && j <= jb)) atomicOr(&bits[j >> 5], 1u << (j & 31));
  }
  __syncthreads();
  uint32_t* dst = bitmap + row * words;
  for (int w = tid; w < words; w += kSelThreads) dst[w] = bits[w];
  if (tid == 0) counts[row] = (int32_t)k;
}

// Same selection with one wave per row for rows of at most 64 * kWaveMaxPer
// blocks: lane l keeps the keys and masses of blocks l + 64 e in registers,
// reductions are DPP / permlane steps and broadcasts are lane reads (no LDS
// round trips), the per-digit histogram lives in the wave's own LDS slice,
// and the kept set is written as ballots (block 64 e + l is bit l of word
// pair 2e, 2e + 1).  No workgroup barrier is needed; four rows share a
// workgroup.  Rows of 1,025-1,280 blocks (PER = 20) run at three waves per
// SIMD: the 168-register cap spills a few registers, and the extra wave per
// SIMD still makes the kernel faster than two unspilled waves.
// ---------------------------------------------------------------------------
constexpr int kWaveMaxPer = 32;   // n <= 2048

// LDS accesses of one wave take effect in program order; this keeps the
// compiler from moving them across the point.
__device__ inline void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Value of lane src (wave-uniform; a negative src, from an empty ballot,
// reads lane 0 and the caller ignores the result) at every lane.
template <typename T>
__device__ inline T wave_bcast(T v, int src) {
  const int s = src < 0 ? 0 : src;
  if constexpr (sizeof(T) == 4) {
    return __builtin_bit_cast(T, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), s));
  } else {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, s);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), s);
    return __builtin_bit_cast(T, (uint64_t)lo | ((uint64_t)hi << 32));
  }
}

// Wave-wide reductions without the LDS crossbar that __shfl_xor goes
// through: DPP moves inside each row of 16 lanes (quad lanes xor 1 and xor 2,
// then the half-row mirror and the row mirror, each pairing two partial
// results), then the permlane swaps of rows 2r / 2r + 1 and of the two
// halves of the wave.  Each step combines the same two partial values at
// every lane it reaches, so for a commutative op all lanes end with one
// bitwise-identical result.
template <int CTRL>
__device__ inline uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, false);
}
template <int CTRL, typename T>
__device__ inline T dpp_of(T v) {
  if constexpr (sizeof(T) == 4) {
    return __builtin_bit_cast(T, dpp_u32<CTRL>(__builtin_bit_cast(uint32_t, v)));
  } else {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint64_t lo = dpp_u32<CTRL>((uint32_t)u), hi = dpp_u32<CTRL>((uint32_t)(u >> 32));
    return __builtin_bit_cast(T, lo | (hi << 32));
  }
}
// a, b = the value of the lower and of the upper row of a pair of rows
// (HALVES: of the two halves of the wave), at every lane of both
template <bool HALVES, typename T>
__device__ inline void swap_pair(T v, T& a, T& b) {
  if constexpr (sizeof(T) == 4) {
    const uint32_t u = __builtin_bit_cast(uint32_t, v);
    const auto r = HALVES ? __builtin_amdgcn_permlane32_swap(u, u, false, false)
                          : __builtin_amdgcn_permlane16_swap(u, u, false, false);
    a = __builtin_bit_cast(T, (uint32_t)r[0]);
    b = __builtin_bit_cast(T, (uint32_t)r[1]);
  } else {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = (uint32_t)u, hi = (uint32_t)(u >> 32);
    const auto rl = HALVES ? __builtin_amdgcn_permlane32_swap(lo, lo, false, false)
                           : __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
    const auto rh = HALVES ? __builtin_amdgcn_permlane32_swap(hi, hi, false, false)
                           : __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
    a = __builtin_bit_cast(T, (uint64_t)(uint32_t)rl[0] | ((uint64_t)(uint32_t)rh[0] << 32));
    b = __builtin_bit_cast(T, (uint64_t)(uint32_t)rl[1] | ((uint64_t)(uint32_t)rh[1] << 32));
  }
}
template <typename T, class Op>
__device__ inline T wave_reduce(T v, Op op) {
  v = op(v, dpp_of<0xB1>(v));    // quad_perm [1, 0, 3, 2]
  v = op(v, dpp_of<0x4E>(v));    // quad_perm [2, 3, 0, 1]
  v = op(v, dpp_of<0x141>(v));   // row_half_mirror
  v = op(v, dpp_of<0x140>(v));   // row_mirror
  T a, b;
  swap_pair<false>(v, a, b);
  v = op(a, b);
  swap_pair<true>(v, a, b);
  return op(a, b);
}
struct OpMax { template <typename T> __device__ T operator()(T a, T b) const { return a > b ? a : b; } };
struct OpMin { template <typename T> __device__ T operator()(T a, T b) const { return a < b ? a : b; } };
struct OpAdd { template <typename T> __device__ T operator()(T a, T b) const { return a + b; } };
struct OpFMax { __device__ double operator()(double a, double b) const { return fmax(a, b); } };
struct OpFMin { __device__ double operator()(double a, double b) const { return fmin(a, b); } };

template <int PER, bool FROM_MASS>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(PER <= 16 ? 4 : PER <= 20 ? 3 : PER <= 24 ? 2 : 1))) void select_wave_kernel(const void* __restrict__ in, int n, int64_t rows,
                                                          double top_p, int k_min, int32_t* __restrict__ counts,
                                                          uint32_t* __restrict__ bitmap, int words) {
  __shared__ uint32_t hist_cnt_all[4][256];
  __shared__ uint64_t hist_mass_all[4][256];
  __shared__ uint64_t cand_key_all[4][64];
  __shared__ uint64_t cand_mass_all[4][64];
  __shared__ int32_t cand_idx_all[4][64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + wave;
  if (row >= rows) return;
  uint32_t* hist_cnt = hist_cnt_all[wave];
  uint64_t* hist_mass = hist_mass_all[wave];
  auto value = [&](int j) -> double {
    return FROM_MASS ? (double)(static_cast<const float*>(in) + row * n)[j]
                     : (static_cast<const double*>(in) + row * n)[j];
  };

  uint64_t key[PER], mass[PER];
  uint32_t binw[(PER + 3) / 4];   // 8-bit value bins, four per word
  double m = -INFINITY, mn = INFINITY;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int j = lane + 64 * e;
    const double v = j < n ? value(j) : -INFINITY;
    key[e] = (uint64_t)__double_as_longlong(v);
    m = fmax(m, v);
    if (j < n) mn = fmin(mn, v);
  }
  m = wave_reduce(m, OpFMax());
  mn = wave_reduce(mn, OpFMin());
  // value bins: floor((v - min) * 255.5 / (max - min)), non-decreasing in v,
  // so every block of a higher bin comes before every block of a lower one
  const double bscale = m > mn ? 255.5 / (m - mn) : 0.0;
  double z = 0.0;
#pragma unroll
  for (int e = 0; e < (PER + 3) / 4; ++e) binw[e] = 0u;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int j = lane + 64 * e;
    const double v = __longlong_as_double((long long)key[e]);
    double x = 0.0;
    if (j < n) x = FROM_MASS ? v : exp(v - m);
    mass[e] = (uint64_t)__double_as_longlong(x);
    z += x;
    if (j < n) {
      const uint32_t bin = (uint32_t)((v - mn) * bscale);
      binw[e >> 2] |= (bin > 255u ? 255u : bin) << (8 * (e & 3));
    }
    key[e] = j < n ? order_key(v) : 0;
  }
  z = wave_reduce(z, OpAdd());
  // block masses as 62-bit fixed point: round(x * 2^62 / z)
  const double to_fixed = z > 0.0 ? kMassOne / z : 0.0;
  uint64_t total = 0;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int j = lane + 64 * e;
    mass[e] = j < n ? __double2ull_rn(__longlong_as_double((long long)mass[e]) * to_fixed) : 0;
    total += mass[e];
  }
  total = wave_reduce(total, OpAdd());

  SelCond cond;
  cond.any_mass = !(top_p > 0.0);
  cond.target = cond.any_mass ? 0 : (uint64_t)ceil(fmin(top_p, 1.0) * kMassOne);
  cond.kk = (uint32_t)(k_min > 1 ? k_min : 1);
  const bool keep_all = top_p >= 1.0 || cond.kk >= (uint32_t)n || !cond((uint32_t)n, total);

  uint64_t kb = 0;   // keep blocks with key > kb, and key == kb with index <= jb
  int jb = n;
  uint32_t k = (uint32_t)n;
  bool found = false;
  if (!keep_all) {
    // Histogram of (count, mass) over the value bins, scanned from the top:
    // the first bin whose cumulative (count, mass) meets both conditions holds
    // the boundary block.
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      hist_cnt[4 * lane + q] = 0u;
      hist_mass[4 * lane + q] = 0ull;
    }
    wave_lds_sync();
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int j = lane + 64 * e;
      if (j < n) {
        const int bin = (int)((binw[e >> 2] >> (8 * (e & 3))) & 255u);
        atomicAdd(&hist_cnt[bin], 1u);
        atomicAdd((unsigned long long*)&hist_mass[bin], (unsigned long long)mass[e]);
      }
    }
    wave_lds_sync();
    uint32_t c[4], c4 = 0;
    uint64_t ms[4], m4 = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      c[q] = hist_cnt[4 * lane + q];
      ms[q] = hist_mass[4 * lane + q];
      c4 += c[q];
      m4 += ms[q];
    }
    uint32_t cs = c4;
    uint64_t msum = m4;
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t vc = __shfl_down(cs, o);
      const uint64_t vm = __shfl_down(msum, o);
      if (lane + o < 64) {
        cs += vc;
        msum += vm;
      }
    }
    uint32_t cc = cs - c4;
    uint64_t mm = msum - m4;
    bool before = cond(cc, mm);
    int f_bin = -1;
    uint32_t f_cnt_above = 0, f_bin_cnt = 0;
    uint64_t f_mass_above = 0;
#pragma unroll
    for (int q = 3; q >= 0; --q) {
      const uint32_t c2 = cc + c[q];
      const uint64_t m2 = mm + ms[q];
      const bool now = cond(c2, m2);
      if (now && !before) {
        f_bin = 4 * lane + q;
        f_cnt_above = cc;
        f_mass_above = mm;
        f_bin_cnt = c[q];
      }
      before = now;
      cc = c2;
      mm = m2;
    }
    const int src = __ffsll((long long)__builtin_amdgcn_ballot_w64(f_bin >= 0)) - 1;
    const int bin_b = wave_bcast(f_bin, src);
    const uint32_t cnt_b = wave_bcast(f_cnt_above, src);
    const uint64_t mass_b = wave_bcast(f_mass_above, src);
    const uint32_t n_cand = wave_bcast(f_bin_cnt, src);
    wave_lds_sync();
    if (src >= 0 && n_cand <= 64) {
      // The bin's blocks, one per lane, ranked by (key descending, index
      // ascending); the boundary is the first of them, in that order, at which
      // both conditions hold.
      uint64_t* ck = cand_key_all[wave];
      uint64_t* cm = cand_mass_all[wave];
      int32_t* cj = cand_idx_all[wave];
      uint32_t at = 0;
#pragma unroll
      for (int e = 0; e < PER; ++e) {
        const int j = lane + 64 * e;
        const bool is_c = j < n && (int)((binw[e >> 2] >> (8 * (e & 3))) & 255u) == bin_b;
        const uint64_t bm = __builtin_amdgcn_ballot_w64(is_c);
        if (is_c) {
          const uint32_t pos = at + (uint32_t)__builtin_amdgcn_mbcnt_hi((uint32_t)(bm >> 32),
                                                                       __builtin_amdgcn_mbcnt_lo((uint32_t)bm, 0u));
          ck[pos] = key[e];
          cm[pos] = mass[e];
          cj[pos] = j;
        }
        at += (uint32_t)__popcll(bm);
      }
      wave_lds_sync();
      const bool mine = (uint32_t)lane < n_cand;
      const uint64_t my_k = mine ? ck[lane] : 0;
      const uint64_t my_m = mine ? cm[lane] : 0;
      const int my_j = mine ? cj[lane] : 0;
      uint32_t rank = 0;
      uint64_t cum = 0;
      for (uint32_t t = 0; t < n_cand; ++t) {
        const uint64_t kt = ck[t];
        const int jt = cj[t];
        const bool pre = kt > my_k || (kt == my_k && jt < my_j);
        rank += pre ? 1u : 0u;
        cum += pre ? cm[t] : 0ull;
      }
      wave_lds_sync();
      const bool ok = mine && cond(cnt_b + rank + 1, mass_b + cum + my_m);
      uint32_t r_min = ok ? rank : 0xffffffffu;
      r_min = wave_reduce(r_min, OpMin());
      const int src2 = __ffsll((long long)__builtin_amdgcn_ballot_w64(ok && rank == r_min)) - 1;
      if (src2 >= 0) {
        kb = wave_bcast(my_k, src2);
        jb = wave_bcast(my_j, src2);
        k = cnt_b + r_min + 1;
        found = true;
      }
    }
  }
  if (!keep_all && !found) {
    // Fallback: radix descent over the order keys (a bin holding more than 64
    // blocks).
    uint64_t kmin = ~0ull, kmax = 0;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int j = lane + 64 * e;
      if (j < n) {
        kmin = key[e] < kmin ? key[e] : kmin;
        kmax = key[e] > kmax ? key[e] : kmax;
      }
    }
    kmin = wave_reduce(kmin, OpMin());
    kmax = wave_reduce(kmax, OpMax());
    const uint64_t diff = kmin ^ kmax;
    int lo = diff ? 64 - __clzll((long long)diff) : 0;
    uint64_t prefix = lo == 64 ? 0 : (kmin >> lo) << lo;
    uint64_t mass_above = 0;
    uint32_t cnt_above = 0, bin_cnt = (uint32_t)n;
    // The first digit (below the bits all keys share) takes few values across
    // a row (the sign and top exponent bits of the scores), so histogram adds
    // would pile onto a handful of LDS words.  Walk its distinct values from
    // the top with wave reductions instead; after kTopScan values without the
    // boundary, the histogram takes the remaining (smaller) digits.
    int dig_limit = 256;
    if (lo > 0) {
      const int shift = lo > 8 ? lo - 8 : 0;
      for (int it = 0; it < kTopScan; ++it) {
        int dmax = -1;
#pragma unroll
        for (int e = 0; e < PER; ++e) {
          const int j = lane + 64 * e;
          const int d = (int)((key[e] >> shift) & 255);
          if (j < n && (lo == 64 || ((key[e] ^ prefix) >> lo) == 0) && d < dig_limit) dmax = d > dmax ? d : dmax;
        }
        dmax = wave_reduce(dmax, OpMax());
        if (dmax < 0) break;
        uint32_t c = 0;
        uint64_t m = 0;
#pragma unroll
        for (int e = 0; e < PER; ++e) {
          const int j = lane + 64 * e;
          if (j < n && (lo == 64 || ((key[e] ^ prefix) >> lo) == 0) && (int)((key[e] >> shift) & 255) == dmax) {
            ++c;
            m += mass[e];
          }
        }
        c = wave_reduce(c, OpAdd());
        m = wave_reduce(m, OpAdd());
        if (cond(cnt_above + c, mass_above + m)) {
          // the boundary block has this digit
          prefix = (prefix & ~(255ull << shift)) | ((uint64_t)dmax << shift);
          lo = shift;
          bin_cnt = c;
          dig_limit = 256;
          break;
        }
        cnt_above += c;
        mass_above += m;
        dig_limit = dmax;
      }
    }
    while (lo > 0 && bin_cnt > 1) {
      const int shift = lo > 8 ? lo - 8 : 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        hist_cnt[4 * lane + q] = 0u;
        hist_mass[4 * lane + q] = 0ull;
      }
      wave_lds_sync();
#pragma unroll
      for (int e = 0; e < PER; ++e) {
        const int j = lane + 64 * e;
        if (j < n && (lo == 64 || ((key[e] ^ prefix) >> lo) == 0) && (int)((key[e] >> shift) & 255) < dig_limit) {
          const int bin = (int)((key[e] >> shift) & 255);
          atomicAdd(&hist_cnt[bin], 1u);
          atomicAdd((unsigned long long*)&hist_mass[bin], (unsigned long long)mass[e]);
        }
      }
      wave_lds_sync();
      uint32_t c[4], c4 = 0;
      uint64_t ms[4], m4 = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        c[q] = hist_cnt[4 * lane + q];
        ms[q] = hist_mass[4 * lane + q];
        c4 += c[q];
        m4 += ms[q];
      }
      wave_lds_sync();
      uint32_t cs = c4;
      uint64_t msum = m4;
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t vc = __shfl_down(cs, o);
        const uint64_t vm = __shfl_down(msum, o);
        if (lane + o < 64) {
          cs += vc;
          msum += vm;
        }
      }
      uint32_t cc = cnt_above + (cs - c4);
      uint64_t mm = mass_above + (msum - m4);
      bool before = cond(cc, mm);
      int f_bin = -1;
      uint32_t f_cnt_above = 0, f_bin_cnt = 0;
      uint64_t f_mass_above = 0;
#pragma unroll
      for (int q = 3; q >= 0; --q) {
        const uint32_t c2 = cc + c[q];
        const uint64_t m2 = mm + ms[q];
        const bool now = cond(c2, m2);
        if (now && !before) {
          f_bin = 4 * lane + q;
          f_cnt_above = cc;
          f_mass_above = mm;
          f_bin_cnt = c[q];
        }
        before = now;
        cc = c2;
        mm = m2;
      }
      const int src = __ffsll((long long)__builtin_amdgcn_ballot_w64(f_bin >= 0)) - 1;
      const int bin = wave_bcast(f_bin, src);
      cnt_above = wave_bcast(f_cnt_above, src);
      mass_above = wave_bcast(f_mass_above, src);
      bin_cnt = wave_bcast(f_bin_cnt, src);
      prefix = (prefix & ~(255ull << shift)) | ((uint64_t)bin << shift);
      lo = shift;
      dig_limit = 256;
      if (bin_cnt == 1) break;
    }
    if (bin_cnt == 1) {
      // the boundary block is the only candidate left
      uint64_t my_key = 0;
      int my_j = -1;
#pragma unroll
      for (int e = 0; e < PER; ++e) {
        const int j = lane + 64 * e;
        if (j < n && (lo == 64 || ((key[e] ^ prefix) >> lo) == 0)) {
          my_key = key[e];
          my_j = j;
        }
      }
      const int src = __ffsll((long long)__builtin_amdgcn_ballot_w64(my_j >= 0)) - 1;
      kb = wave_bcast(my_key, src);
      jb = wave_bcast(my_j, src);
      k = cnt_above + 1;
    } else {
      // bin_cnt blocks share the score `prefix` (and so one mass): the
      // boundary is the t-th of them in index order
      uint64_t my_mass = 0;
      bool has_tie = false;
#pragma unroll
      for (int e = 0; e < PER; ++e) {
        const int j = lane + 64 * e;
        if (j < n && key[e] == prefix) {
          my_mass = mass[e];
          has_tie = true;
        }
      }
      const int src = __ffsll((long long)__builtin_amdgcn_ballot_w64(has_tie)) - 1;
      const uint64_t tie_mass = wave_bcast(my_mass, src);
      uint32_t t = 1;
      if (!cond.any_mass && mass_above < cond.target && tie_mass > 0)
        t = (uint32_t)((cond.target - mass_above + tie_mass - 1) / tie_mass);
      if (cond.kk > cnt_above && cond.kk - cnt_above > t) t = cond.kk - cnt_above;
      if (t > bin_cnt) t = bin_cnt;
      // tied blocks in index order: ballot e covers blocks 64 e .. 64 e + 63
      uint32_t before_e = 0;
      int found = -1;
#pragma unroll
      for (int e = 0; e < PER; ++e) {
        const int j = lane + 64 * e;
        const uint64_t bm = __builtin_amdgcn_ballot_w64(j < n && key[e] == prefix);
        const uint32_t c = (uint32_t)__popcll(bm);
        if (found < 0 && before_e + c >= t) {
          uint64_t x = bm;
          for (uint32_t r = t - before_e; r > 1; --r) x &= x - 1;
          found = 64 * e + (__ffsll((long long)x) - 1);
        }
        before_e += c;
      }
      kb = prefix;
      jb = found;
      k = cnt_above + t;
    }
  }
  uint32_t* dst = bitmap + row * words;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int j = lane + 64 * e;
    const bool keep = j < n && (keep_all || key[e] > kb || (key[e] == kb && j <= jb));
    const uint64_t bm = __builtin_amdgcn_ballot_w64(keep);
    if (lane < 2 && 2 * e + lane < words) dst[2 * e + lane] = (uint32_t)(bm >> (32 * lane));
  }
  if (lane == 0) counts[row] = (int32_t)k;
}

// ---------------------------------------------------------------------------
// 3. Exclusive scan of the row counts into row_ptr.  Workgroup b scans rows
// [1024 b, 1024 b + 1024): it first sums every count before its range itself
// (coalesced reads; the counts are small and L2-resident), then scans its own
// 1024 counts with wave prefix sums.  No inter-workgroup communication.
// ---------------------------------------------------------------------------
constexpr int kScanThreads = 1024;

__device__ inline int32_t wave_incl_scan(int32_t v, int lane) {
  for (int o = 1; o < 64; o <<= 1) {
    const int32_t u = __shfl_up(v, o);
    if (lane >= o) v += u;
  }
  return v;
}

__global__ __launch_bounds__(kScanThreads) void scan_kernel(const int32_t* __restrict__ counts, int64_t rows,
                                                            int32_t* __restrict__ row_ptr) {
  __shared__ int32_t wsum[kScanThreads / 64];
  __shared__ int32_t base_s;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t r0 = (int64_t)blockIdx.x * kScanThreads;
  // sum of all counts before this workgroup's range
  int32_t before = 0;
  for (int64_t r = tid; r < r0; r += kScanThreads) before += counts[r];
  for (int o = 32; o > 0; o >>= 1) before += __shfl_xor(before, o);
  if (lane == 0) wsum[wave] = before;
  __syncthreads();
  if (tid == 0) {
    int32_t t = 0;
    for (int w = 0; w < kScanThreads / 64; ++w) t += wsum[w];
    base_s = t;
  }
  __syncthreads();
  const int64_t r = r0 + tid;
  const int32_t c = r < rows ? counts[r] : 0;
  const int32_t incl = wave_incl_scan(c, lane);
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  int32_t off = base_s;
  for (int w = 0; w < wave; ++w) off += wsum[w];
  if (r < rows) row_ptr[r + 1] = off + incl;
  if (r == 0) row_ptr[0] = 0;
}

// ---------------------------------------------------------------------------
// 4. Compact each row's bitmap into ascending col_idx (one wave per row; each
// lane holds two consecutive 32-bit words, so n <= 4096).  The row is walked
// 64 blocks at a time: lane l owns block 64 c + l of chunk c and writes it at
// the chunk's base plus the number of set bits below it, so every store of
// the wave is contiguous whatever the row's density.
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
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  int32_t* dst = col_idx + row_ptr[row];
  const int chunks = (words + 1) / 2;
  for (int ch = 0; ch < chunks; ++ch) {
    const uint64_t bits = (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)a, ch) |
                          ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)c, ch) << 32);
    if ((bits >> lane) & 1ull) dst[__popcll(bits & below)] = ch * 64 + lane;
    dst += __popcll(bits);
  }
}

// ---------------------------------------------------------------------------
// 5. Work plan: head units u = b * H + h with cost sum_i (blocks(b,h,i) + 1),
// a listed kv block counting as per_id 64-token blocks (2 for kv blocks of 128),
// are assigned to the 8 XCDs greedily, heaviest first, each to the
// least-loaded XCD that still has room (equal unit counts per XCD); the order
// lists the units XCD by XCD, ascending unit id inside an XCD.  One
// workgroup, everything in LDS: costs, a rank sort by (cost desc, id asc),
// the greedy pass on one wave (the eight loads live in registers, the sorted
// costs are read lane by lane, so a step is a few dozen ALU operations), then
// the placement of every unit in parallel.  Beyond kPlanMaxUnits units the
// natural order is kept.
// ---------------------------------------------------------------------------
constexpr int kPlanMaxUnits = 4096;

// Minimum of a 64-bit value with the value a DPP pattern brings in; lanes the
// pattern gives no source keep their own.
template <int kCtrl>
__device__ inline uint64_t dpp_min_u64(uint64_t v) {
  const int lo = (int)(uint32_t)v, hi = (int)(uint32_t)(v >> 32);
  const uint32_t olo = (uint32_t)__builtin_amdgcn_update_dpp(lo, lo, kCtrl, 0xF, 0xF, false);
  const uint32_t ohi = (uint32_t)__builtin_amdgcn_update_dpp(hi, hi, kCtrl, 0xF, 0xF, false);
  const uint64_t o = (uint64_t)ohi << 32 | olo;
  return o < v ? o : v;
}

__global__ __launch_bounds__(256) void plan_kernel(const int32_t* __restrict__ row_ptr, int mask_batch, int B,
                                                   int H, int n, int per_id, int32_t* __restrict__ order) {
  __shared__ int32_t cost[kPlanMaxUnits];
  __shared__ int32_t by_cost[kPlanMaxUnits];
  __shared__ int32_t sorted_cost[kPlanMaxUnits];
  __shared__ uint8_t xcd_of[kPlanMaxUnits];
  const int U = B * H;
  const int tid = threadIdx.x;
  if (U > kPlanMaxUnits) {
    for (int u = tid; u < U; u += 256) order[u] = u;
    return;
  }
  for (int u = tid; u < U; u += 256) {
    const int b = u / H, h = u % H;
    const int64_t r0 = ((int64_t)(mask_batch > 1 ? b : 0) * H + h) * n;
    cost[u] = (row_ptr[r0 + n] - row_ptr[r0]) * per_id + n;
  }
  __syncthreads();
  for (int u = tid; u < U; u += 256) {
    const int32_t cu = cost[u];
    int rank = 0;
    for (int v = 0; v < U; ++v) {
      const int32_t cv = cost[v];
      rank += (cv > cu || (cv == cu && v < u)) ? 1 : 0;
    }
    by_cost[rank] = u;
    sorted_cost[rank] = cu;
  }
  __syncthreads();
  const int base_cap = U / kNumXcd, extra = U % kNumXcd;
  if (tid < 64) {
    // Lane x < 8 owns XCD x; its key (load << 3 | x) orders by load, then id,
    // and a full XCD (or a lane beyond 8) carries the largest key.
    int64_t load = 0;
    int left = tid < kNumXcd ? base_cap + (tid < extra ? 1 : 0) : 0;
    for (int p0 = 0; p0 < U; p0 += 64) {
      const int mine_p = p0 + tid;
      const int32_t c_lane = mine_p < U ? sorted_cost[mine_p] : 0;
      const int steps = U - p0 < 64 ? U - p0 : 64;
      int mine = 0;
      for (int j = 0; j < steps; ++j) {
        const int32_t c = __builtin_amdgcn_readlane(c_lane, j);
        uint64_t key = left > 0 ? ((uint64_t)load << 3 | (uint64_t)tid) : ~0ull;
        key = dpp_min_u64<0xB1>(key);   // quad_perm [1,0,3,2]
        key = dpp_min_u64<0x4E>(key);   // quad_perm [2,3,0,1]
        key = dpp_min_u64<0x114>(key);  // row_shr:4 -> lanes 4..7 hold the minimum of lanes 0..7
        const int best = __builtin_amdgcn_readlane((int)(uint32_t)key, 4) & (kNumXcd - 1);
        load += tid == best ? c : 0;
        left -= tid == best ? 1 : 0;
        mine = tid == j ? best : mine;
      }
      if (mine_p < U) xcd_of[by_cost[mine_p]] = (uint8_t)mine;
    }
  }
  __syncthreads();
  // Unit u lands after every unit of a lower XCD and every lower unit of its own.
  for (int u = tid; u < U; u += 256) {
    const int x = xcd_of[u];
    int pos = x * base_cap + (x < extra ? x : extra);
    for (int v = 0; v < u; ++v) pos += xcd_of[v] == x ? 1 : 0;
    order[pos] = u;
  }
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

hipError_t launch_pool_fp8(TensorArg q, const float* q_scale, TensorArg k, const float* k_scale, int B, int S,
                           int H, int kvb, KeyScale ks, double* qbar, double* kbar, hipStream_t st) {
  const int n = blocks_of(S), nk = (S + kvb - 1) / kvb;
  hipLaunchKernelGGL(pool_fp8_kernel, dim3(n, H, 2 * B), dim3(64), 0, st, q, q_scale, k, k_scale, S, H, n, kvb, nk,
                     ks, qbar, kbar);
  return hipGetLastError();
}

hipError_t launch_means_from_sums(const double* q_sums, const double* k_sums, int B, int S, int H, int kvb,
                                  double* qbar, double* kbar, hipStream_t st) {
  const int n = blocks_of(S), nk = (S + kvb - 1) / kvb;
  hipLaunchKernelGGL(means_from_sums_kernel, dim3(n, H, 2 * B), dim3(kHeadDim), 0, st, q_sums, k_sums, S, H, n, kvb,
                     nk, qbar, kbar);
  return hipGetLastError();
}

hipError_t launch_pool(chorus_dtype dt, TensorArg q, TensorArg k, int B, int S, int H, int kvb, KeyScale ks,
                       double* qbar, double* kbar, hipStream_t st) {
  const int n = blocks_of(S), nk = (S + kvb - 1) / kvb;
  hipLaunchKernelGGL(pool_kernel, dim3(n, H, 2 * B), dim3(64), 0, st, q, k, S, H, n, kvb, nk, dt == CHORUS_BF16,
                     ks, qbar, kbar);
  return hipGetLastError();
}

namespace {
template <bool FROM_MASS>
hipError_t launch_select(const void* in, int64_t rows, int n, double top_p, int k_min, int32_t* counts,
                         uint32_t* bitmap, int words, hipStream_t st) {
  const dim3 wave_grid((unsigned)((rows + 3) / 4)), wave_block(256);
  if (n <= 64 * 8) {
    hipLaunchKernelGGL((select_wave_kernel<8, FROM_MASS>), wave_grid, wave_block, 0, st, in, n, rows, top_p, k_min,
                       counts, bitmap, words);
  } else if (n <= 64 * 16) {
    hipLaunchKernelGGL((select_wave_kernel<16, FROM_MASS>), wave_grid, wave_block, 0, st, in, n, rows, top_p, k_min,
                       counts, bitmap, words);
  } else if (n <= 64 * 20) {
    hipLaunchKernelGGL((select_wave_kernel<20, FROM_MASS>), wave_grid, wave_block, 0, st, in, n, rows, top_p, k_min,
                       counts, bitmap, words);
  } else if (n <= 64 * 24) {
    hipLaunchKernelGGL((select_wave_kernel<24, FROM_MASS>), wave_grid, wave_block, 0, st, in, n, rows, top_p, k_min,
                       counts, bitmap, words);
  } else if (n <= 64 * kWaveMaxPer) {
    hipLaunchKernelGGL((select_wave_kernel<kWaveMaxPer, FROM_MASS>), wave_grid, wave_block, 0, st, in, n, rows,
                       top_p, k_min, counts, bitmap, words);
  } else {
    const size_t shmem = 2 * (size_t)n * sizeof(uint64_t);
    hipLaunchKernelGGL((select_kernel<FROM_MASS>), dim3((unsigned)rows), dim3(kSelThreads), shmem, st, in, n, top_p,
                       k_min, counts, bitmap, words);
  }
  return hipGetLastError();
}
}  // namespace

hipError_t launch_score_select(const double* qbar, const double* kbar, int B, int H, int n, int nk,
                               double sm_scale, double top_p, int k_min, double* scores, int32_t* counts,
                               uint32_t* bitmap, int words, float* block_scores, hipStream_t st) {
  const int tiles_q = (n + kST - 1) / kST, tiles_k = (nk + kST - 1) / kST;
  hipLaunchKernelGGL(score_kernel, dim3(tiles_k, tiles_q, B * H), dim3(512), 0, st, qbar, kbar, n, nk, sm_scale,
                     scores, block_scores);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_select<false>(scores, (int64_t)B * H * n, nk, top_p, k_min, counts, bitmap, words, st);
}

hipError_t launch_select_from_mass(const float* mass, int64_t rows, int n, double top_p, int k_min,
                                   int32_t* counts, uint32_t* bitmap, int words, hipStream_t st) {
  return launch_select<true>(mass, rows, n, top_p, k_min, counts, bitmap, words, st);
}

hipError_t launch_scan_counts(const int32_t* counts, int64_t rows, int32_t* row_ptr, hipStream_t st) {
  const unsigned blocks = (unsigned)((rows + kScanThreads - 1) / kScanThreads);
  hipLaunchKernelGGL(scan_kernel, dim3(blocks), dim3(kScanThreads), 0, st, counts, rows, row_ptr);
  return hipGetLastError();
}

hipError_t launch_compact(const uint32_t* bitmap, int words, const int32_t* row_ptr, int64_t rows, int32_t* col_idx,
                          hipStream_t st) {
  hipLaunchKernelGGL(compact_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, bitmap, words, row_ptr,
                     rows, col_idx);
  return hipGetLastError();
}

hipError_t launch_plan(const int32_t* row_ptr, int mask_batch, int B, int H, int n, int per_id, int32_t* order,
                       hipStream_t st) {
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(256), 0, st, row_ptr, mask_batch, B, H, n, per_id, order);
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
