// True block attention mass and mask coverage (Chorus II Sec. 3.2 "Mask
// Caching and Retrieval": a historical request's masks are selected from its
// own attention map; Sec. 3.2 Obs. 1: a mask is judged by the share of a
// request's attention mass that falls inside its blocks).
//
// block_mass_kernel: one workgroup per (request, head, q-block i), two waves
// of 32 queries.  For every kv block j it recomputes S^T = K_j Q^T with
// v_mfma_f32_32x32x16 (as the attention kernel does: each lane holds 32
// scores of one query), turns the scores into the dense attention
// probabilities with the log-sum-exp of the dense forward pass,
// p = 2^(s log2(e) sm_scale - lse log2(e)), and sums them over the block's
// queries and keys: mass[i, j] = sum / |T_i|.  For kv blocks of 128 tokens the
// sums of the two 64-key halves are added before the division.  K tiles are double-buffered in
// LDS with direct global -> LDS loads; one barrier per kv block, which also
// publishes the two waves' partial sums.
#include "attn_common.h"

namespace chorus {
namespace {

constexpr int kMassTile = kBlock * kHeadDim * 2;   // 16 KB per 16-bit K tile

__device__ inline int km_swz(int r, int c) { return c ^ (r & 15); }

template <bool BF16>
struct MassElt;
template <>
struct MassElt<true> {
  using vec8 = bf16x8;
  using scalar = __bf16;
  static __device__ inline f32x16 mfma(vec8 a, vec8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <>
struct MassElt<false> {
  using vec8 = f16x8;
  using scalar = _Float16;
  static __device__ inline f32x16 mfma(vec8 a, vec8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
};

// This wave's half of a 64 x 128 K tile: instruction u fills LDS rows
// 8u + 4 wave .. + 3 (lane-linear), each lane fetching the global chunk that
// the swizzle places at its slot; rows past the sequence end re-read row S - 1.
__device__ inline void load_k_half(uint32_t lds, const char* base, uint32_t ss, int j, int S, int wave, int lane) {
  const int r0 = 4 * wave + (lane >> 4), p = lane & 15;
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const int r = 8 * u + r0;
    const int tok = min(j * kBlock + r, S - 1);
    dma16(lds + wave * 1024 + u * 2048, base, (uint32_t)tok * ss + (uint32_t)km_swz(r, p) * 16);
  }
}

template <bool BF16>
__global__ __launch_bounds__(128) __attribute__((amdgpu_waves_per_eu(2)))
void block_mass_kernel(TensorArg q, TensorArg k, const float* __restrict__ lse, int S, int H, int n,
                       float sm_scale, KeyScale ks, bool kv2, float* __restrict__ mass) {
  using E = MassElt<BF16>;
  using vec8 = typename E::vec8;
  using scalar = typename E::scalar;
  __shared__ __attribute__((aligned(1024))) char k_s[2][kMassTile];
  __shared__ float red[2][2];

  const int i = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int l32 = lane & 31, hl = lane >> 5;

  const char* kbase = static_cast<const char*>(k.data) + ((int64_t)b * k.sb + (int64_t)h * k.sh) * 2;
  const uint32_t kss = (uint32_t)(k.ss * 2);
  const uint32_t lds0 = (uint32_t)(size_t)(__attribute__((address_space(3))) char*)&k_s[0][0];
  load_k_half(lds0, kbase, kss, 0, S, wave, lane);

  const int qrow = i * kBlock + wave * 32 + l32;
  const bool q_valid = qrow < S;
  vec8 qf[8];
  {
    const uint16_t* qp = static_cast<const uint16_t*>(q.data) + (int64_t)b * q.sb + (int64_t)qrow * q.ss +
                         (int64_t)h * q.sh + 8 * hl;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      if (q_valid) {
        qf[s] = *reinterpret_cast<const vec8*>(qp + 16 * s);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[s][e] = (scalar)0.f;
      }
    }
  }
  const float lse2 = q_valid ? lse[((int64_t)b * H + h) * S + qrow] * kLog2e : 0.f;
  const float cl2 = sm_scale * kLog2e;
  const float cnt_i = (float)min(kBlock, S - i * kBlock);
  __builtin_amdgcn_s_waitcnt(0xF70);   // vmcnt(0): Q and the first K tile
  __syncthreads();

  const int k_row_off = l32 * 256;
  const int k_swzl = l32 & 15;
  // kv2: kv blocks of 128 tokens, each the sum of two 64-token halves
  const int nk = kv2 ? (n + 1) / 2 : n;
  float* out = mass + (((int64_t)b * H + h) * n + i) * nk;
  float half = 0.f;   // first half of the current 128-token block (thread 0)
  for (int j = 0; j < n; ++j) {
    if (j + 1 < n) load_k_half(lds0 + ((j + 1) & 1) * kMassTile, kbase, kss, j + 1, S, wave, lane);
    const char* kt = &k_s[j & 1][0];
    f32x16 sacc[2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[t][r] = 0.f;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int koff = k_row_off + (((2 * s + hl) ^ k_swzl) << 4);
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const vec8 kf = *reinterpret_cast<const vec8*>(kt + t * 32 * 256 + koff);
        sacc[t] = E::mfma(kf, qf[s], sacc[t]);
      }
    }
    // first-frame keys (Eq. 1): their logits count beta times
    if (j * kBlock < ks.n_first) {
      const int lim = ks.n_first - j * kBlock;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (32 * t + 8 * (r >> 2) + 4 * hl + (r & 3) < lim) sacc[t][r] *= ks.beta;
    }
    float sum = 0.f;
    const bool partial = j * kBlock + kBlock > S;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 32 * t + 8 * (r >> 2) + 4 * hl + (r & 3);
        const float p = __builtin_amdgcn_exp2f(sacc[t][r] * cl2 - lse2);
        sum += (!partial || j * kBlock + key < S) ? p : 0.f;
      }
    sum = q_valid ? sum : 0.f;
    for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
    if (lane == 0) red[j & 1][wave] = sum;
    CHORUS_WAIT_VMCNT(0);   // K_{j+1} landed
    __syncthreads();
    if (tid == 0) {
      const float v = red[j & 1][0] + red[j & 1][1];
      if (!kv2) {
        out[j] = v / cnt_i;
      } else if (j & 1) {
        out[j >> 1] = (half + v) / cnt_i;
      } else if (j == n - 1) {
        out[j >> 1] = v / cnt_i;
      } else {
        half = v;
      }
    }
  }
}

// Coverage of a mask: one workgroup per (request, head); thread t sums the
// masses of the blocks listed in rows t, t + 256, ... weighted by the rows'
// valid-token counts, in float64.
__global__ __launch_bounds__(256) void coverage_kernel(const int32_t* __restrict__ row_ptr,
                                                       const int32_t* __restrict__ col_idx, int mask_batch,
                                                       const float* __restrict__ mass, int S, int H, int n, int nk,
                                                       double* __restrict__ coverage) {
  __shared__ double red[4];
  const int h = blockIdx.x, b = blockIdx.y;
  const int tid = threadIdx.x;
  const float* mb = mass + ((int64_t)b * H + h) * n * nk;
  double acc = 0.0;
  for (int i = tid; i < n; i += 256) {
    const int64_t r = ((int64_t)(mask_batch > 1 ? b : 0) * H + h) * n + i;
    double row = 0.0;
    for (int e = row_ptr[r]; e < row_ptr[r + 1]; ++e) {
      const int j = col_idx[e];
      if (j >= 0 && j < nk) row += (double)mb[(int64_t)i * nk + j];
    }
    acc += row * (double)min(kBlock, S - i * kBlock);
  }
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if ((tid & 63) == 0) red[tid >> 6] = acc;
  __syncthreads();
  if (tid == 0) coverage[(int64_t)b * H + h] = (red[0] + red[1] + red[2] + red[3]) / (double)S;
}

}  // namespace

hipError_t launch_block_mass(chorus_dtype dt, TensorArg q, TensorArg k, const float* lse, int B, int S, int H,
                             float sm_scale, KeyScale ks, int kvb, float* mass, hipStream_t st) {
  const bool kv2 = kvb == 2 * kBlock;
  const int n = blocks_of(S);
  const dim3 grid(n, H, B), block(128);
  if (dt == CHORUS_BF16)
    hipLaunchKernelGGL(block_mass_kernel<true>, grid, block, 0, st, q, k, lse, S, H, n, sm_scale, ks, kv2, mass);
  else
    hipLaunchKernelGGL(block_mass_kernel<false>, grid, block, 0, st, q, k, lse, S, H, n, sm_scale, ks, kv2, mass);
  return hipGetLastError();
}

hipError_t launch_coverage(const int32_t* row_ptr, const int32_t* col_idx, int mask_batch, const float* mass, int B,
                           int S, int H, int kvb, double* coverage, hipStream_t st) {
  const int n = blocks_of(S), nk = (S + kvb - 1) / kvb;
  hipLaunchKernelGGL(coverage_kernel, dim3(H, B), dim3(256), 0, st, row_ptr, col_idx, mask_batch, mass, S, H, n, nk,
                     coverage);
  return hipGetLastError();
}

}  // namespace chorus
