// FP8 (OCP e4m3fn) blockwise quantiser for the FP8 attention path
// (Chorus II Sec. 3.2 "Efficient block-sparse kernel": FP8 products with
// high-precision accumulation).  One scale per (request, head, 64-token block):
//   amax = max|x|, inv = 448 / amax (IEEE fp32 divide), code = e4m3fn RNE of
//   clamp(x * inv, -448, 448), scale = amax / 448; amax == 0 -> inv 0, scale 1.
//   Blocks with amax < 2^-64 take x and amax times 2^64 (exact) before the
//   reciprocal, which would overflow below 448 / FLT_MAX; the codes depend on
//   x / amax only, so every other block is unchanged.
// HBM-bound: each value is read once (2 bytes) and written once (1 byte).
// The SUMS variant also writes, per block, the float64 sum over its valid
// tokens of each of the 128 columns (first-frame tokens weighted by beta when
// a key scale is given, Eq. 1): the mask builder's block means (Sec. 3.2
// Obs. 2) then need no second pass over Q and K.
#include "chorus_internal.h"

namespace chorus {
namespace {

__device__ inline float to_f32(uint16_t bits, bool is_bf16) {
  if (is_bf16) return __uint_as_float(uint32_t(bits) << 16);
  return static_cast<float>(*reinterpret_cast<const _Float16*>(&bits));
}

// One workgroup of 256 threads per (b, h, block); thread t owns tokens
// t/16 + 16u (u = 0..3) and the 8-value column chunk (t % 16) * 8.  The
// grid runs the heads fastest, so the workgroups in flight together cover
// whole token rows of the [B, S, H, D] tensor rather than one head's 256
// bytes of many rows.
template <bool SUMS>
__global__ __launch_bounds__(256) void quant_fp8_kernel(TensorArg x, TensorArg codes, int S, int H, int n,
                                                        bool bf16, float* __restrict__ scales, KeyScale ks,
                                                        double* __restrict__ sums) {
  __shared__ float red[4];
  __shared__ double part[SUMS ? 4 * kHeadDim : 1];   // per-wave column sums
  const int h = blockIdx.x, blk = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const int c = (tid & 15) * 8;
  const int t0 = blk * kBlock;
  const int cnt = min(kBlock, S - t0);
  const uint16_t* src = static_cast<const uint16_t*>(x.data) + (int64_t)b * x.sb + (int64_t)h * x.sh + c;
  uint8_t* dst = static_cast<uint8_t*>(const_cast<void*>(codes.data)) + (int64_t)b * codes.sb +
                 (int64_t)h * codes.sh + c;
  // all four loads of the thread are issued before the first is used
  uint4 raw[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int tok = (tid >> 4) + 16 * u;
    raw[u] = tok < cnt ? *reinterpret_cast<const uint4*>(src + (int64_t)(t0 + tok) * x.ss) : make_uint4(0, 0, 0, 0);
  }
  float v[4][8];
  float amax = 0.f;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const uint32_t w[4] = {raw[u].x, raw[u].y, raw[u].z, raw[u].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[u][2 * e] = to_f32(uint16_t(w[e] & 0xffff), bf16);
      v[u][2 * e + 1] = to_f32(uint16_t(w[e] >> 16), bf16);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf(v[u][e]));
  }
  if (SUMS) {
    // column sums of the thread's four tokens (rows past the block end hold
    // zeros), then over the four token rows of the wave (lanes l ^ 16, l ^ 32)
    double acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.0;
    const double beta = (double)ks.beta;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const double wt = t0 + (tid >> 4) + 16 * u < ks.n_first ? beta : 1.0;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] = __builtin_fma(wt, (double)v[u][e], acc[e]);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      acc[e] += __shfl_xor(acc[e], 16);
      acc[e] += __shfl_xor(acc[e], 32);
    }
    if ((tid & 63) < 16) {
#pragma unroll
      for (int e = 0; e < 8; ++e) part[(tid >> 6) * kHeadDim + c + e] = acc[e];
    }
  }
  for (int o = 32; o > 0; o >>= 1) amax = fmaxf(amax, __shfl_xor(amax, o));
  if ((tid & 63) == 0) red[tid >> 6] = amax;
  __syncthreads();
  amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  if (SUMS && tid < kHeadDim)
    sums[(((int64_t)b * H + h) * n + blk) * kHeadDim + tid] =
        (part[tid] + part[kHeadDim + tid]) + (part[2 * kHeadDim + tid] + part[3 * kHeadDim + tid]);
  const float up = amax < 0x1p-64f ? 0x1p64f : 1.f;
  const float inv = amax > 0.f ? 448.f / (amax * up) : 0.f;
  if (tid == 0) scales[((int64_t)b * H + h) * n + blk] = amax > 0.f ? amax / 448.f : 1.f;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int tok = (tid >> 4) + 16 * u;
    if (tok >= cnt) continue;
    int packed[2];
#pragma unroll
    for (int hw = 0; hw < 2; ++hw) {
      float y[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) y[e] = fminf(fmaxf((v[u][4 * hw + e] * up) * inv, -448.f), 448.f);
      int word = __builtin_amdgcn_cvt_pk_fp8_f32(y[0], y[1], 0, false);
      word = __builtin_amdgcn_cvt_pk_fp8_f32(y[2], y[3], word, true);
      packed[hw] = word;
    }
    *reinterpret_cast<uint2*>(dst + (int64_t)(t0 + tok) * codes.ss) = make_uint2(packed[0], packed[1]);
  }
}

}  // namespace

hipError_t launch_quant_fp8(chorus_dtype in_dt, TensorArg x, TensorArg codes, int B, int S, int H, float* scales,
                            KeyScale ks, double* sums, hipStream_t st) {
  const int n = blocks_of(S);
  if (sums)
    hipLaunchKernelGGL(quant_fp8_kernel<true>, dim3(H, n, B), dim3(256), 0, st, x, codes, S, H, n,
                       in_dt == CHORUS_BF16, scales, ks, sums);
  else
    hipLaunchKernelGGL(quant_fp8_kernel<false>, dim3(H, n, B), dim3(256), 0, st, x, codes, S, H, n,
                       in_dt == CHORUS_BF16, scales, ks, sums);
  return hipGetLastError();
}

}  // namespace chorus
