// Block-sparse attention forward, FP8 e4m3 inputs, bf16 output (Chorus II
// Sec. 3.2 "Efficient block-sparse kernel": FP8 products, fp32 accumulation).
//
// Same work decomposition as the 16-bit kernel (one workgroup per
// (request, head, 64-query block), two waves of 32 queries), with
// v_mfma_scale_f32_32x32x64_f8f6f4 (unit scales) for both products:
//   * S^T = K_j Q^T on codes; the true logit is acc * s_q,i * s_k,j * sm_scale,
//     folded into one per-block multiplier (log2 domain);
//   * K rows are written to LDS in a permuted order so that after QK^T lane
//     half hl of tile t holds the 16 consecutive keys 32 t + 16 hl .. + 15;
//     V^T fragments are then plain 8-consecutive-key transposed reads
//     (ds_read_b64_tr_b8) of the row-major V tile;
//   * the per-kv-block V scale is folded into the exponent: with
//     f_j = s_v,j / s_ref (s_ref = largest V scale among the row's blocks),
//     P~ = 2^(x - m + log2 f_j + 8) = 256 f_j p <= 256 is rounded to e4m3 and
//     O^T += V_codes^T P~^T; the row sum adds (sum P~) / (256 f_j) and the
//     epilogue multiplies by s_ref / 256.  P~ never leaves registers.
#include "attn_common.h"

namespace chorus {
namespace {

constexpr int kS8 = 144;   // LDS row stride in bytes for the K and V code tiles
constexpr float kPShift = 8.f;

// K row held by MFMA A-row m (m = 8 a + 4 h + c) is key 16 h + 4 a + c, i.e. LDS row
// m stores key sigma(m); the inverse places key kappa at row sigma^-1(kappa).
__device__ inline int k_row_of_key(int kappa) {
  const int t = kappa & ~31, k = kappa & 31;
  return t + 8 * ((k >> 2) & 3) + 4 * (k >> 4) + (k & 3);
}

template <bool DENSE>
__global__ __launch_bounds__(128) void attn_fwd_fp8_kernel(AttnArgs a, int chunk, int W) {
  __shared__ __attribute__((aligned(16))) uint8_t k_s[kBlock * kS8];
  __shared__ __attribute__((aligned(16))) uint8_t v_s[kBlock * kS8];
  __shared__ float red[2];

  const int item = work_item(a.order, chunk, W);
  if (item < 0) return;
  const int n = a.n, H = a.H, S = a.S;
  const int i = item % n;
  const int bh = item / n;
  const int h = bh % H, b = bh / H;
  int kb0 = 0, kb1 = n;
  if (!DENSE) {
    const int64_t mrow = ((int64_t)(a.mask_batch > 1 ? b : 0) * H + h) * n + i;
    kb0 = a.row_ptr[mrow];
    kb1 = a.row_ptr[mrow + 1];
  }
  auto kv_block = [&](int jj) { return DENSE ? jj : a.col_idx[jj]; };
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int l32 = lane & 31, hl = lane >> 5;
  const float* qsc = a.q_scale + (int64_t)bh * n;
  const float* ksc = a.k_scale + (int64_t)bh * n;
  const float* vsc = a.v_scale + (int64_t)bh * n;

  // reference V scale: the largest among the listed blocks
  float sref = 0.f;
  for (int jj = kb0 + tid; jj < kb1; jj += 128) {
    const int j = kv_block(jj);
    if (j >= 0 && j < n) sref = fmaxf(sref, vsc[j]);
  }
  for (int o = 32; o > 0; o >>= 1) sref = fmaxf(sref, __shfl_xor(sref, o));
  if (lane == 0) red[wave] = sref;
  __syncthreads();
  sref = fmaxf(red[0], red[1]);
  const float log2_sref = __builtin_log2f(sref > 0.f ? sref : 1.f);

  // Q^T fragments (codes): query qrow, head-dim bytes 64 s + 32 hl .. + 32
  const int qrow = i * kBlock + wave * 32 + l32;
  i32x8 qf[2];
  {
    const uint8_t* qp = static_cast<const uint8_t*>(a.q.data) + (int64_t)b * a.q.sb + (int64_t)qrow * a.q.ss +
                        (int64_t)h * a.q.sh + 32 * hl;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      if (qrow < S) {
        const uint4 x0 = *reinterpret_cast<const uint4*>(qp + 64 * s);
        const uint4 x1 = *reinterpret_cast<const uint4*>(qp + 64 * s + 16);
        qf[s] = (i32x8){(int)x0.x, (int)x0.y, (int)x0.z, (int)x0.w, (int)x1.x, (int)x1.y, (int)x1.z, (int)x1.w};
      } else {
        qf[s] = (i32x8){0, 0, 0, 0, 0, 0, 0, 0};
      }
    }
  }
  const float cq = qsc[i] * a.sm_scale * kLog2e;

  const uint8_t* kbase = static_cast<const uint8_t*>(a.k.data) + (int64_t)b * a.k.sb + (int64_t)h * a.k.sh;
  const uint8_t* vbase = static_cast<const uint8_t*>(a.v.data) + (int64_t)b * a.v.sb + (int64_t)h * a.v.sh;
  const int srow = tid >> 3;          // staging rows srow + 16 u (u = 0..3), 16-byte chunk scol
  const int scol = (tid & 7) * 16;
  uint4 kreg[4], vreg[4];
  auto load_kv = [&](int j) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int tok = j * kBlock + srow + 16 * u;
      if (tok < S) {
        kreg[u] = *reinterpret_cast<const uint4*>(kbase + (int64_t)tok * a.k.ss + scol);
        vreg[u] = *reinterpret_cast<const uint4*>(vbase + (int64_t)tok * a.v.ss + scol);
      } else {
        kreg[u] = make_uint4(0, 0, 0, 0);
        vreg[u] = make_uint4(0, 0, 0, 0);
      }
    }
  };

  float m_run = -INFINITY, l_run = 0.f;
  f32x16 o[4];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[u][r] = 0.f;

  int jn = kb0 < kb1 ? kv_block(kb0) : 0;
  if (kb0 < kb1 && jn >= 0 && jn < n) load_kv(jn);
  for (int jj = kb0; jj < kb1; ++jj) {
    const int j = jn;
    if (jj + 1 < kb1) jn = kv_block(jj + 1);
    if (j < 0 || j >= n) {
      if (jj + 1 < kb1 && jn >= 0 && jn < n) load_kv(jn);
      continue;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int key = srow + 16 * u;
      *reinterpret_cast<uint4*>(k_s + k_row_of_key(key) * kS8 + scol) = kreg[u];
      *reinterpret_cast<uint4*>(v_s + key * kS8 + scol) = vreg[u];
    }
    __syncthreads();
    if (jj + 1 < kb1 && jn >= 0 && jn < n) load_kv(jn);

    // S^T tiles: lane (l32, hl) of tile t ends up with keys 32 t + 16 hl + r, r = 0..15
    f32x16 sacc[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[t][r] = 0.f;
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const uint8_t* kp = k_s + (32 * t + l32) * kS8 + 64 * s + 32 * hl;
        const uint4 x0 = *reinterpret_cast<const uint4*>(kp);
        const uint4 x1 = *reinterpret_cast<const uint4*>(kp + 16);
        const i32x8 kf = {(int)x0.x, (int)x0.y, (int)x0.z, (int)x0.w, (int)x1.x, (int)x1.y, (int)x1.z, (int)x1.w};
        sacc[t] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(kf, qf[s], sacc[t], 0, 0, 0, 127, 0, 127);
      }
    }
    if (j * kBlock + kBlock > S) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (j * kBlock + 32 * t + 16 * hl + r >= S) sacc[t][r] = -INFINITY;
    }
    const float cj = cq * ksc[j];
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[t][r]);
    mx = pair_max(mx);
    const float m_new = fmaxf(m_run, mx * cj);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    const float bias = __builtin_log2f(vsc[j]) - log2_sref + kPShift;   // log2(256 f_j)
    const float mb = m_new - bias;
    float rs = 0.f;
    i32x8 pw;
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      const int t = w >> 2, r0 = (w & 3) * 4;
      float p[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        p[e] = __builtin_amdgcn_exp2f(sacc[t][r0 + e] * cj - mb);
        rs += p[e];
      }
      int word = __builtin_amdgcn_cvt_pk_fp8_f32(p[0], p[1], 0, false);
      pw[w] = __builtin_amdgcn_cvt_pk_fp8_f32(p[2], p[3], word, true);
    }
    l_run = l_run * alpha + rs * __builtin_amdgcn_exp2f(-bias);
    m_run = m_new;
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[u][r] *= alpha;

    // O^T[u] += V^T[u] P~^T: byte e of lane half hl is key 32 (e / 16) + 16 hl + e % 16
    const int g = lane >> 4, j16 = lane & 15;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int col = 32 * u + 16 * (g & 1) + 8 * (j16 & 1);
      i32x2 x[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int k0 = 32 * (q >> 1) + 16 * (g >> 1) + 8 * (q & 1) + (j16 >> 1);
        x[q] = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i32x2*)(v_s + k0 * kS8 + col));
      }
      const i32x4 x01 = __builtin_shufflevector(x[0], x[1], 0, 1, 2, 3);
      const i32x4 x23 = __builtin_shufflevector(x[2], x[3], 0, 1, 2, 3);
      const i32x8 vf = __builtin_shufflevector(x01, x23, 0, 1, 2, 3, 4, 5, 6, 7);
      o[u] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(vf, pw, o[u], 0, 0, 0, 127, 0, 127);
    }
    __syncthreads();
  }

  const float l_tot = pair_sum(l_run);
  const bool live = kb1 > kb0 && l_tot > 0.f;
  const float post = live ? sref * __builtin_amdgcn_exp2f(-kPShift) / l_tot : 0.f;
  if (qrow < S) {
    uint16_t* op = static_cast<uint16_t*>(const_cast<void*>(a.o.data)) + (int64_t)b * a.o.sb +
                   (int64_t)qrow * a.o.ss + (int64_t)h * a.o.sh;
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        __bf16 v4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v4[e] = (__bf16)(o[u][4 * rr + e] * post);
        uint2 packed;
        __builtin_memcpy(&packed, v4, 8);
        *reinterpret_cast<uint2*>(op + 32 * u + 8 * rr + 4 * hl) = packed;
      }
    if (a.lse && hl == 0)
      a.lse[((int64_t)b * H + h) * S + qrow] = live ? (m_run + __builtin_log2f(l_tot)) * kLn2 : -INFINITY;
  }
}

}  // namespace

hipError_t launch_attn_fwd_fp8(const AttnArgs& a, hipStream_t st) {
  const int W = a.B * a.H * a.n;
  const int chunk = (W + kNumXcd - 1) / kNumXcd;
  if (a.row_ptr == nullptr)
    hipLaunchKernelGGL(attn_fwd_fp8_kernel<true>, dim3(chunk * kNumXcd), dim3(128), 0, st, a, chunk, W);
  else
    hipLaunchKernelGGL(attn_fwd_fp8_kernel<false>, dim3(chunk * kNumXcd), dim3(128), 0, st, a, chunk, W);
  return hipGetLastError();
}

}  // namespace chorus
