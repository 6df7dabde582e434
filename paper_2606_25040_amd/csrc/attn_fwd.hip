// Block-sparse attention forward, fp16 / bf16 (Chorus II Sec. 3.2 "Efficient
// block-sparse kernel": only the listed block pairs enter QK^T, softmax, PV).
//
// One workgroup = one work item (request b, head h, 64-query block i), two
// waves of 32 queries.  For each listed kv block j (64 keys):
//   * K_j and V_j are staged global -> registers -> LDS; the next block's
//     global loads are issued before the current block is computed;
//   * S^T = K_j Q^T with v_mfma_f32_32x32x16 (A = K rows from LDS, B = Q
//     fragments kept in registers), so each lane holds 32 scores of ONE query
//     (lane l and l ^ 32 split that query's 64 keys): row max and row sum are
//     lane-local plus one half-wave exchange;
//   * online softmax in the log2 domain (exp2, scale folded into one multiply);
//   * O^T += V_j^T P^T with the same MFMA; V^T fragments come straight from
//     the row-major LDS tile through ds_read_b64_tr_b16, and the P fragment is
//     the score accumulator itself converted to 16-bit, so P never leaves
//     registers.
// Epilogue: O = O^T / l written as 16-bit, lse = ln(sum exp) in fp32.
#include "attn_common.h"

namespace chorus {
namespace {

constexpr int kKS = 136;  // K tile row stride in 16-bit elements (272 B: conflict-free b128 reads)
constexpr int kVS = 144;  // V tile row stride (288 B: conflict-free transposed b64 reads)

template <bool BF16>
struct Elt;
// The transposed LDS reads are issued through the typed builtins and joined
// with __builtin_shufflevector: assembling the operand element by element
// from the i16 variant was miscompiled (lanes received repeated elements).
template <>
struct Elt<true> {
  using vec8 = bf16x8;
  using scalar = __bf16;
  static __device__ inline f32x16 mfma(vec8 a, vec8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ inline vec8 tr_pair(const uint16_t* lo, const uint16_t* hi) {
    const bf16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)lo);
    const bf16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)hi);
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
  }
};
template <>
struct Elt<false> {
  using vec8 = f16x8;
  using scalar = _Float16;
  static __device__ inline f32x16 mfma(vec8 a, vec8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
  static __device__ inline vec8 tr_pair(const uint16_t* lo, const uint16_t* hi) {
    const f16x4 a = __builtin_bit_cast(f16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)lo));
    const f16x4 b = __builtin_bit_cast(f16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)hi));
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
  }
};

template <bool BF16, bool DENSE>
__global__ __launch_bounds__(128) void attn_fwd_16_kernel(AttnArgs a, int chunk, int W) {
  using E = Elt<BF16>;
  using vec8 = typename E::vec8;
  using scalar = typename E::scalar;
  __shared__ __attribute__((aligned(16))) uint16_t k_s[kBlock * kKS];
  __shared__ __attribute__((aligned(16))) uint16_t v_s[kBlock * kVS];

  const int item = work_item(a.order, chunk, W);
  if (item < 0) return;
  const int n = a.n, H = a.H, S = a.S;
  const int i = item % n;
  const int bh = item / n;
  const int h = bh % H, b = bh / H;
  // DENSE: every kv block (no mask); otherwise the CSR row of (b, h, i)
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

  // Q^T fragments: query qrow, head-dim slice 16 s + 8 hl .. + 8
  const int qrow = i * kBlock + wave * 32 + l32;
  vec8 qf[8];
  {
    const uint16_t* qp = static_cast<const uint16_t*>(a.q.data) + (int64_t)b * a.q.sb + (int64_t)qrow * a.q.ss +
                         (int64_t)h * a.q.sh + 8 * hl;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      if (qrow < S) {
        qf[s] = *reinterpret_cast<const vec8*>(qp + 16 * s);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[s][e] = (scalar)0.f;
      }
    }
  }

  const uint16_t* kbase = static_cast<const uint16_t*>(a.k.data) + (int64_t)b * a.k.sb + (int64_t)h * a.k.sh;
  const uint16_t* vbase = static_cast<const uint16_t*>(a.v.data) + (int64_t)b * a.v.sb + (int64_t)h * a.v.sh;
  const int srow = tid >> 4;          // staging: rows srow + 8 u, 16-byte column chunk scol
  const int scol = (tid & 15) * 8;
  uint4 kreg[8], vreg[8];
  auto load_kv = [&](int j) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int tok = j * kBlock + srow + 8 * u;
      if (tok < S) {
        kreg[u] = *reinterpret_cast<const uint4*>(kbase + (int64_t)tok * a.k.ss + scol);
        vreg[u] = *reinterpret_cast<const uint4*>(vbase + (int64_t)tok * a.v.ss + scol);
      } else {
        kreg[u] = make_uint4(0, 0, 0, 0);
        vreg[u] = make_uint4(0, 0, 0, 0);
      }
    }
  };

  const float cl2 = a.sm_scale * kLog2e;
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
    if (j < 0 || j >= n) {           // ids outside [0, n) are skipped (the builder never emits them)
      if (jj + 1 < kb1 && jn >= 0 && jn < n) load_kv(jn);
      continue;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      *reinterpret_cast<uint4*>(k_s + (srow + 8 * u) * kKS + scol) = kreg[u];
      *reinterpret_cast<uint4*>(v_s + (srow + 8 * u) * kVS + scol) = vreg[u];
    }
    __syncthreads();
    if (jj + 1 < kb1 && jn >= 0 && jn < n) load_kv(jn);

    // S^T tiles t = 0, 1 (keys 32 t .. 32 t + 31) x 32 queries
    f32x16 sacc[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[t][r] = 0.f;
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const vec8 kf = *reinterpret_cast<const vec8*>(k_s + (32 * t + l32) * kKS + 16 * s + 8 * hl);
        sacc[t] = E::mfma(kf, qf[s], sacc[t]);
      }
    }
    // keys at or beyond S (partial last block) carry no weight
    if (j * kBlock + kBlock > S) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = 32 * t + 8 * (r >> 2) + 4 * hl + (r & 3);
          if (j * kBlock + key >= S) sacc[t][r] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[t][r]);
    mx = pair_max(mx);
    const float m_new = fmaxf(m_run, mx * cl2);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    float rs = 0.f;
    vec8 pf[2][2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(sacc[t][r] * cl2 - m_new);
        rs += p;
        pf[t][r >> 3][r & 7] = (scalar)p;
      }
    l_run = l_run * alpha + rs;
    m_run = m_new;
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[u][r] *= alpha;

    // O^T[u] += V^T[u] P^T: k-slot i of lane half hl maps to key
    // 32 t + 16 hh + 8 (i / 4) + 4 hl + i % 4 in both operands.
    const int g = lane >> 4, j16 = lane & 15;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int n0 = 32 * u + 16 * (g & 1) + 4 * (j16 & 3);
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const int k0 = 32 * t + 16 * hh + 4 * (g >> 1) + (j16 >> 2);
          const vec8 vf = E::tr_pair(v_s + k0 * kVS + n0, v_s + (k0 + 8) * kVS + n0);
          o[u] = E::mfma(vf, pf[t][hh], o[u]);
        }
    }
    __syncthreads();
  }

  // epilogue: lane pair (l, l ^ 32) holds partial sums of the same query
  const float l_tot = pair_sum(l_run);
  const bool live = kb1 > kb0 && l_tot > 0.f;
  const float inv_l = live ? 1.f / l_tot : 0.f;
  if (qrow < S) {
    uint16_t* op = static_cast<uint16_t*>(const_cast<void*>(a.o.data)) + (int64_t)b * a.o.sb +
                   (int64_t)qrow * a.o.ss + (int64_t)h * a.o.sh;
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        scalar v4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v4[e] = (scalar)(o[u][4 * rr + e] * inv_l);
        uint2 packed;
        __builtin_memcpy(&packed, v4, 8);
        *reinterpret_cast<uint2*>(op + 32 * u + 8 * rr + 4 * hl) = packed;
      }
    if (a.lse && hl == 0)
      a.lse[((int64_t)b * H + h) * S + qrow] = live ? (m_run + __builtin_log2f(l_tot)) * kLn2 : -INFINITY;
  }
}

}  // namespace

hipError_t launch_attn_fwd_16(chorus_dtype dt, const AttnArgs& a, hipStream_t st) {
  const int W = a.B * a.H * a.n;
  const int chunk = (W + kNumXcd - 1) / kNumXcd;
  const dim3 grid(chunk * kNumXcd), block(128);
  const bool dense = a.row_ptr == nullptr;
  if (dt == CHORUS_BF16) {
    if (dense)
      hipLaunchKernelGGL((attn_fwd_16_kernel<true, true>), grid, block, 0, st, a, chunk, W);
    else
      hipLaunchKernelGGL((attn_fwd_16_kernel<true, false>), grid, block, 0, st, a, chunk, W);
  } else {
    if (dense)
      hipLaunchKernelGGL((attn_fwd_16_kernel<false, true>), grid, block, 0, st, a, chunk, W);
    else
      hipLaunchKernelGGL((attn_fwd_16_kernel<false, false>), grid, block, 0, st, a, chunk, W);
  }
  return hipGetLastError();
}

}  // namespace chorus
