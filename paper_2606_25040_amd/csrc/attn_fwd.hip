// Block-sparse attention forward, fp16 / bf16 (Chorus II Sec. 3.2 "Efficient
// block-sparse kernel": only the listed block pairs enter QK^T, softmax, PV).
//
// One workgroup = one work item (request b, head h, 64-query block i), two
// waves of 32 queries, 32 KB of LDS, so four workgroups (two waves per SIMD)
// share a CU and hide each other's latencies.  For each listed kv block j:
//   * the list is walked from a rotated start (walk_target), so the q-blocks
//     in flight on an XCD read about the same kv blocks at the same time;
//   * K_j and V_j go global -> LDS with global_load_lds_dwordx4 (no register
//     staging); each tile has its own single buffer, refilled as soon as the
//     phase that reads it is over (K after QK^T, V after PV), so the next
//     block's loads overlap this block's softmax and PV;
//   * S^T = K_j Q^T with v_mfma_f32_32x32x16 (A = K rows from LDS, B = Q
//     fragments kept in registers): each lane holds 32 scores of ONE query
//     (lanes l and l ^ 32 split its 64 keys), so the row max and row sum are
//     lane-local plus one half-wave exchange;
//   * online softmax in the log2 domain; the running max is only moved (and
//     O, l rescaled) when some row's max grew by more than kRescaleLog2, so
//     P <= 2^kRescaleLog2 and most blocks skip the 64-register rescale;
//   * O^T += V_j^T P^T with the same MFMA; V^T fragments come from the
//     row-major tile through ds_read_b64_tr_b16; P is the score accumulator
//     converted to 16-bit in registers.
// LDS tiles are XOR-swizzled in 16-byte chunks (the direct loads permute the
// global addresses instead of the LDS ones) so that the b128 K reads and the
// transposed b64 V reads are bank-conflict free.
// Epilogue: O = O^T / l written as 16-bit, lse = ln(sum exp) in fp32.
// Template flags: DENSE walks every kv block (no mask); KSCALE multiplies the
// logits of keys below n_first by beta (first-frame key enhancement, Eq. 1);
// KV2 reads a mask of 128-token kv blocks and walks each as its two 64-token
// halves.  Each flag is its own instantiation, so the plain path carries none
// of the others' work.
#include "attn_common.h"

namespace chorus {
namespace {

constexpr float kRescaleLog2 = 8.f;
constexpr int kTileBytes = kBlock * kHeadDim * 2;   // 16 KB per 16-bit tile

// 16-byte chunk position of chunk c in row r.
__device__ inline int k_swz(int r, int c) { return c ^ (r & 15); }
__device__ inline int v_swz_bits(int r) { return (0xE4A0 >> (4 * (r & 3))) & 15; }   // {0, 10, 4, 14}
__device__ inline int v_swz(int r, int c) { return c ^ v_swz_bits(r); }

template <bool BF16>
struct Elt;
// The transposed LDS reads go through the typed builtin (or a whole-vector
// bitcast) and are joined with __builtin_shufflevector: assembling the
// operand element by element from the i16 variant was miscompiled.
template <>
struct Elt<true> {
  using vec8 = bf16x8;
  using scalar = __bf16;
  static __device__ inline f32x16 mfma(vec8 a, vec8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ inline vec8 tr_pair(const char* lo, const char* hi) {
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
  static __device__ inline vec8 tr_pair(const char* lo, const char* hi) {
    const f16x4 a = __builtin_bit_cast(f16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)lo));
    const f16x4 b = __builtin_bit_cast(f16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)hi));
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
  }
};

// This wave's share of one 64 x 128 16-bit tile: instruction u fills LDS rows
// 8u + 4 wave .. + 3 (1 KB, lane-linear), each lane fetching the global chunk
// that the swizzle places at its slot.  Full blocks take the row offset from
// the scalar base and a per-lane offset fixed for the whole kernel; the
// partial last block clamps rows past the sequence end to row S - 1 (their
// keys are masked and their probabilities are zero).
struct TileLoader {
  const char* base;    // token 0 of this (b, h)
  uint32_t ss;         // token stride in bytes
  uint32_t off[2];     // lane offset for even / odd u (row r0, swizzled chunk)
  int r0, p;
  template <bool IS_K>
  __device__ void init(const uint16_t* b, int64_t stride, int wave, int lane) {
    base = reinterpret_cast<const char*>(b);
    ss = (uint32_t)(stride * 2);
    r0 = 4 * wave + (lane >> 4);
    p = lane & 15;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int c = IS_K ? k_swz(r0 + 8 * e, p) : v_swz(r0 + 8 * e, p);
      off[e] = (uint32_t)r0 * ss + (uint32_t)c * 16;
    }
  }
  template <bool IS_K>
  __device__ void load(char* tile, int j, int S, int wave) const {
    const uint32_t lds = (uint32_t)(size_t)(__attribute__((address_space(3))) char*)tile + wave * 1024;
    if (j * kBlock + kBlock <= S) {
      const char* rowj = base + (int64_t)j * kBlock * ss;
#pragma unroll
      for (int u = 0; u < 8; ++u) dma16(lds + u * 2048, rowj + (int64_t)(8 * u) * ss, off[u & 1]);
    } else {
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int r = 8 * u + r0;
        const int c = IS_K ? k_swz(r, p) : v_swz(r, p);
        const int tok = min(j * kBlock + r, S - 1);
        dma16(lds + u * 2048, base, (uint32_t)tok * ss + (uint32_t)c * 16);
      }
    }
  }
};

template <bool BF16, bool DENSE, bool KSCALE, bool KV2>
__global__ __launch_bounds__(128) __attribute__((amdgpu_waves_per_eu(2)))
void attn_fwd_16_kernel(AttnArgs a) {
  using E = Elt<BF16>;
  using vec8 = typename E::vec8;
  using scalar = typename E::scalar;
  __shared__ __attribute__((aligned(1024))) char k_s[kTileBytes];
  __shared__ __attribute__((aligned(1024))) char v_s[kTileBytes];

  const int item = work_item(a.order, a.B * a.H, a.n);
  if (item < 0) return;
  const int n = a.n, H = a.H, S = a.S;
  const int i = item % n;
  const int bh = item / n;
  const int h = bh % H, b = bh / H;
  // DENSE: every kv block (no mask); otherwise the CSR row of (b, h, i).
  // KV2: the row lists kv blocks of 128 tokens; the walk visits both 64-token
  // halves of each (positions 2 p and 2 p + 1 of the doubled list).
  int kb0 = 0, kb1 = n;
  if (!DENSE) {
    const int64_t mrow = ((int64_t)(a.mask_batch > 1 ? b : 0) * H + h) * n + i;
    kb0 = a.row_ptr[mrow];
    kb1 = a.row_ptr[mrow + 1];
    if (KV2) {
      kb0 *= 2;
      kb1 *= 2;
    }
  }
  ConstI32* cidx = as_constant(a.col_idx);   // scalar loads
  auto kv_at = [&](int p) { return DENSE ? p : KV2 ? 2 * cidx[p >> 1] + (p & 1) : cidx[p]; };
  // walk step v visits list position kb0 + (v + rot) mod L (see walk_target);
  // without a mask every q-block lists every block and starts at block 0
  const int L = kb1 - kb0;
  const int rot = DENSE ? 0 : walk_rotation(kb0, kb1, walk_target(i, n), kv_at);
  auto kv_block = [&](int v) {
    const int p = v + rot;
    return kv_at(kb0 + (p >= L ? p - L : p));
  };
  // ids outside [0, n) are skipped (the builder never emits them; with KV2
  // this also drops the missing half of a last block of 64 tokens)
  auto next_valid = [&](int jj) {
    while (jj < L) {
      const int j = kv_block(jj);
      if (j >= 0 && j < n) break;
      ++jj;
    }
    return jj;
  };

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
  const int lane = tid & 63;
  const int l32 = lane & 31, hl = lane >> 5;
  const int g = lane >> 4, j16 = lane & 15;

  const uint16_t* kbase = static_cast<const uint16_t*>(a.k.data) + (int64_t)b * a.k.sb + (int64_t)h * a.k.sh;
  const uint16_t* vbase = static_cast<const uint16_t*>(a.v.data) + (int64_t)b * a.v.sb + (int64_t)h * a.v.sh;

  TileLoader kl, vl;
  kl.init<true>(kbase, a.k.ss, wave, lane);
  vl.init<false>(vbase, a.v.ss, wave, lane);
  int jj = next_valid(0);
  if (jj < L) {
    const int j0 = kv_block(jj);
    kl.load<true>(k_s, j0, S, wave);
    vl.load<false>(v_s, j0, S, wave);
  }

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
  // Drain the Q loads (and the first tiles) with an s_waitcnt the compiler
  // sees, so that it does not re-wait for Q inside the loop.
  __builtin_amdgcn_s_waitcnt(0xF70);   // vmcnt(0)

  // per-lane LDS byte offsets of the K (A operand) and V^T (transposed) reads
  const int k_row_off = l32 * 256;
  const int k_swzl = l32 & 15;
  const int v_lane_off = (j16 >> 2) * 256 + 8 * (j16 & 1);
  const int v_c0 = 2 * (g & 1) + ((j16 & 3) >> 1);
  const int v_sl = v_swz_bits(j16 >> 2);

  const float cl2 = a.sm_scale * kLog2e;
  float m_run = -INFINITY, l_run = 0.f;
  f32x16 o[4];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[u][r] = 0.f;

  while (jj < L) {
    const int j = kv_block(jj);
    const int jn = next_valid(jj + 1);
    const bool has_next = jn < L;
    const int j_next = has_next ? kv_block(jn) : 0;

    // K_j resident: at most this block's V loads (8) are still in flight
    CHORUS_WAIT_VMCNT(8);
    __syncthreads();
    f32x16 sacc[2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[t][r] = 0.f;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int koff = k_row_off + (((2 * s + hl) ^ k_swzl) << 4);
#pragma unroll
      for (int t = 0; t < 2; ++t) {       // two independent accumulation chains
        const vec8 kf = *reinterpret_cast<const vec8*>(k_s + t * 32 * 256 + koff);
        sacc[t] = E::mfma(kf, qf[s], sacc[t]);
      }
    }
    __syncthreads();                               // every wave is done with K_j
    if (has_next) kl.load<true>(k_s, j_next, S, wave);

    // first-frame keys (Eq. 1): their logits count beta times
    if (KSCALE && j * kBlock < a.ks.n_first) {
      const int lim = a.ks.n_first - j * kBlock;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = 32 * t + 8 * (r >> 2) + 4 * hl + (r & 3);
          if (key < lim) sacc[t][r] *= a.ks.beta;
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
    if (__builtin_amdgcn_ballot_w64(m_new > m_run + kRescaleLog2) != 0) {
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[u][r] *= alpha;
    }
    float rs = 0.f;
    vec8 pf[2][2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(sacc[t][r] * cl2 - m_run);
        rs += p;
        pf[t][r >> 3][r & 7] = (scalar)p;
      }
    l_run += rs;

    // V_j resident: only the next K tile's loads (8, if issued) may be in flight
    if (has_next) {
      CHORUS_WAIT_VMCNT(8);
    } else {
      CHORUS_WAIT_VMCNT(0);
    }
    __syncthreads();
    // O^T[u] += V^T[u] P^T: k-slot i of lane half hl maps to key
    // 32 t + 16 hh + 8 (i / 4) + 4 hl + i % 4 in both operands.
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int k0 = 32 * t + 16 * hh + 4 * (g >> 1);
#pragma unroll
        for (int u = 0; u < 4; ++u) {     // four independent accumulators
          const int cu = (4 * u + v_c0) ^ v_sl;
          const char* lo = v_s + k0 * 256 + v_lane_off + (cu << 4);
          const vec8 vf = E::tr_pair(lo, lo + 8 * 256);
          o[u] = E::mfma(vf, pf[t][hh], o[u]);
        }
      }
    __syncthreads();                               // every wave is done with V_j
    if (has_next) vl.load<false>(v_s, j_next, S, wave);
    jj = jn;
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

namespace {
template <bool BF16, bool DENSE, bool KV2>
void launch_16(const AttnArgs& a, dim3 grid, hipStream_t st) {
  if (a.ks.n_first > 0)
    hipLaunchKernelGGL((attn_fwd_16_kernel<BF16, DENSE, true, KV2>), grid, dim3(128), 0, st, a);
  else
    hipLaunchKernelGGL((attn_fwd_16_kernel<BF16, DENSE, false, KV2>), grid, dim3(128), 0, st, a);
}

template <bool BF16>
void launch_16_mask(const AttnArgs& a, dim3 grid, hipStream_t st) {
  if (a.row_ptr == nullptr)
    launch_16<BF16, true, false>(a, grid, st);
  else if (a.kv_block == 2 * kBlock)
    launch_16<BF16, false, true>(a, grid, st);
  else
    launch_16<BF16, false, false>(a, grid, st);
}
}  // namespace

hipError_t launch_attn_fwd_16(chorus_dtype dt, const AttnArgs& a, hipStream_t st) {
  const dim3 grid(work_grid(a.B * a.H, a.n));
  if (dt == CHORUS_BF16)
    launch_16_mask<true>(a, grid, st);
  else
    launch_16_mask<false>(a, grid, st);
  return hipGetLastError();
}

}  // namespace chorus
