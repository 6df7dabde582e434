// Block-sparse attention forward, FP8 e4m3 inputs, bf16 output (Chorus II
// Sec. 3.2 "Efficient block-sparse kernel": FP8 products, fp32 accumulation).
//
// Same work decomposition as the 16-bit kernel: a workgroup takes a pair of
// neighbouring q-blocks of one (request, head), four waves of 32 queries,
// walks the union of the two kv lists (from the rotated start of the pair,
// see walk_target), and double-buffers the 8 KB K and V
// code tiles in LDS (direct global -> LDS loads, one barrier per kv block).
// Both products use v_mfma_scale_f32_32x32x64_f8f6f4 with unit scales:
//   * S^T = K_j Q^T on codes; the true logit is acc * s_q,i * s_k,j * sm_scale,
//     folded into one per-block multiplier (log2 domain);
//   * LDS row m of the K tile holds key sigma(m) (m = 8a + 4h + c holds
//     16h + 4a + c inside each 32-key half), so after QK^T lane half hl of tile
//     t holds the 16 consecutive keys 32t + 16hl .. + 15 and the V^T fragments
//     are plain 8-consecutive-key transposed reads (ds_read_b64_tr_b8) of the
//     row-major V tile;
//   * the per-kv-block V scale is folded into the exponent: with
//     f_j = s_v,j / s_ref (s_ref = largest V scale among the pair's blocks),
//     P~ = 2^(x - m + log2 f_j + kPShift) = 2^kPShift f_j p is rounded to e4m3
//     and O^T += V_codes^T P~^T; the row sum adds (sum P~) 2^-(log2 f_j +
//     kPShift) and the epilogue multiplies by s_ref 2^-kPShift;
//   * the running max moves only when a row max grew by more than
//     kRescaleLog2, which keeps P~ <= 2^(kPShift + kRescaleLog2) < 448.
// P~ never leaves registers.
// Template flags as in the 16-bit kernel: DENSE (no mask), KSCALE (Eq. 1
// first-frame key enhancement on the dequantised keys), KV2 (kv blocks of 128
// tokens walked as their 64-token halves).
#include "attn_common.h"

namespace chorus {
namespace {

constexpr int kTile8 = kBlock * kHeadDim;   // 8 KB per code tile
constexpr int kWaves = 4;
constexpr float kPShift = 7.f;
constexpr float kRescaleLog2 = 1.5f;

// MFMA A-row m of a 32-key half holds key sigma(m) = 16 h + 4 a + c for
// m = 8 a + 4 h + c; the loader therefore fetches key sigma(row) into row.
__device__ inline int k_key_of_row(int r) {
  const int t = r & ~31, m = r & 31;
  return t + 16 * ((m >> 2) & 1) + 4 * (m >> 3) + (m & 3);
}
// 16-byte chunk position of chunk c (0..7) in row r of the K / V code tiles.
__device__ inline int k8_swz(int r, int c) { return c ^ ((r >> 1) & 7); }
__device__ inline int v8_swz(int r, int c) { return c ^ (2 * ((r >> 1) & 3)); }

// This wave's share of one 64 x 128 code tile: instruction u (0, 1) fills LDS
// rows 8 (4u + wave) .. + 7 (1 KB, lane-linear: lane -> row + lane / 8,
// chunk lane % 8); K rows fetch the permuted key.  Full blocks take the row
// offset from the scalar base and a per-lane offset fixed for the whole
// kernel; rows of a partial last block past the sequence end re-read token
// S - 1 (masked keys, zero probabilities).
template <bool IS_K>
struct Tile8Loader {
  const char* base;
  uint32_t ss;
  uint32_t off[2];
  __device__ void init(const char* b, uint32_t s, int wave, int lane) {
    base = b;
    ss = s;
#pragma unroll
    for (int u = 0; u < 2; ++u) off[u] = (uint32_t)key(u, wave, lane) * ss + (uint32_t)chunk(u, wave, lane) * 16;
  }
  static __device__ int row(int u, int wave, int lane) { return 8 * (4 * u + wave) + (lane >> 3); }
  static __device__ int chunk(int u, int wave, int lane) {
    const int r = row(u, wave, lane), p = lane & 7;
    return IS_K ? k8_swz(r, p) : v8_swz(r, p);
  }
  static __device__ int key(int u, int wave, int lane) {
    const int r = row(u, wave, lane);
    return IS_K ? k_key_of_row(r) : r;
  }
  __device__ void load(uint32_t lds, int j, int S, int wave, int lane) const {
    if (j * kBlock + kBlock <= S) {
      const char* rowj = base + (int64_t)j * kBlock * ss;
#pragma unroll
      for (int u = 0; u < 2; ++u) dma16(lds + (4 * u + wave) * 1024, rowj, off[u]);
    } else {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int tok = min(j * kBlock + key(u, wave, lane), S - 1);
        dma16(lds + (4 * u + wave) * 1024, base, (uint32_t)tok * ss + (uint32_t)chunk(u, wave, lane) * 16);
      }
    }
  }
};

// At most 168 registers, so that every instantiation runs three waves per
// SIMD (three workgroups per CU): left free, the compiler gives the KSCALE
// ones about 200 registers and two waves per SIMD, 11 % slower.
template <bool DENSE, bool KSCALE, bool KV2>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3)))
void attn_fwd_fp8_kernel(AttnArgs a, int np) {
  __shared__ __attribute__((aligned(1024))) uint8_t tiles[2][2][kTile8];   // [buffer][K, V]
  __shared__ float red[kWaves];

  const int item = work_item(a.order, a.B * a.H, np);
  if (item < 0) return;
  const int n = a.n, H = a.H, S = a.S;
  const int ip = item % np;
  const int bh = item / np;
  const int h = bh % H, b = bh / H;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int l32 = lane & 31, hl = lane >> 5;
  const int g = lane >> 4, j16 = lane & 15;
  const int sel = wave >> 1;
  const int i = 2 * ip + sel;
  const bool q_active = i < n;
  ConstF32* qsc = as_constant(a.q_scale) + (int64_t)bh * n;   // scalar loads
  ConstF32* ksc = as_constant(a.k_scale) + (int64_t)bh * n;
  ConstF32* vsc = as_constant(a.v_scale) + (int64_t)bh * n;

  PairWalk<KV2> walk;
  walk.init(a, DENSE, b, h, ip);
  const bool listed_any = q_active && walk.listed(sel);

  // reference V scale: the largest among the pair's listed blocks
  float sref = 0.f;
  {
    const int la = walk.la;
    for (int t = tid; t < la + walk.lb; t += 64 * kWaves) {
      const int j = t < la ? walk.id_at(walk.a0 + t) : walk.id_at(walk.b0 + t - la);
      if (j >= 0 && j < n) sref = fmaxf(sref, vsc[j]);
    }
    for (int o = 32; o > 0; o >>= 1) sref = fmaxf(sref, __shfl_xor(sref, o));
    if (lane == 0) red[wave] = sref;
    __syncthreads();
    sref = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  }
  constexpr float kMinNormal = 1.17549435e-38f;
  const float log2_sref = __builtin_log2f(sref > 0.f ? fmaxf(sref, kMinNormal) : 1.f);

  const char* kbase = static_cast<const char*>(a.k.data) + (int64_t)b * a.k.sb + (int64_t)h * a.k.sh;
  const char* vbase = static_cast<const char*>(a.v.data) + (int64_t)b * a.v.sb + (int64_t)h * a.v.sh;
  Tile8Loader<true> kl;
  Tile8Loader<false> vl;
  kl.init(kbase, (uint32_t)a.k.ss, wave, lane);
  vl.init(vbase, (uint32_t)a.v.ss, wave, lane);
  const uint32_t lds0 = (uint32_t)(size_t)(__attribute__((address_space(3))) uint8_t*)&tiles[0][0][0];

  bool in_a, in_b;
  int j = walk.next(in_a, in_b);
  if (j != INT32_MAX) {
    kl.load(lds0, j, S, wave, lane);
    vl.load(lds0 + kTile8, j, S, wave, lane);
  }

  // Q^T fragments (codes): query qrow, head-dim bytes 64 s + 32 hl .. + 32
  const int qrow = i * kBlock + (wave & 1) * 32 + l32;
  i32x8 qf[2];
  {
    const uint8_t* qp = static_cast<const uint8_t*>(a.q.data) + (int64_t)b * a.q.sb + (int64_t)qrow * a.q.ss +
                        (int64_t)h * a.q.sh + 32 * hl;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      if (q_active && qrow < S) {
        const uint4 x0 = *reinterpret_cast<const uint4*>(qp + 64 * s);
        const uint4 x1 = *reinterpret_cast<const uint4*>(qp + 64 * s + 16);
        qf[s] = (i32x8){(int)x0.x, (int)x0.y, (int)x0.z, (int)x0.w, (int)x1.x, (int)x1.y, (int)x1.z, (int)x1.w};
      } else {
        qf[s] = (i32x8){0, 0, 0, 0, 0, 0, 0, 0};
      }
    }
  }
  const float cq = q_active ? qsc[i] * a.sm_scale * kLog2e : 0.f;
  __builtin_amdgcn_s_waitcnt(0xF70);   // vmcnt(0): Q and the first tiles

  // per-lane LDS byte offsets: K A-operand rows and V^T transposed reads
  const int k_row_off = l32 * 128;
  const int k_sw = (l32 >> 1) & 7;
  const int v_lane_off = (j16 >> 1) * 128 + 8 * (j16 & 1);
  const int v_sw = 2 * ((j16 >> 2) & 3);

  float m_run = -INFINITY, l_run = 0.f;
  f32x16 o[4];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[u][r] = 0.f;

  int buf = 0;
  while (j != INT32_MAX) {
    const bool mine = sel == 0 ? in_a : in_b;
    bool na, nb;
    const int jn = walk.next(na, nb);
    CHORUS_WAIT_VMCNT(0);
    __syncthreads();
    if (jn != INT32_MAX) {
      const uint32_t nxt = lds0 + (buf ^ 1) * 2 * kTile8;
      kl.load(nxt, jn, S, wave, lane);
      vl.load(nxt + kTile8, jn, S, wave, lane);
    }
    if (mine && q_active) {
      const uint8_t* k_s = &tiles[buf][0][0];
      const uint8_t* v_s = &tiles[buf][1][0];
      f32x16 sacc[2];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[t][r] = 0.f;
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const int c0 = 4 * s + 2 * hl;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const uint8_t* kr = k_s + t * 32 * 128 + k_row_off;
          const uint4 x0 = *reinterpret_cast<const uint4*>(kr + ((c0 ^ k_sw) << 4));
          const uint4 x1 = *reinterpret_cast<const uint4*>(kr + (((c0 + 1) ^ k_sw) << 4));
          const i32x8 kf = {(int)x0.x, (int)x0.y, (int)x0.z, (int)x0.w, (int)x1.x, (int)x1.y, (int)x1.z,
                            (int)x1.w};
          sacc[t] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(kf, qf[s], sacc[t], 0, 0, 0, 127, 0, 127);
        }
      }
      // first-frame keys (Eq. 1, on the dequantised keys): logits count beta times
      if (KSCALE && j * kBlock < a.ks.n_first) {
        const int lim = a.ks.n_first - j * kBlock;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (32 * t + 16 * hl + r < lim) sacc[t][r] *= a.ks.beta;
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
      if (__builtin_amdgcn_ballot_w64(m_new > m_run + kRescaleLog2) != 0) {
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[u][r] *= alpha;
      }
      // log2(2^kPShift f_j); both scales are clamped to the smallest normal
      // float (the raw v_log_f32 takes no denormals), so f_j <= 1 still holds
      const float bias = __builtin_amdgcn_logf(fmaxf(vsc[j], kMinNormal)) - log2_sref + kPShift;
      const float mb = m_run - bias;
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
        const int word = __builtin_amdgcn_cvt_pk_fp8_f32(p[0], p[1], 0, false);
        pw[w] = __builtin_amdgcn_cvt_pk_fp8_f32(p[2], p[3], word, true);
      }
      l_run += rs * __builtin_amdgcn_exp2f(-bias);
      // O^T[u] += V^T[u] P~^T: byte e of lane half hl is key 32 (e / 16) + 16 hl + e % 16
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = 2 * u + (g & 1);
        const uint8_t* vc = v_s + v_lane_off + ((c ^ v_sw) << 4);
        i32x2 x[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int k0 = 32 * (q >> 1) + 16 * (g >> 1) + 8 * (q & 1);
          x[q] = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i32x2*)(vc + k0 * 128));
        }
        const i32x4 x01 = __builtin_shufflevector(x[0], x[1], 0, 1, 2, 3);
        const i32x4 x23 = __builtin_shufflevector(x[2], x[3], 0, 1, 2, 3);
        const i32x8 vf = __builtin_shufflevector(x01, x23, 0, 1, 2, 3, 4, 5, 6, 7);
        o[u] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(vf, pw, o[u], 0, 0, 0, 127, 0, 127);
      }
    }
    j = jn;
    in_a = na;
    in_b = nb;
    buf ^= 1;
  }

  const float l_tot = pair_sum(l_run);
  const bool live = listed_any && l_tot > 0.f;
  const float post = live ? sref * __builtin_amdgcn_exp2f(-kPShift) / l_tot : 0.f;
  if (q_active && qrow < S) {
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
  const int np = (a.n + 1) / 2;
  const dim3 grid(work_grid(a.B * a.H, np)), block(64 * kWaves);
  const bool ks = a.ks.n_first > 0;
  if (a.row_ptr == nullptr) {
    if (ks)
      hipLaunchKernelGGL((attn_fwd_fp8_kernel<true, true, false>), grid, block, 0, st, a, np);
    else
      hipLaunchKernelGGL((attn_fwd_fp8_kernel<true, false, false>), grid, block, 0, st, a, np);
  } else if (a.kv_block == 2 * kBlock) {
    if (ks)
      hipLaunchKernelGGL((attn_fwd_fp8_kernel<false, true, true>), grid, block, 0, st, a, np);
    else
      hipLaunchKernelGGL((attn_fwd_fp8_kernel<false, false, true>), grid, block, 0, st, a, np);
  } else {
    if (ks)
      hipLaunchKernelGGL((attn_fwd_fp8_kernel<false, true, false>), grid, block, 0, st, a, np);
    else
      hipLaunchKernelGGL((attn_fwd_fp8_kernel<false, false, false>), grid, block, 0, st, a, np);
  }
  return hipGetLastError();
}

}  // namespace chorus
