// Device helpers shared by the fp16/bf16 and fp8 block-sparse attention kernels.
#pragma once

#include "chorus_internal.h"

namespace chorus {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef bf16x4 __attribute__((address_space(3))) lds_bf16x4;
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef i16x4 __attribute__((address_space(3))) lds_i16x4;
typedef i32x2 __attribute__((address_space(3))) lds_i32x2;

// Read-only data seen through the constant address space: the compiler reads
// it with scalar loads (counted by lgkmcnt), which do not wait behind the tile
// loads still in flight (vmcnt).  Used for the kv lists and the fp8 block
// scales, which no kernel writes while attention runs.
typedef const __attribute__((address_space(4))) int32_t ConstI32;
typedef const __attribute__((address_space(4))) float ConstF32;
__device__ inline ConstI32* as_constant(const int32_t* p) { return (ConstI32*)p; }
__device__ inline ConstF32* as_constant(const float* p) { return (ConstF32*)p; }

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// max / sum of a value over the lane pair (l, l ^ 32): one v_permlane32_swap
// exchanges the two halves of the wave, so both outputs hold one value of
// each half at every lane.
__device__ inline float pair_max(float v) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float pair_sum(float v) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Work item of dispatch slot p.  Items are runs of neighbouring q-blocks,
// `np` per (request, head) unit, numbered unit * np + index, listed in the
// unit order (the planned order of (request, head) units, or the natural
// one).  Slots are dealt round-robin to the 8 XCDs, so slot p runs on XCD
// x = p % 8 as its (p / 8)-th slot there.  With U >= 8 units XCD x walks the
// items of units [s_x, s_x + c_x) of the order, c_x = U / 8 (+1 for the first
// U % 8 XCDs) and s_x the sum of the earlier c: exactly the groups the plan
// balances, listed XCD by XCD.  With fewer units than XCDs whole units would
// leave XCDs idle, so XCD x walks item positions [x * chunk, (x + 1) * chunk),
// chunk = ceil(U * np / 8), instead.  Returns -1 for idle slots.
__device__ inline int work_item(const int32_t* order, int U, int np) {
  const int p = blockIdx.x;
  const int x = p % kNumXcd, k = p / kNumXcd;
  int pos;
  if (U >= kNumXcd) {
    const int base = U / kNumXcd, extra = U % kNumXcd;
    const int cnt = (base + (x < extra ? 1 : 0)) * np;
    if (k >= cnt) return -1;
    pos = (x * base + (x < extra ? x : extra)) * np + k;
  } else {
    const int W = U * np;
    const int chunk = (W + kNumXcd - 1) / kNumXcd;
    pos = x * chunk + k;
    if (k >= chunk || pos >= W) return -1;
  }
  const int unit = order ? order[pos / np] : pos / np;
  return (unit >= 0 && unit < U) ? unit * np + pos % np : -1;
}
inline unsigned work_grid(int U, int np) {
  const int per_xcd = U >= kNumXcd ? (U + kNumXcd - 1) / kNumXcd * np : (U * np + kNumXcd - 1) / kNumXcd;
  return (unsigned)(kNumXcd * per_xcd);
}

// Starting point of a q-block's kv walk.  The workgroups an XCD runs at one
// time hold about 128 neighbouring q-blocks, whose lists share most of their
// kv blocks; walked from the lowest id they drift apart, because each one
// starts when an earlier one ends.  Starting q-block i at its first listed
// block with id >= (i n / kRotDiv) mod n and wrapping round moves the start
// along with the dispatch, so the workgroups in flight read nearly the same
// kv blocks at the same time and more of those reads hit the XCD's L2.  The
// rotation changes only the order in which a row's blocks are accumulated.
// Dense attention (no mask) keeps the natural order: there every q-block
// lists every block, and starting all of them at block 0 shares more.
constexpr int kRotDiv = 192;
__device__ inline int walk_target(int i, int n) { return (int)((int64_t)i * n / kRotDiv % n); }

// Offset in [0, p1 - p0) of the first position p of [p0, p1) whose id(p)
// reaches `target` (ids ascending), 0 when none does: the rotation of the
// walk over [p0, p1).  Any other id order still gives a rotation, so every
// position is visited once whatever the row holds.
template <class F>
__device__ inline int walk_rotation(int p0, int p1, int target, F id) {
  int lo = p0, hi = p1;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (id(mid) < target)
      lo = mid + 1;
    else
      hi = mid;
  }
  return lo == p1 ? 0 : lo - p0;
}

// One global -> LDS direct load (16 bytes per lane, lane-linear destination
// at `lds`, a wave-uniform LDS byte address).  The LDS address travels in
// m0; the statement saves m0 to a scratch SGPR, sets it, waits the one wait
// state an m0 write needs before an LDS-DMA read of it, issues the load and
// puts m0 back, so whatever the compiler keeps in m0 is unchanged after it.
// Inline asm rather than __builtin_amdgcn_global_load_lds: the compiler
// cannot tell which tile a direct load writes, and with the builtin it waits
// for every outstanding load (vmcnt(0)) before the next LDS read of any tile,
// which drains the prefetch of the following tile; the kernels wait on the
// vector-memory counter themselves.
__device__ inline void dma16(uint32_t lds, const void* sbase, uint32_t voff) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, %3\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds), "v"(voff), "s"(sbase)
      : "memory");
}

// Wait until at most n vector-memory loads of this wave are outstanding.
#define CHORUS_WAIT_VMCNT(n) asm volatile("s_waitcnt vmcnt(" #n ")" ::: "memory")

// Walk of the merged kv lists of the two q-blocks (2p, 2p + 1) of a pair,
// skipping ids outside [0, n).  Each list is walked from its rotated start
// (walk_target of q-block 2p, the same target for both; 0 for dense
// attention, where every q-block of a unit lists the same blocks and the
// natural order already keeps them together), and the merge takes
// the smaller of the two heads in that rotated order, key (id - target) mod n,
// so a block both lists hold is visited once.  All lanes hold the same state
// (it lives in scalar registers).  KV2: the lists hold kv blocks of 128 tokens
// and the walk visits both 64-token halves of each (positions of the doubled
// list), so ids stay in 64-token units.
template <bool KV2>
struct PairWalk {
  ConstI32* col;
  int a0, la, ra, ca;   // list A: first position, length, rotation, steps taken
  int b0, lb, rb, cb;
  int n, target;
  bool dense;
  __device__ void init(const AttnArgs& a, bool is_dense, int b, int h, int ip) {
    col = as_constant(a.col_idx);
    n = a.n;
    dense = is_dense;
    const int ia = 2 * ip, ib = 2 * ip + 1;
    // without a mask every q-block lists every block: natural order from block 0
    target = dense ? 0 : walk_target(ia, n);
    if (dense) {
      a0 = 0;
      la = n;
      b0 = 0;
      lb = ib < n ? n : 0;
    } else {
      const int64_t r0 = ((int64_t)(a.mask_batch > 1 ? b : 0) * a.H + h) * n;
      a0 = a.row_ptr[r0 + ia];
      la = a.row_ptr[r0 + ia + 1] - a0;
      b0 = ib < n ? a.row_ptr[r0 + ib] : 0;
      lb = ib < n ? a.row_ptr[r0 + ib + 1] - b0 : 0;
      if (KV2) {
        a0 *= 2;
        la *= 2;
        b0 *= 2;
        lb *= 2;
      }
    }
    auto id = [&](int p) { return id_at(p); };
    ra = walk_rotation(a0, a0 + la, target, id);
    rb = walk_rotation(b0, b0 + lb, target, id);
    ca = cb = 0;
  }
  __device__ bool listed(int sel) const { return sel == 0 ? la > 0 : lb > 0; }
  __device__ int id_at(int p) const { return dense ? p : KV2 ? 2 * col[p >> 1] + (p & 1) : col[p]; }
  __device__ int pos_a() const { const int p = ra + ca; return a0 + (p >= la ? p - la : p); }
  __device__ int pos_b() const { const int p = rb + cb; return b0 + (p >= lb ? p - lb : p); }
  __device__ int head_a() {
    while (ca < la) {
      const int j = id_at(pos_a());
      if (j >= 0 && j < n) return j;
      ++ca;
    }
    return INT32_MAX;
  }
  __device__ int head_b() {
    while (cb < lb) {
      const int j = id_at(pos_b());
      if (j >= 0 && j < n) return j;
      ++cb;
    }
    return INT32_MAX;
  }
  __device__ int key(int j) const { return j == INT32_MAX ? INT32_MAX : j >= target ? j - target : j - target + n; }
  // next kv block of the union (INT32_MAX when done) and which q-blocks list it
  __device__ int next(bool& in_a, bool& in_b) {
    const int ja = head_a(), jb = head_b();
    const int ka = key(ja), kb = key(jb);
    const int k = min(ka, kb);
    in_a = ka == k && k != INT32_MAX;
    in_b = kb == k && k != INT32_MAX;
    if (in_a) ++ca;
    if (in_b) ++cb;
    return in_a ? ja : jb;
  }
};

}  // namespace chorus
