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

// Work item of dispatch slot p: slots are dealt round-robin to the 8 XCDs, so
// slot p runs on XCD p % 8; XCD x walks positions [x * chunk, (x + 1) * chunk)
// of the (optionally planned) item order.  Returns -1 for idle slots.
__device__ inline int work_item(const int32_t* order, int chunk, int W) {
  const int p = blockIdx.x;
  const int pos = (p % kNumXcd) * chunk + p / kNumXcd;
  if (pos >= W) return -1;
  const int item = order ? order[pos] : pos;
  return (item >= 0 && item < W) ? item : -1;
}

}  // namespace chorus
