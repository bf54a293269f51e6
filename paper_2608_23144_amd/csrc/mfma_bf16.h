// Operand types and the exact bf16 split shared by the matrix-core screens
// (device code only).
#pragma once

#include "awsrc_internal.h"

namespace awsrc {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Exact three-way bf16 split of eight fp32 values, packed two per dword:
// each part is the previous remainder truncated to bf16, so hi + mid + lo
// equals the fp32 value (24 significand bits in three 8-bit pieces).
__device__ __forceinline__ void split3(const float (&u)[8], u32x4& hi, u32x4& mid, u32x4& lo) {
  uint32_t h[8], m[8], l[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint32_t ub = __float_as_uint(u[e]);
    h[e] = ub & 0xFFFF0000u;
    const float r1 = u[e] - __uint_as_float(h[e]);
    m[e] = __float_as_uint(r1) & 0xFFFF0000u;
    const float r2 = r1 - __uint_as_float(m[e]);
    l[e] = __float_as_uint(r2) & 0xFFFF0000u;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    hi[i] = (h[2 * i] >> 16) | h[2 * i + 1];
    mid[i] = (m[2 * i] >> 16) | m[2 * i + 1];
    lo[i] = (l[2 * i] >> 16) | l[2 * i + 1];
  }
}

}  // namespace awsrc
