// Device helpers shared by libaep's kernels: element-format conversions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace aep {

__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

// f32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// OCP e4m3fn code -> bf16 bits, exact: normal codes move the exponent (bias
// 7 -> 127) and the mantissa (3 -> 7 bits); subnormal codes m * 2^-9 go
// through an exact f32 product; S.1111.111 becomes a quiet NaN.
__device__ __forceinline__ uint32_t e4m3_to_bf16_bits(uint32_t b) {
  const uint32_t sgn = (b & 0x80u) << 8;
  const uint32_t em = b & 0x7fu;
  if (em == 0x7fu) return sgn | 0x7fc0u;
  if (em >= 8u) return sgn | ((em + (120u << 3)) << 4);
  return sgn | (__float_as_uint((float)em * 0x1p-9f) >> 16);
}

}  // namespace aep
