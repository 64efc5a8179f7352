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

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Four OCP e4m3fn codes (one 32-bit word, lowest byte first) -> four bf16
// (two words, lowest first).  gfx950's fp8 conversions use the OCP e4m3fn
// encoding; with a scale of 1 the conversion is exact (every e4m3 value is a
// bf16 value).
__device__ __forceinline__ uint2 e4m3x4_to_bf16x4(uint32_t w) {
  const bf16x2_t lo = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, false);
  const bf16x2_t hi = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, true);
  return make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
}

}  // namespace aep
