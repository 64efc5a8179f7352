// Top-K merge (combine) and the fp8 -> bf16 decode utility.
//
// combine: one wave per token; each lane owns 16-byte column chunks of the
// output row.  The token's (row, weight) pairs are read once into registers;
// partial sums stay in f32 in slot order, then shared-expert rows are added,
// and the result is rounded once.  No atomics: the order is fixed, so the
// output is bit-reproducible.
#include "aep_device.h"
#include "aep_internal.h"

namespace aep {

template <bool BF16>
__global__ __launch_bounds__(256) void combine_kernel(const void* __restrict__ y, int64_t N,
                                                      int n_tokens, int S, int k,
                                                      const int32_t* __restrict__ pos,
                                                      const float* __restrict__ posw,
                                                      void* __restrict__ out, int d) {
  constexpr int kPer = BF16 ? 8 : 4;  // elements per 16-byte chunk
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= n_tokens) return;
  int p[kMaxTopK];
  float w[kMaxTopK];
#pragma unroll
  for (int j = 0; j < kMaxTopK; ++j) {
    p[j] = (j < k) ? pos[t * k + j] : -1;
    w[j] = (j < k) ? posw[t * k + j] : 0.f;
  }
  const int esz = BF16 ? 2 : 4;
  const char* yb = reinterpret_cast<const char*>(y);
  const int nchunk = d / kPer;
  for (int c = lane; c < nchunk; c += 64) {
    float acc[kPer];
#pragma unroll
    for (int i = 0; i < kPer; ++i) acc[i] = 0.f;
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
      if (p[j] < 0) continue;
      const uint4 v = *reinterpret_cast<const uint4*>(yb + ((int64_t)p[j] * d + (int64_t)c * kPer) * esz);
      const uint32_t u[4] = {v.x, v.y, v.z, v.w};
      if constexpr (BF16) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          acc[2 * i] = fmaf(w[j], bf16_lo(u[i]), acc[2 * i]);
          acc[2 * i + 1] = fmaf(w[j], bf16_hi(u[i]), acc[2 * i + 1]);
        }
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] = fmaf(w[j], __uint_as_float(u[i]), acc[i]);
      }
    }
    for (int s = 0; s < S; ++s) {
      const int64_t row = N + (int64_t)s * n_tokens + t;
      const uint4 v = *reinterpret_cast<const uint4*>(yb + (row * d + (int64_t)c * kPer) * esz);
      const uint32_t u[4] = {v.x, v.y, v.z, v.w};
      if constexpr (BF16) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          acc[2 * i] += bf16_lo(u[i]);
          acc[2 * i + 1] += bf16_hi(u[i]);
        }
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] += __uint_as_float(u[i]);
      }
    }
    uint4 o;
    if constexpr (BF16) {
      o.x = f32_to_bf16_rne(acc[0]) | (f32_to_bf16_rne(acc[1]) << 16);
      o.y = f32_to_bf16_rne(acc[2]) | (f32_to_bf16_rne(acc[3]) << 16);
      o.z = f32_to_bf16_rne(acc[4]) | (f32_to_bf16_rne(acc[5]) << 16);
      o.w = f32_to_bf16_rne(acc[6]) | (f32_to_bf16_rne(acc[7]) << 16);
    } else {
      o.x = __float_as_uint(acc[0]);
      o.y = __float_as_uint(acc[1]);
      o.z = __float_as_uint(acc[2]);
      o.w = __float_as_uint(acc[3]);
    }
    *reinterpret_cast<uint4*>(reinterpret_cast<char*>(out) + (t * d + (int64_t)c * kPer) * esz) = o;
  }
}

__global__ void fp8_to_bf16_kernel(const uint8_t* __restrict__ in, uint16_t* __restrict__ out,
                                   int64_t n) {
  const int64_t i0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;  // four codes per thread
  if (i0 >= n) return;
  const int m = n - i0 < 4 ? (int)(n - i0) : 4;
  uint32_t w = 0;
  for (int j = 0; j < m; ++j) w |= (uint32_t)in[i0 + j] << (8 * j);
  const uint2 v = e4m3x4_to_bf16x4(w);
  const uint16_t h[4] = {(uint16_t)v.x, (uint16_t)(v.x >> 16), (uint16_t)v.y, (uint16_t)(v.y >> 16)};
  for (int j = 0; j < m; ++j) out[i0 + j] = h[j];
}

hipError_t launch_combine(int act_dtype, const void* y, int64_t N, int n_tokens, int S, int k,
                          const int32_t* pos, const float* posw, void* out, int d, hipStream_t s) {
  if (n_tokens == 0) return hipSuccess;
  const int nb = (n_tokens + 3) / 4;
  if (act_dtype == 1)
    combine_kernel<true><<<nb, 256, 0, s>>>(y, N, n_tokens, S, k, pos, posw, out, d);
  else
    combine_kernel<false><<<nb, 256, 0, s>>>(y, N, n_tokens, S, k, pos, posw, out, d);
  return hipGetLastError();
}

hipError_t launch_fp8_to_bf16(const uint8_t* codes, uint16_t* out, int64_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int64_t nb = ((n + 3) / 4 + 255) / 256;
  fp8_to_bf16_kernel<<<(unsigned)nb, 256, 0, s>>>(codes, out, n);
  return hipGetLastError();
}

}  // namespace aep
