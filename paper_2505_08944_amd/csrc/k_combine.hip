// Top-K merge (combine) and the fp8 -> bf16 decode utility.
//
// combine: one wave per token; each lane owns 16-byte column chunks of the
// output row (two per pass).  The token's (row, weight) pairs are read once
// (wave-uniform); a pass loads the chunks of every slot's row before adding
// any, so the loads are in flight together; partial sums stay in f32 in slot
// order, then shared-expert rows are added, and the result is rounded once.
// No atomics: the order is fixed, so the output is bit-reproducible.
#include "aep_device.h"
#include "aep_internal.h"

namespace aep {

typedef unsigned v4u __attribute__((ext_vector_type(4)));

template <bool BF16>
__device__ __forceinline__ void add_row(float (&acc)[BF16 ? 8 : 4], const v4u v, float w) {
  const uint32_t u[4] = {v.x, v.y, v.z, v.w};
  if constexpr (BF16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc[2 * i] = fmaf(w, bf16_lo(u[i]), acc[2 * i]);
      acc[2 * i + 1] = fmaf(w, bf16_hi(u[i]), acc[2 * i + 1]);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = fmaf(w, __uint_as_float(u[i]), acc[i]);
  }
}

template <bool BF16>
__device__ __forceinline__ void add_shared(float (&acc)[BF16 ? 8 : 4], const v4u v) {
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

template <bool BF16, int K>
__global__ __launch_bounds__(256) void combine_kernel(const void* __restrict__ y, int64_t N,
                                                      int n_tokens, int S,
                                                      const int32_t* __restrict__ pos,
                                                      const float* __restrict__ posw,
                                                      void* __restrict__ out, int d) {
  constexpr int kPer = BF16 ? 8 : 4;  // elements per 16-byte chunk
  constexpr int kU = 2;               // chunks per lane per pass
  constexpr int kSh = 2;              // shared rows loaded together
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= n_tokens) return;
  // the token's slots, wave-uniform; an absent slot (-1) reads row 0 and
  // adds nothing
  int p[K];
  float w[K];
  bool ok[K];
#pragma unroll
  for (int j = 0; j < K; ++j) {
    const int pj = __builtin_amdgcn_readfirstlane(pos[t * K + j]);
    ok[j] = pj >= 0;
    p[j] = ok[j] ? pj : 0;
    w[j] = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(posw[t * K + j])));
  }
  typedef const __attribute__((address_space(1))) v4u* gsrc_t;
  const gsrc_t yb = (gsrc_t)y;
  const int64_t rowc = d / kPer;  // 16-byte chunks per row
  const int nchunk = (int)rowc;
  for (int c0 = 0; c0 < nchunk; c0 += 64 * kU) {
    // every load of a pass is issued before the first addition (no branch
    // between a load and its use); additions keep slot order
    int cc[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) cc[u] = min(c0 + lane + 64 * u, nchunk - 1);
    v4u v[K][kU];
#pragma unroll
    for (int j = 0; j < K; ++j)
#pragma unroll
      for (int u = 0; u < kU; ++u) v[j][u] = yb[p[j] * rowc + cc[u]];
    float acc[kU][kPer];
#pragma unroll
    for (int u = 0; u < kU; ++u)
#pragma unroll
      for (int i = 0; i < kPer; ++i) acc[u][i] = 0.f;
#pragma unroll
    for (int j = 0; j < K; ++j)
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        float nx[kPer];
#pragma unroll
        for (int i = 0; i < kPer; ++i) nx[i] = acc[u][i];
        add_row<BF16>(nx, v[j][u], w[j]);
#pragma unroll
        for (int i = 0; i < kPer; ++i) acc[u][i] = ok[j] ? nx[i] : acc[u][i];
      }
    for (int s0 = 0; s0 < S; s0 += kSh) {
      v4u vs[kSh][kU];
#pragma unroll
      for (int q = 0; q < kSh; ++q) {
        const int64_t row = N + (int64_t)min(s0 + q, S - 1) * n_tokens + t;
#pragma unroll
        for (int u = 0; u < kU; ++u) vs[q][u] = yb[row * rowc + cc[u]];
      }
#pragma unroll
      for (int q = 0; q < kSh; ++q)
#pragma unroll
        for (int u = 0; u < kU; ++u) {
          float nx[kPer];
#pragma unroll
          for (int i = 0; i < kPer; ++i) nx[i] = acc[u][i];
          add_shared<BF16>(nx, vs[q][u]);
#pragma unroll
          for (int i = 0; i < kPer; ++i) acc[u][i] = (s0 + q < S) ? nx[i] : acc[u][i];
        }
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int c = c0 + lane + 64 * u;
      if (c0 + 64 * kU > nchunk && c >= nchunk) continue;  // only the row's last pass checks
      v4u o;
      if constexpr (BF16) {
        o.x = f32_to_bf16_rne(acc[u][0]) | (f32_to_bf16_rne(acc[u][1]) << 16);
        o.y = f32_to_bf16_rne(acc[u][2]) | (f32_to_bf16_rne(acc[u][3]) << 16);
        o.z = f32_to_bf16_rne(acc[u][4]) | (f32_to_bf16_rne(acc[u][5]) << 16);
        o.w = f32_to_bf16_rne(acc[u][6]) | (f32_to_bf16_rne(acc[u][7]) << 16);
      } else {
        o.x = __float_as_uint(acc[u][0]);
        o.y = __float_as_uint(acc[u][1]);
        o.z = __float_as_uint(acc[u][2]);
        o.w = __float_as_uint(acc[u][3]);
      }
      reinterpret_cast<v4u*>(out)[t * rowc + c] = o;
    }
  }
}

template <bool BF16>
static void combine_dispatch(int k, unsigned nb, const void* y, int64_t N, int n_tokens, int S,
                             const int32_t* pos, const float* posw, void* out, int d, hipStream_t s) {
  switch (k) {
    case 1: combine_kernel<BF16, 1><<<nb, 256, 0, s>>>(y, N, n_tokens, S, pos, posw, out, d); break;
    case 2: combine_kernel<BF16, 2><<<nb, 256, 0, s>>>(y, N, n_tokens, S, pos, posw, out, d); break;
    case 3: combine_kernel<BF16, 3><<<nb, 256, 0, s>>>(y, N, n_tokens, S, pos, posw, out, d); break;
    case 4: combine_kernel<BF16, 4><<<nb, 256, 0, s>>>(y, N, n_tokens, S, pos, posw, out, d); break;
    case 5: combine_kernel<BF16, 5><<<nb, 256, 0, s>>>(y, N, n_tokens, S, pos, posw, out, d); break;
    case 6: combine_kernel<BF16, 6><<<nb, 256, 0, s>>>(y, N, n_tokens, S, pos, posw, out, d); break;
    case 7: combine_kernel<BF16, 7><<<nb, 256, 0, s>>>(y, N, n_tokens, S, pos, posw, out, d); break;
    default: combine_kernel<BF16, 8><<<nb, 256, 0, s>>>(y, N, n_tokens, S, pos, posw, out, d); break;
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
  const unsigned nb = (unsigned)((n_tokens + 3) / 4);
  if (k < 1 || k > kMaxTopK) return hipErrorInvalidValue;
  if (act_dtype == 1)
    combine_dispatch<true>(k, nb, y, N, n_tokens, S, pos, posw, out, d, s);
  else
    combine_dispatch<false>(k, nb, y, N, n_tokens, S, pos, posw, out, d, s);
  return hipGetLastError();
}

hipError_t launch_fp8_to_bf16(const uint8_t* codes, uint16_t* out, int64_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int64_t nb = ((n + 3) / 4 + 255) / 256;
  fp8_to_bf16_kernel<<<(unsigned)nb, 256, 0, s>>>(codes, out, n);
  return hipGetLastError();
}

}  // namespace aep
