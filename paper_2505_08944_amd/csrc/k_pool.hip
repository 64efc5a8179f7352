// Token pool: the top-K merge across drains.  When a layer's experts are
// drained one at a time, a token's k rows are computed in different drains;
// each drain adds its rows, weighted by their gate weights, into the token's
// f32 pool row, and a token is released -- rounded once to the activation
// type and its pool row cleared -- when all k rows have been added.
//
// accumulate: one wave per batch row.  A single-expert batch holds at most one
// row per token, so no two waves touch the same pool row and no atomics are
// needed; the per-token count of rows still to come is decremented by lane 0.
// release: one wave per token id; tokens that are not complete are skipped
// after two loads.
#include "aep_device.h"
#include "aep_internal.h"

namespace aep {

template <bool BF16>
__global__ __launch_bounds__(256) void pool_accumulate_kernel(const void* __restrict__ y, int64_t N,
                                                              const int32_t* __restrict__ offsets,
                                                              int E, const int32_t* __restrict__ row_token,
                                                              const float* __restrict__ row_w,
                                                              float* __restrict__ pool,
                                                              int32_t* __restrict__ pend, int d) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= N || r >= offsets[E]) return;
  const int tok = row_token[r];
  const float w = row_w[r];
  float* dst = pool + (int64_t)tok * d;
  if (BF16) {
    const uint16_t* src = reinterpret_cast<const uint16_t*>(y) + r * d;
    for (int c = lane * 2; c < d; c += 128) {
      const uint32_t v = *reinterpret_cast<const uint32_t*>(src + c);
      float2 a = *reinterpret_cast<float2*>(dst + c);
      a.x = fmaf(w, bf16_lo(v), a.x);
      a.y = fmaf(w, bf16_hi(v), a.y);
      *reinterpret_cast<float2*>(dst + c) = a;
    }
  } else {
    const float* src = reinterpret_cast<const float*>(y) + r * d;
    for (int c = lane; c < d; c += 64) dst[c] = fmaf(w, src[c], dst[c]);
  }
  if (lane == 0) pend[tok] -= 1;
}

template <bool BF16>
__global__ __launch_bounds__(256) void pool_release_kernel(float* __restrict__ pool,
                                                           int32_t* __restrict__ live,
                                                           int32_t* __restrict__ pend, int n_ids,
                                                           void* __restrict__ out,
                                                           int32_t* __restrict__ ready, int d) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= n_ids) return;
  const bool done = live[t] != 0 && pend[t] == 0;
  if (ready && lane == 0) ready[t] = done ? 1 : 0;
  if (!done) return;
  float* src = pool + (int64_t)t * d;
  if (BF16) {
    uint16_t* o = reinterpret_cast<uint16_t*>(out) + (int64_t)t * d;
    for (int c = lane * 2; c < d; c += 128) {
      const float2 a = *reinterpret_cast<const float2*>(src + c);
      *reinterpret_cast<uint32_t*>(o + c) = f32_to_bf16_rne(a.x) | (f32_to_bf16_rne(a.y) << 16);
      *reinterpret_cast<float2*>(src + c) = make_float2(0.f, 0.f);
    }
  } else {
    float* o = reinterpret_cast<float*>(out) + (int64_t)t * d;
    for (int c = lane; c < d; c += 64) {
      o[c] = src[c];
      src[c] = 0.f;
    }
  }
  if (lane == 0) live[t] = 0;
}

hipError_t launch_pool_accumulate(int act_dtype, const void* y, int64_t N, const int32_t* offsets,
                                  int E, const int32_t* row_token, const float* row_w, float* pool,
                                  int32_t* pend, int d, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  const unsigned nb = (unsigned)((N + 3) / 4);
  if (act_dtype == 0)
    pool_accumulate_kernel<false><<<nb, 256, 0, s>>>(y, N, offsets, E, row_token, row_w, pool, pend, d);
  else
    pool_accumulate_kernel<true><<<nb, 256, 0, s>>>(y, N, offsets, E, row_token, row_w, pool, pend, d);
  return hipGetLastError();
}

hipError_t launch_pool_release(int act_dtype, float* pool, int32_t* live, int32_t* pend, int n_ids,
                               void* out, int32_t* ready, int d, hipStream_t s) {
  const unsigned nb = (unsigned)((n_ids + 3) / 4);
  if (act_dtype == 0)
    pool_release_kernel<false><<<nb, 256, 0, s>>>(pool, live, pend, n_ids, out, ready, d);
  else
    pool_release_kernel<true><<<nb, 256, 0, s>>>(pool, live, pend, n_ids, out, ready, d);
  return hipGetLastError();
}

}  // namespace aep
