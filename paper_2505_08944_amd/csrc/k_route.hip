// Receptor kernels: top-k router + mu-queue append, and explicit-row enqueue.
//
// route_count: eight lanes per token, 32 tokens per workgroup.  Lane g of a
// token holds the f32 gate logits of experts g, g + 8, g + 16, ...; each of
// the k selection rounds takes every lane's best remaining expert and reduces
// the eight candidates with xor shuffles (larger logit first, equal -> lower
// id), so all eight lanes agree on the pick and its owner lane retires it.
// The softmax weights of the selected experts follow; lane j keeps slot j.
// Each (token, slot) is then ranked among the workgroup's rows bound for the
// same expert: one thread per expert walks the 32 tokens' selection masks in
// token order.  Per-workgroup expert counts go to `blockcnt`.
//
// append: the same 32-token workgroups.  Every workgroup adds the counts of
// the workgroups before it (and the queue's current depth) to get stable
// global positions, then lane j of each token writes the queue entry of slot
// j -- the order is exactly (fragment, token, slot) within each expert's
// queue, with no atomics.  The last workgroup publishes the new depths into
// the other half of the layer's depth ping-pong buffer; the host flips
// halves after the launch.
#include <float.h>
#include <limits.h>

#include "aep_internal.h"

namespace aep {

static_assert(kMaxTopK <= kRouteLanes, "one slot per lane of a token");
static_assert(kMaxRouteExperts <= kRouteThreads, "one thread per expert in the rank walk");

template <int EPL>
__global__ __launch_bounds__(kRouteThreads) void route_count_kernel(
    const float* __restrict__ logits, int T, int E, int k, int renorm, int32_t* __restrict__ r_idx,
    float* __restrict__ r_w, int32_t* __restrict__ r_rank, int32_t* __restrict__ blockcnt,
    int32_t* __restrict__ idx_out, float* __restrict__ w_out, int32_t* __restrict__ err) {
  __shared__ uint64_t sel_mask[kRouteTokens];
  __shared__ uint8_t rank_s[kRouteTokens][kMaxRouteExperts];
  const int tid = threadIdx.x, g = tid & (kRouteLanes - 1), tb = tid / kRouteLanes;
  const int t = blockIdx.x * kRouteTokens + tb;
  const bool valid = t < T;

  float v[EPL];
  unsigned avail = 0;
  bool bad = false;
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = i * kRouteLanes + g;
    float x = -FLT_MAX;
    if (valid && e < E) {
      x = logits[(int64_t)t * E + e];
      if (!__builtin_isfinite(x)) {
        bad = true;
        x = -FLT_MAX;
      }
      avail |= 1u << i;
    }
    v[i] = x;
  }

  // k selection rounds; the renormalised sum adds the slots in slot order
  uint64_t mask = 0;
  float m = 0.f, s = 0.f, my_ex = 0.f;
  int my_e = 0;
#pragma unroll
  for (int j = 0; j < kMaxTopK; ++j) {
    if (j < k) {
      float bv = -__builtin_inff();
      int be = INT_MAX;
#pragma unroll
      for (int i = 0; i < EPL; ++i)
        if (((avail >> i) & 1u) && v[i] > bv) {
          bv = v[i];
          be = i * kRouteLanes + g;
        }
#pragma unroll
      for (int off = 1; off < kRouteLanes; off <<= 1) {
        const float ov = __shfl_xor(bv, off, kRouteLanes);
        const int oe = __shfl_xor(be, off, kRouteLanes);
        if (ov > bv || (ov == bv && oe < be)) {
          bv = ov;
          be = oe;
        }
      }
      if (j == 0) m = bv;
      const float ex = expf(bv - m);
      s += ex;
      if (g == j) {
        my_e = be;
        my_ex = ex;
      }
      if (valid) {
        mask |= 1ull << be;
        if ((be & (kRouteLanes - 1)) == g) avail &= ~(1u << (be / kRouteLanes));
      }
    }
  }
  if (!renorm) {
    // softmax over all E experts, then the top-k weights
    float p = 0.f;
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if (i * kRouteLanes + g < E) p += expf(v[i] - m);
#pragma unroll
    for (int off = 1; off < kRouteLanes; off <<= 1) p += __shfl_xor(p, off, kRouteLanes);
    s = p;
  }

  // rank of each (token, slot) among this workgroup's rows for its expert
  if (g == 0) sel_mask[tb] = valid ? mask : 0ull;
  __syncthreads();
  if (tid < E) {
    int acc = 0;
#pragma unroll 8
    for (int i = 0; i < kRouteTokens; ++i)
      if ((sel_mask[i] >> tid) & 1ull) rank_s[i][tid] = (uint8_t)acc++;
    blockcnt[(int64_t)blockIdx.x * E + tid] = acc;
  }
  __syncthreads();

  if (valid && g < k) {
    const int64_t o = (int64_t)t * k + g;
    const float w = my_ex / s;
    r_idx[o] = my_e;
    r_w[o] = w;
    r_rank[o] = rank_s[tb][my_e];
    if (idx_out) idx_out[o] = my_e;
    if (w_out) w_out[o] = w;
  }
  if (bad) atomicOr(err, kErrNonFinite);
}

__global__ __launch_bounds__(kRouteThreads) void append_kernel(
    const int32_t* __restrict__ r_idx, const float* __restrict__ r_w,
    const int32_t* __restrict__ r_rank, const int32_t* __restrict__ blockcnt, int T, int E, int k,
    const char* x, int64_t row_bytes, int32_t token_base, const int32_t* __restrict__ depth_cur,
    int32_t* __restrict__ depth_nxt, QEntry* __restrict__ q, int64_t q_stride,
    const void** __restrict__ tok_row, const int32_t* __restrict__ token_ids, int n_ids,
    int32_t* __restrict__ live, int32_t* __restrict__ pend, int32_t* __restrict__ err) {
  constexpr int kParts = kRouteThreads / kMaxRouteExperts;
  __shared__ int32_t part[kParts][kMaxRouteExperts];
  __shared__ int32_t base[kMaxRouteExperts];
  const int tid = threadIdx.x;
  {
    // counts of the workgroups before this one, split over kParts threads
    // per expert
    const int e = tid % kMaxRouteExperts, p = tid / kMaxRouteExperts;
    int acc = 0;
    if (e < E) {
      // 8 independent loads per round
      int b = p;
      for (; b + 7 * kParts < (int)blockIdx.x; b += 8 * kParts) {
        int v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = blockcnt[(int64_t)(b + i * kParts) * E + e];
#pragma unroll
        for (int i = 0; i < 8; ++i) acc += v[i];
      }
      for (; b < (int)blockIdx.x; b += kParts) acc += blockcnt[(int64_t)b * E + e];
    }
    part[p][e] = acc;
  }
  __syncthreads();
  if (tid < E) {
    int acc = depth_cur[tid];
#pragma unroll
    for (int p = 0; p < kParts; ++p) acc += part[p][tid];
    base[tid] = acc;
    if (blockIdx.x == gridDim.x - 1) depth_nxt[tid] = acc + blockcnt[(int64_t)blockIdx.x * E + tid];
  }
  __syncthreads();
  const int g = tid & (kRouteLanes - 1);
  const int t = blockIdx.x * kRouteTokens + tid / kRouteLanes;
  if (t >= T) return;
  const char* row = x + (int64_t)t * row_bytes;
  int tok = token_base + t;
  if (token_ids) {
    // caller id: claim its pool entry (an id still claimed, or out of
    // range, is an error; the row is filed under a clamped id)
    tok = token_ids[t];
    if (tok < 0 || tok >= n_ids) {
      if (g == 0) atomicOr(err, kErrTokenRange);
      tok = tok < 0 ? 0 : n_ids - 1;
    } else if (g == 0 && atomicExch(&live[tok], 1) != 0) {
      atomicOr(err, kErrCollision);
    }
    if (g == 0) pend[tok] = k;
  }
  if (g < k) {
    const int64_t o = (int64_t)t * k + g;
    const int e = r_idx[o];
    QEntry en;
    en.row = row;
    en.token_slot = tok | (g << kTokenBits);
    en.w = r_w[o];
    q[(int64_t)e * q_stride + base[e] + r_rank[o]] = en;
  }
  if (g == 0) tok_row[tok] = row;
}

__global__ __launch_bounds__(256) void enqueue_rows_kernel(
    const char* rows, int64_t row_bytes, const int32_t* __restrict__ token_ids,
    const int32_t* __restrict__ slots, const float* __restrict__ gate_w, int n, int n_tokens, int k,
    int expert, int E, const int32_t* __restrict__ depth_cur, int32_t* __restrict__ depth_nxt,
    QEntry* __restrict__ q, int64_t q_stride, int32_t* __restrict__ err) {
  if (blockIdx.x == 0)
    for (int e = threadIdx.x; e < E; e += blockDim.x)
      depth_nxt[e] = depth_cur[e] + (e == expert ? n : 0);
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  int tok = token_ids[i];
  int s = slots ? slots[i] : 0;
  int flag = 0;
  if (tok < 0 || tok >= n_tokens) {
    flag |= kErrTokenRange;
    tok = 0;
  }
  if (s < 0 || s >= k) {
    flag |= kErrSlotRange;
    s = 0;
  }
  if (flag) atomicOr(err, flag);
  QEntry en;
  en.row = rows + (int64_t)i * row_bytes;
  en.token_slot = tok | (s << kTokenBits);
  en.w = gate_w[i];
  q[(int64_t)expert * q_stride + depth_cur[expert] + i] = en;
}

hipError_t launch_route(const float* logits, int T, int E, int k, int renorm, int32_t* r_idx,
                        float* r_w, int32_t* r_rank, int32_t* blockcnt, int32_t* idx_out,
                        float* w_out, int32_t* err, hipStream_t s) {
  const int nb = (T + kRouteTokens - 1) / kRouteTokens;
  if (E <= 8)
    route_count_kernel<1><<<nb, kRouteThreads, 0, s>>>(logits, T, E, k, renorm, r_idx, r_w, r_rank,
                                                        blockcnt, idx_out, w_out, err);
  else if (E <= 16)
    route_count_kernel<2><<<nb, kRouteThreads, 0, s>>>(logits, T, E, k, renorm, r_idx, r_w, r_rank,
                                                        blockcnt, idx_out, w_out, err);
  else if (E <= 32)
    route_count_kernel<4><<<nb, kRouteThreads, 0, s>>>(logits, T, E, k, renorm, r_idx, r_w, r_rank,
                                                        blockcnt, idx_out, w_out, err);
  else
    route_count_kernel<8><<<nb, kRouteThreads, 0, s>>>(logits, T, E, k, renorm, r_idx, r_w, r_rank,
                                                        blockcnt, idx_out, w_out, err);
  return hipGetLastError();
}

hipError_t launch_append(const int32_t* r_idx, const float* r_w, const int32_t* r_rank,
                         const int32_t* blockcnt, int T, int E, int k, const char* x,
                         int64_t row_bytes, int32_t token_base, const int32_t* depth_cur,
                         int32_t* depth_nxt, QEntry* q, int64_t q_stride, const void** tok_row,
                         const int32_t* token_ids, int n_ids, int32_t* live, int32_t* pend,
                         int32_t* err, hipStream_t s) {
  const int nb = (T + kRouteTokens - 1) / kRouteTokens;
  append_kernel<<<nb, kRouteThreads, 0, s>>>(r_idx, r_w, r_rank, blockcnt, T, E, k, x, row_bytes,
                                              token_base, depth_cur, depth_nxt, q, q_stride, tok_row,
                                              token_ids, n_ids, live, pend, err);
  return hipGetLastError();
}

hipError_t launch_enqueue_rows(const char* rows, int64_t row_bytes, const int32_t* token_ids,
                               const int32_t* slots, const float* gate_w, int n, int n_tokens,
                               int k, int expert, int E, const int32_t* depth_cur,
                               int32_t* depth_nxt, QEntry* q, int64_t q_stride, int32_t* err,
                               hipStream_t s) {
  const int nb = (n + 255) / 256;
  enqueue_rows_kernel<<<nb, 256, 0, s>>>(rows, row_bytes, token_ids, slots, gate_w, n, n_tokens, k,
                                          expert, E, depth_cur, depth_nxt, q, q_stride, err);
  return hipGetLastError();
}

}  // namespace aep
