// Receptor kernels: top-k router + mu-queue append, and explicit-row enqueue.
//
// route_count: one thread per token.  Selects the top-k experts on the f32
// gate logits (larger first, equal -> lower id), computes the softmax weights
// of the selected experts, and ranks each (token, slot) among the block's
// rows bound for the same expert with a wave64 ballot + popcount and a scan
// over the block's four waves.  Per-block expert counts go to `blockcnt`.
//
// append: every block adds the counts of the blocks before it (and the
// queue's current depth) to get stable global positions, then writes one
// queue entry per (token, slot) -- the order is exactly (fragment, token,
// slot) within each expert's queue, with no atomics.  The last block
// publishes the new depths into the other half of the layer's depth
// ping-pong buffer; the host flips halves after the launch.
#include <float.h>

#include "aep_internal.h"

namespace aep {

template <int EMAX>
__global__ __launch_bounds__(kRouteThreads) void route_count_kernel(
    const float* __restrict__ logits, int T, int E, int k, int renorm, int32_t* __restrict__ r_idx,
    float* __restrict__ r_w, int32_t* __restrict__ r_rank, int32_t* __restrict__ blockcnt,
    int32_t* __restrict__ idx_out, float* __restrict__ w_out, int32_t* __restrict__ err) {
  constexpr int kWaves = kRouteThreads / 64;
  __shared__ int32_t wave_cnt[kWaves][EMAX];
  __shared__ int32_t wave_off[kWaves][EMAX];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t = blockIdx.x * kRouteThreads + tid;
  const bool valid = t < T;

  float v[EMAX];
  bool bad = false;
#pragma unroll
  for (int e = 0; e < EMAX; ++e) {
    float x = -FLT_MAX;
    if (valid && e < E) {
      x = logits[(int64_t)t * E + e];
      if (!__builtin_isfinite(x)) {
        bad = true;
        x = -FLT_MAX;
      }
    }
    v[e] = x;
  }

  // top-k: k passes of an arg-max over the not-yet-selected experts
  uint64_t mask = 0;
  int sel_i[kMaxTopK];
  float sel_v[kMaxTopK];
#pragma unroll
  for (int j = 0; j < kMaxTopK; ++j) {
    int bi = -1;
    float bv = 0.f;
    if (j < k) {
#pragma unroll
      for (int e = 0; e < EMAX; ++e) {
        if (e < E && !((mask >> e) & 1ull) && (bi < 0 || v[e] > bv)) {
          bi = e;
          bv = v[e];
        }
      }
      mask |= 1ull << bi;
    }
    sel_i[j] = bi;
    sel_v[j] = bv;
  }

  // softmax weights of the selected experts
  const float m = sel_v[0];
  float ex[kMaxTopK];
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < kMaxTopK; ++j) ex[j] = (j < k) ? expf(sel_v[j] - m) : 0.f;
  if (renorm) {
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j)
      if (j < k) s += ex[j];
  } else {
#pragma unroll
    for (int e = 0; e < EMAX; ++e)
      if (e < E) s += expf(v[e] - m);
  }

  // rank of each (token, slot) among this wave's rows for the same expert
  const uint64_t my = valid ? mask : 0ull;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  int rank_w[kMaxTopK];
#pragma unroll
  for (int j = 0; j < kMaxTopK; ++j) rank_w[j] = 0;
  for (int e = 0; e < E; ++e) {
    const uint64_t b = __ballot((int)((my >> e) & 1ull));
    if (lane == 0) wave_cnt[wave][e] = __popcll(b);
    if ((my >> e) & 1ull) {
      const int r = __popcll(b & below);
#pragma unroll
      for (int j = 0; j < kMaxTopK; ++j)
        if (j < k && sel_i[j] == e) rank_w[j] = r;
    }
  }
  __syncthreads();
  if (tid < E) {
    int acc = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      wave_off[w][tid] = acc;
      acc += wave_cnt[w][tid];
    }
    blockcnt[(int64_t)blockIdx.x * E + tid] = acc;
  }
  __syncthreads();

  if (valid) {
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
      if (j < k) {
        const int64_t o = (int64_t)t * k + j;
        const float w = ex[j] / s;
        r_idx[o] = sel_i[j];
        r_w[o] = w;
        r_rank[o] = wave_off[wave][sel_i[j]] + rank_w[j];
        if (idx_out) idx_out[o] = sel_i[j];
        if (w_out) w_out[o] = w;
      }
    }
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
  __shared__ int32_t base[kMaxRouteExperts];
  const int tid = threadIdx.x;
  if (tid < E) {
    int acc = depth_cur[tid];
    for (int b = 0; b < (int)blockIdx.x; ++b) acc += blockcnt[(int64_t)b * E + tid];
    base[tid] = acc;
    if (blockIdx.x == gridDim.x - 1) depth_nxt[tid] = acc + blockcnt[(int64_t)blockIdx.x * E + tid];
  }
  __syncthreads();
  const int t = blockIdx.x * kRouteThreads + tid;
  if (t >= T) return;
  const char* row = x + (int64_t)t * row_bytes;
  int tok = token_base + t;
  if (token_ids) {
    // caller id: claim its pool entry (an id still claimed, or out of
    // range, is an error; the row is filed under a clamped id)
    tok = token_ids[t];
    if (tok < 0 || tok >= n_ids) {
      atomicOr(err, kErrTokenRange);
      tok = tok < 0 ? 0 : n_ids - 1;
    } else if (atomicExch(&live[tok], 1) != 0) {
      atomicOr(err, kErrCollision);
    }
    pend[tok] = k;
  }
  for (int j = 0; j < k; ++j) {
    const int64_t o = (int64_t)t * k + j;
    const int e = r_idx[o];
    QEntry en;
    en.row = row;
    en.token_slot = tok | (j << kTokenBits);
    en.w = r_w[o];
    q[(int64_t)e * q_stride + base[e] + r_rank[o]] = en;
  }
  tok_row[tok] = row;
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
  const int nb = (T + kRouteThreads - 1) / kRouteThreads;
  if (E <= 8)
    route_count_kernel<8><<<nb, kRouteThreads, 0, s>>>(logits, T, E, k, renorm, r_idx, r_w, r_rank,
                                                        blockcnt, idx_out, w_out, err);
  else if (E <= 16)
    route_count_kernel<16><<<nb, kRouteThreads, 0, s>>>(logits, T, E, k, renorm, r_idx, r_w, r_rank,
                                                         blockcnt, idx_out, w_out, err);
  else if (E <= 32)
    route_count_kernel<32><<<nb, kRouteThreads, 0, s>>>(logits, T, E, k, renorm, r_idx, r_w, r_rank,
                                                         blockcnt, idx_out, w_out, err);
  else
    route_count_kernel<64><<<nb, kRouteThreads, 0, s>>>(logits, T, E, k, renorm, r_idx, r_w, r_rank,
                                                         blockcnt, idx_out, w_out, err);
  return hipGetLastError();
}

hipError_t launch_append(const int32_t* r_idx, const float* r_w, const int32_t* r_rank,
                         const int32_t* blockcnt, int T, int E, int k, const char* x,
                         int64_t row_bytes, int32_t token_base, const int32_t* depth_cur,
                         int32_t* depth_nxt, QEntry* q, int64_t q_stride, const void** tok_row,
                         const int32_t* token_ids, int n_ids, int32_t* live, int32_t* pend,
                         int32_t* err, hipStream_t s) {
  const int nb = (T + kRouteThreads - 1) / kRouteThreads;
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
