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
// append: the same 32-token workgroups.  Lane j of each token writes the
// queue entry of slot j at its workgroup's first slot for that expert plus
// its rank -- the order is exactly (fragment, token, slot) within each
// expert's queue, with no atomics on the entries.  A workgroup's first slot
// is the queue's current depth plus the counts of the workgroups before it.
// Up to kDirectPrefixBlocks workgroups each append workgroup sums those
// counts itself (at most 63 per expert) and the last one publishes the new
// depths into the other half of the layer's depth ping-pong buffer (the host
// flips halves after the launch).  Above that, the router workgroup that
// finishes last (a counter, reset by that workgroup) scans every count once
// -- linear in T -- rewriting them into first slots and publishing the
// depths; small fragments skip it because its device-wide fences cost a few
// microseconds on the critical path.
#include <float.h>
#include <limits.h>

#include "aep_internal.h"

namespace aep {

static_assert(kMaxTopK <= kRouteLanes, "one slot per lane of a token");
static_assert(kMaxRouteExperts <= kRouteThreads, "one thread per expert in the rank walk");

// Per expert e, over workgroups b < nb of one router launch: blockcnt[b][e]
// (rows of workgroup b bound for e) becomes depth_cur[e] + sum_{b' < b}
// blockcnt[b'][e], the first queue slot of workgroup b's rows, and
// depth_nxt[e] = depth_cur[e] + sum_b blockcnt[b][e].  One workgroup:
// P = 256 / ES threads per expert (ES = E rounded up to a power of two)
// each own a contiguous run of workgroups; a first pass sums the runs, the
// run totals are scanned in LDS, a second pass writes the prefixes.  Counts
// written by other workgroups of the launch are visible after the acquire
// fence the caller issues before the scan (it invalidates this CU's vector
// cache).
__device__ void scan_counts(int32_t* blockcnt, int nb, int E, const int32_t* depth_cur, int32_t* depth_nxt) {
  __shared__ int32_t run_sum[kRouteThreads];
  const int tid = threadIdx.x;
  int es = 1;
  while (es < E) es <<= 1;
  const int P = kRouteThreads / es;
  const int e = tid % es, p = tid / es;
  const int per = (nb + P - 1) / P;
  const int b0 = min(nb, p * per), b1 = min(nb, b0 + per);
  int acc = 0;
  if (e < E)
    for (int b = b0; b < b1; ++b)
      acc += blockcnt[(int64_t)b * E + e];
  run_sum[tid] = acc;
  __syncthreads();
  if (tid < E) {
    // exclusive scan over the runs of expert tid, seeded with its depth
    int x = depth_cur[tid];
    for (int q = 0; q < P; ++q) {
      const int v = run_sum[q * es + tid];
      run_sum[q * es + tid] = x;
      x += v;
    }
    depth_nxt[tid] = x;
  }
  __syncthreads();
  if (e < E) {
    int x = run_sum[tid];
    for (int b = b0; b < b1; ++b) {
      const int64_t i = (int64_t)b * E + e;
      const int v = blockcnt[i];
      blockcnt[i] = x;
      x += v;
    }
  }
}

template <int EPL>
__global__ __launch_bounds__(kRouteThreads) void route_count_kernel(
    const float* __restrict__ logits, int T, int E, int k, int renorm, int32_t* __restrict__ r_idx,
    float* __restrict__ r_w, int32_t* __restrict__ r_rank, int32_t* blockcnt,
    int32_t* __restrict__ idx_out, float* __restrict__ w_out, const int32_t* __restrict__ depth_cur,
    int32_t* __restrict__ depth_nxt, int32_t* done, int32_t* __restrict__ err) {
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

  // Large launches: the last workgroup to finish scans every workgroup's
  // counts (smaller ones are summed by the append workgroups).
  if ((int)gridDim.x <= kDirectPrefixBlocks) return;
  __shared__ int last;
  __threadfence();  // this workgroup's counts are visible device-wide
  __syncthreads();
  if (tid == 0) last = atomicAdd(done, 1) == (int)gridDim.x - 1;
  __syncthreads();
  if (!last) return;
  __threadfence();
  scan_counts(blockcnt, (int)gridDim.x, E, depth_cur, depth_nxt);
  if (tid == 0) *done = 0;  // ready for the next launch
}

__global__ __launch_bounds__(kRouteThreads) void append_kernel(
    const int32_t* __restrict__ r_idx, const float* __restrict__ r_w,
    const int32_t* __restrict__ r_rank, const int32_t* __restrict__ first_slot, int T, int E, int k,
    const char* x, int64_t row_bytes, int32_t token_base, const int32_t* __restrict__ depth_cur,
    int32_t* __restrict__ depth_nxt, QEntry* __restrict__ q, int64_t q_stride,
    const void** __restrict__ tok_row, const int32_t* __restrict__ token_ids, int n_ids,
    int32_t* __restrict__ live, int32_t* __restrict__ pend, int32_t* __restrict__ err) {
  __shared__ int32_t base[kMaxRouteExperts];
  const int tid = threadIdx.x;
  if ((int)gridDim.x > kDirectPrefixBlocks) {
    if (tid < E) base[tid] = first_slot[(int64_t)blockIdx.x * E + tid];  // scanned by the router
  } else {
    // the counts of the workgroups before this one, split over kParts
    // threads per expert
    constexpr int kParts = kRouteThreads / kMaxRouteExperts;
    __shared__ int32_t part[kParts][kMaxRouteExperts];
    const int e = tid % kMaxRouteExperts, pp = tid / kMaxRouteExperts;
    int acc = 0;
    if (e < E)
      for (int b = pp; b < (int)blockIdx.x; b += kParts) acc += first_slot[(int64_t)b * E + e];
    part[pp][e] = acc;
    __syncthreads();
    if (tid < E) {
      int a = depth_cur[tid];
#pragma unroll
      for (int i = 0; i < kParts; ++i) a += part[i][tid];
      base[tid] = a;
      if (blockIdx.x == gridDim.x - 1) depth_nxt[tid] = a + first_slot[(int64_t)blockIdx.x * E + tid];
    }
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

// Rows of several experts in one launch: rows [pre[e], pre[e+1]) go to
// queue e (pre is the exclusive prefix of the per-expert counts, E + 1
// entries), each expert's rows in order -- the entries one enqueue_rows
// launch per expert, experts in ascending order, would write.
__global__ __launch_bounds__(256) void enqueue_grouped_kernel(
    const char* rows, int64_t row_bytes, const int32_t* __restrict__ token_ids,
    const int32_t* __restrict__ slots, const float* __restrict__ gate_w, int n, int n_tokens, int k, int E,
    const int32_t* __restrict__ pre, const int32_t* __restrict__ depth_cur, int32_t* __restrict__ depth_nxt,
    QEntry* __restrict__ q, int64_t q_stride, int32_t* __restrict__ err) {
  __shared__ int32_t sp[kMaxGroups + 1];
  for (int e = threadIdx.x; e <= E; e += blockDim.x) sp[e] = pre[e];
  __syncthreads();
  if (blockIdx.x == 0)
    for (int e = threadIdx.x; e < E; e += blockDim.x) depth_nxt[e] = depth_cur[e] + (sp[e + 1] - sp[e]);
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  int lo = 0, hi = E;  // sp[lo] <= i < sp[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (sp[mid] <= i)
      lo = mid;
    else
      hi = mid;
  }
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
  q[(int64_t)lo * q_stride + depth_cur[lo] + (i - sp[lo])] = en;
}

hipError_t launch_enqueue_grouped(const char* rows, int64_t row_bytes, const int32_t* token_ids,
                                  const int32_t* slots, const float* gate_w, int n, int n_tokens, int k, int E,
                                  const int32_t* pre, const int32_t* depth_cur, int32_t* depth_nxt, QEntry* q,
                                  int64_t q_stride, int32_t* err, hipStream_t s) {
  const int nb = (n + 255) / 256;
  enqueue_grouped_kernel<<<nb, 256, 0, s>>>(rows, row_bytes, token_ids, slots, gate_w, n, n_tokens, k, E, pre,
                                             depth_cur, depth_nxt, q, q_stride, err);
  return hipGetLastError();
}

hipError_t launch_route(const float* logits, int T, int E, int k, int renorm, int32_t* r_idx,
                        float* r_w, int32_t* r_rank, int32_t* blockcnt, int32_t* idx_out,
                        float* w_out, const int32_t* depth_cur, int32_t* depth_nxt, int32_t* done,
                        int32_t* err, hipStream_t s) {
  const int nb = (T + kRouteTokens - 1) / kRouteTokens;
  if (E <= 8)
    route_count_kernel<1><<<nb, kRouteThreads, 0, s>>>(logits, T, E, k, renorm, r_idx, r_w, r_rank,
                                                        blockcnt, idx_out, w_out, depth_cur, depth_nxt, done, err);
  else if (E <= 16)
    route_count_kernel<2><<<nb, kRouteThreads, 0, s>>>(logits, T, E, k, renorm, r_idx, r_w, r_rank,
                                                        blockcnt, idx_out, w_out, depth_cur, depth_nxt, done, err);
  else if (E <= 32)
    route_count_kernel<4><<<nb, kRouteThreads, 0, s>>>(logits, T, E, k, renorm, r_idx, r_w, r_rank,
                                                        blockcnt, idx_out, w_out, depth_cur, depth_nxt, done, err);
  else
    route_count_kernel<8><<<nb, kRouteThreads, 0, s>>>(logits, T, E, k, renorm, r_idx, r_w, r_rank,
                                                        blockcnt, idx_out, w_out, depth_cur, depth_nxt, done, err);
  return hipGetLastError();
}

hipError_t launch_append(const int32_t* r_idx, const float* r_w, const int32_t* r_rank,
                         const int32_t* first_slot, int T, int E, int k, const char* x,
                         int64_t row_bytes, int32_t token_base, const int32_t* depth_cur,
                         int32_t* depth_nxt, QEntry* q, int64_t q_stride, const void** tok_row,
                         const int32_t* token_ids, int n_ids, int32_t* live, int32_t* pend,
                         int32_t* err, hipStream_t s) {
  const int nb = (T + kRouteTokens - 1) / kRouteTokens;
  append_kernel<<<nb, kRouteThreads, 0, s>>>(r_idx, r_w, r_rank, first_slot, T, E, k, x, row_bytes,
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
