// Executor re-batch kernels: drain plan + gather.
//
// plan: workgroup 0 reads the drained layer's per-expert queue depths (or one
// expert's, for a single-expert drain) with one thread per group, and writes
// counts / exclusive-scan offsets / the FFN group table (row-tile families
// and tile ranges) from workgroup-wide scans, then the group of every tile of
// both FFN launches (a binary search of the family's tile starts in LDS per
// tile, all threads); it resets the drained queue depths to zero.  All
// workgroups clear the (token, slot) -> row map.
//
// gather: one wave per batch row.  A routed row finds its expert by binary
// search over the offsets, reads its queue entry and copies the referenced
// row (16-byte vector loads/stores, the whole wave on one row, so each row is
// one contiguous coalesced stream; up to 4 loads per lane in flight before
// the stores); lane 0 records the row's token and gate weight and the
// (token, slot) -> row map.  Shared-expert rows copy every token's row in id
// order.
#include <algorithm>

#include "aep_internal.h"

namespace aep {

struct NT6 {
  int v[6];
};

constexpr int kPlanThreads = 1024;

// Exclusive scan of NV ints per thread over a workgroup of kPlanThreads
// threads (inclusive wave scans with shuffles, then a scan of the wave
// totals by NV threads); `total` receives the workgroup sums.  wsum holds
// kPlanThreads / 64 + 1 rows.
template <int NV>
__device__ __forceinline__ void plan_block_scan(int (&v)[NV], int (&total)[NV],
                                                int32_t (*wsum)[NV]) {
  constexpr int kWaves = kPlanThreads / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) inc[i] = v[i];
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int y = __shfl_up(inc[i], off);
      if (lane >= off) inc[i] += y;
    }
  }
  if (lane == 63)
#pragma unroll
    for (int i = 0; i < NV; ++i) wsum[wave][i] = inc[i];
  __syncthreads();
  if (threadIdx.x < NV) {
    const int i = threadIdx.x;
    int acc = 0;
    for (int w = 0; w < kWaves; ++w) {
      const int x = wsum[w][i];
      wsum[w][i] = acc;
      acc += x;
    }
    wsum[kWaves][i] = acc;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    v[i] = wsum[wave][i] + inc[i] - v[i];
    total[i] = wsum[kWaves][i];
  }
  __syncthreads();
}

// Workgroup 0 plans the drain, one thread per group; every workgroup clears
// its share of the (token, slot) -> row map.
__global__ __launch_bounds__(kPlanThreads) void plan_kernel(int E, int S, int n_tokens, int k,
                                                            int only_expert, int32_t* __restrict__ depth,
                                                            int32_t* __restrict__ depth_other,
                                                            int32_t* __restrict__ counts,
                                                            int32_t* __restrict__ offsets,
                                                            GroupDesc* __restrict__ groups,
                                                            int32_t* __restrict__ tile_totals,
                                                            NT6 nt, int big_bm, int med_bm, int small_bm,
                                                            int num_cu,
                                                            int32_t* __restrict__ tile_group,
                                                            int64_t tile_cap,
                                                            int32_t* __restrict__ pos,
                                                            float* __restrict__ posw) {
  const int tid = threadIdx.x;
  if (blockIdx.x == 0) {
    __shared__ int32_t wsum4[kPlanThreads / 64 + 1][4];
    __shared__ int32_t wsum7[kPlanThreads / 64 + 1][7];
    const int G = E + S;
    const int g = tid;
    const bool real = g < G;
    const int n = !real ? 0 : g < E ? (only_expert < 0 || g == only_expert ? depth[g] : 0) : n_tokens;
    const int full = n / big_bm, r = n - full * big_bm;
    // routed rows; full big gate/up tiles of the whole batch; big row tiles
    // when a remainder above 3/4 of a big tile takes one more (rule A) and
    // when any remainder above one medium tile does (rule B)
    int a[4] = {g < E ? n : 0, full * nt.v[0], full + (r > big_bm - big_bm / 4 ? 1 : 0),
                full + (r > med_bm ? 1 : 0)};
    int sum4[4];
    plan_block_scan<4>(a, sum4, wsum4);
    const int N = sum4[0];
    // A batch whose full big tiles do not fill one round of the grid is
    // cold: its remainders go to medium tiles only (a few long big tiles
    // would be the critical path of a weight-streaming launch).
    const bool cold = sum4[1] < num_cu;
    int nrt[2][3] = {{0, 0, 0}, {0, 0, 0}};
    int fam1_rows[2] = {0, 0};   // rows covered by family 1 before the small tile
    int h1[2] = {med_bm, med_bm};  // rows per family-1 tile
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      // Rule B trades the medium and small tiles of a remainder (each
      // streams the expert's weights again, and their per-tile overheads
      // weigh more) for one big tile with idle rows; it is taken unless its
      // extra big tiles start another round of the grid in a stage that has
      // few rounds (there a round of long big tiles would run nearly alone).
      const int ntb = nt.v[3 * st];
      const int rounds_a = (sum4[2] * ntb + num_cu - 1) / num_cu;
      const int rounds_b = (sum4[3] * ntb + num_cu - 1) / num_cu;
      const int xbig = rounds_b == rounds_a || rounds_a >= 4 ? med_bm : big_bm - big_bm / 4;
      if (small_bm == 0) {
        nrt[st][0] = (n + big_bm - 1) / big_bm;
      } else if (cold && r > med_bm) {
        // full big tiles; a remainder above one medium tile takes one tall
        // tile (kTallBM rows: the expert's weights are read once)
        nrt[st][0] = full;
        nrt[st][1] = 1;
        h1[st] = kTallBM;
      } else if (r > xbig) {
        nrt[st][0] = full + 1;
      } else {
        // full big tiles, then full medium tiles; what is left goes to one
        // more medium tile above small_bm rows, else to one small tile
        nrt[st][0] = full;
        nrt[st][1] = r / med_bm;
        const int rem = r - nrt[st][1] * med_bm;
        if (rem > small_bm)
          nrt[st][1] += 1;
        else if (rem > 0)
          nrt[st][2] = 1;
        fam1_rows[st] = (r / med_bm) * med_bm;
      }
    }
    int b[7];
    b[0] = n;
#pragma unroll
    for (int i = 0; i < 6; ++i) b[1 + i] = nrt[i / 3][i % 3] * nt.v[i];
    int sum7[7];
    plan_block_scan<7>(b, sum7, wsum7);
    if (real) {
      GroupDesc gd;
      gd.n = n;
      gd.x_row0 = g < E ? b[0] : N;
      gd.y_row0 = b[0];
#pragma unroll
      for (int i = 0; i < 6; ++i) gd.t0[i] = b[1 + i];
#pragma unroll
      for (int st = 0; st < 2; ++st) {
#pragma unroll
        for (int f = 0; f < 3; ++f) gd.nrt[st][f] = nrt[st][f];
        gd.row1[st] = full * big_bm;
        gd.row2[st] = full * big_bm + fam1_rows[st];
        gd.h1[st] = h1[st];
      }
      gd.pad[0] = gd.pad[1] = gd.pad[2] = 0;
      groups[g] = gd;
      counts[g] = n;
      offsets[g] = b[0];
    }
    if (g == 0) {
      offsets[G] = sum7[0];
#pragma unroll
      for (int i = 0; i < 6; ++i) tile_totals[i] = sum7[1 + i];
    }
    // The group of every tile of both launches (tiles are numbered per
    // launch: the big family, then the medium, then the small): the last
    // group whose first tile in that family is not above the tile.
    __shared__ int32_t t0s[6][kMaxGroups + 1];
    if (real)
#pragma unroll
      for (int i = 0; i < 6; ++i) t0s[i][g] = b[1 + i];
    if (g == 0)
#pragma unroll
      for (int i = 0; i < 6; ++i) t0s[i][G] = sum7[1 + i];
    __syncthreads();
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const int tot0 = sum7[1 + 3 * st], tot1 = sum7[2 + 3 * st], tot2 = sum7[3 + 3 * st];
      for (int t = tid; t < tot0 + tot1 + tot2; t += kPlanThreads) {
        const int f = t < tot0 ? 0 : (t < tot0 + tot1 ? 1 : 2);
        const int local = t - (f == 0 ? 0 : (f == 1 ? tot0 : tot0 + tot1));
        const int32_t* t0 = t0s[3 * st + f];
        int lo = 0, hi = G;  // t0[lo] <= local < t0[hi]
        while (hi - lo > 1) {
          const int mid = (lo + hi) >> 1;
          if (t0[mid] <= local)
            lo = mid;
          else
            hi = mid;
        }
        tile_group[st * tile_cap + t] = lo;
      }
    }
    // The drained queues are empty again, in both halves of the depth
    // ping-pong: whichever half the next append reads starts from zero (so a
    // captured drain step replays correctly whatever the parity of its
    // appends).  Every read of depth above precedes the scans' barriers.
    if (g < E && (only_expert < 0 || g == only_expert)) depth[g] = depth_other[g] = 0;
  }
  const int64_t nk = (int64_t)n_tokens * k;
  for (int64_t i = (int64_t)blockIdx.x * kPlanThreads + tid; i < nk; i += (int64_t)gridDim.x * kPlanThreads) {
    pos[i] = -1;
    posw[i] = 0.f;
  }
}

__global__ __launch_bounds__(256) void gather_kernel(
    const QEntry* __restrict__ q, int64_t q_stride, const int32_t* __restrict__ offsets, int E,
    int64_t N, int n_tokens, int shared, const void* const* __restrict__ tok_row, char* xp,
    int64_t row_bytes, int32_t* __restrict__ row_token, float* __restrict__ row_w,
    int32_t* __restrict__ pos, float* __restrict__ posw, int k, int32_t* __restrict__ err) {
  __shared__ int32_t off_s[kMaxGroups + 1];
  for (int i = threadIdx.x; i <= E; i += blockDim.x) off_s[i] = offsets[i];
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t R = N + (shared ? n_tokens : 0);
  if (r >= R) return;
  if (r < N && r >= off_s[E]) return;  // N only bounds the routed rows
  const uint4* src;
  if (r < N) {
    int lo = 0, hi = E;  // off_s[lo] <= r < off_s[hi]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (off_s[mid] <= r)
        lo = mid;
      else
        hi = mid;
    }
    const QEntry en = q[(int64_t)lo * q_stride + (r - off_s[lo])];
    src = reinterpret_cast<const uint4*>(en.row);
    if (lane == 0) {
      const int tok = en.token_slot & kTokenMask;
      const int slot = (int)((uint32_t)en.token_slot >> kTokenBits);
      row_token[r] = tok;
      row_w[r] = en.w;
      if (pos) {
        const int64_t pi = (int64_t)tok * k + slot;
        const int old = atomicExch(&pos[pi], (int)r);
        posw[pi] = en.w;
        if (old != -1) atomicOr(err, kErrCollision);
      }
    }
  } else {
    src = reinterpret_cast<const uint4*>(tok_row[r - N]);
  }
  // all of a pass's loads are issued before its stores (the source rows are
  // global memory; the stores cannot alias them)
  typedef unsigned v4u __attribute__((ext_vector_type(4)));
  typedef const __attribute__((address_space(1))) v4u* gsrc_t;
  const gsrc_t gsrc = (gsrc_t)src;
  v4u* dst = reinterpret_cast<v4u*>(xp + r * row_bytes);
  const int nchunk = (int)(row_bytes >> 4);
  constexpr int kB = 4;  // 16-byte chunks per lane per pass
  int c0 = 0;
  for (; c0 + 64 * kB <= nchunk; c0 += 64 * kB) {
    // a full pass: every load is issued before the first store
    v4u v[kB];
#pragma unroll
    for (int i = 0; i < kB; ++i) v[i] = gsrc[c0 + lane + 64 * i];
#pragma unroll
    for (int i = 0; i < kB; ++i) dst[c0 + lane + 64 * i] = v[i];
  }
  for (int c = c0 + lane; c < nchunk; c += 64) dst[c] = gsrc[c];  // the row's tail
}

hipError_t launch_plan(int E, int S, int n_tokens, int k, int only_expert, int32_t* depth,
                       int32_t* depth_other, int32_t* counts, int32_t* offsets, GroupDesc* groups,
                       int32_t* tile_totals, const int* nt, int big_bm, int med_bm, int small_bm,
                       int num_cu, int32_t* tile_group, int64_t tile_cap, int32_t* pos, float* posw,
                       hipStream_t s) {
  NT6 n6;
  for (int i = 0; i < 6; ++i) n6.v[i] = nt[i];
  static_assert(kMaxGroups <= kPlanThreads, "one plan thread per group");
  const int64_t nk = (int64_t)n_tokens * k;
  const unsigned nb = (unsigned)std::min<int64_t>(256, std::max<int64_t>(1, (nk + 4 * kPlanThreads - 1) / (4 * kPlanThreads)));
  plan_kernel<<<nb, kPlanThreads, 0, s>>>(E, S, n_tokens, k, only_expert, depth, depth_other, counts, offsets, groups,
                                  tile_totals, n6, big_bm, med_bm, small_bm, num_cu, tile_group, tile_cap,
                                  pos, posw);
  return hipGetLastError();
}

hipError_t launch_gather(const QEntry* q, int64_t q_stride, const int32_t* offsets, int E,
                         int64_t N, int n_tokens, int shared, const void* const* tok_row,
                         char* xp, int64_t row_bytes, int32_t* row_token, float* row_w,
                         int32_t* pos, float* posw, int k, int32_t* err, hipStream_t s) {
  const int64_t R = N + (shared ? n_tokens : 0);
  if (R == 0) return hipSuccess;
  const int64_t nb = (R + 3) / 4;
  gather_kernel<<<(unsigned)nb, 256, 0, s>>>(q, q_stride, offsets, E, N, n_tokens, shared, tok_row,
                                             xp, row_bytes, row_token, row_w, pos, posw, k, err);
  return hipGetLastError();
}

}  // namespace aep
