// Ragged grouped SwiGLU expert FFN (the contraction hot spot of a drained
// layer).  Two persistent launches per batch:
//
//   gate/up:  h[r, c] = silu(x_r . W_gate[c]) * (x_r . W_up[c])   (K = d)
//   down:     y[r, c] = h_r . W_down[c]                            (K = f)
//
// Every group (expert) contributes ceil(n_g / BM) row tiles x (columns / BN)
// column tiles; the plan kernel laid the tiles of all groups end to end, so
// one launch covers a whole skewed batch, from a 1-row expert to the hottest
// one.  Within a group, consecutive tile ids walk the row tiles of one weight
// column panel, so workgroups running at the same time share that panel.  The
// workgroup -> tile map is XCD aware: hardware dispatches workgroups round
// robin over the 8 XCDs, so workgroup w works on slot (w % 8) * (grid / 8) +
// w / 8, giving each XCD (and its L2) a contiguous run of tiles.
//
// bf16 / fp8-weight path: 256 x 256 output tile per 256-thread workgroup,
// K step 64, four waves each owning a 128 x 128 quadrant computed with
// v_mfma_f32_32x32x16_bf16 (f32 accumulate).  Tiles are staged in LDS with a
// 16-byte row pad (144-byte rows) so the 16-byte fragment reads of 8
// consecutive rows hit distinct banks; the next K step's global loads are in
// flight while the current one is multiplied.  Gate/up tiles hold 128
// features of W_gate and the same 128 of W_up, interleaved per wave quadrant
// (64 gate rows then 64 up rows), so each lane finds the gate and up
// accumulator of the same (row, feature) in its own registers and applies the
// SiLU-and-multiply epilogue without any exchange.  fp8 (OCP e4m3fn) weights
// are widened to bf16 exactly while being staged into LDS; the per-channel
// scale multiplies the f32 accumulator in the epilogue.
//
// f32 path (f32 activations and weights): 64 x 64 tiles, 4 x 4 outputs per
// thread with FMA, for the fp32 workload.
#include "aep_device.h"
#include "aep_internal.h"

namespace aep {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

struct FfnParams {
  const GroupDesc* groups;
  const WeightDesc* wtab;
  const int32_t* tile_totals;
  const void* a;  // x_perm (gate/up) or h (down)
  void* out;      // h (gate/up) or y (down)
  int G;
  int K;      // reduction length: d (gate/up) or f (down)
  int n_out;  // output columns: f (gate/up) or d (down)
};

constexpr int kLds = kBK + 8;  // LDS row stride in bf16 elements (144 bytes)

// 16-byte load through a global (address space 1) pointer, so the compiler
// emits global_load_dwordx4 rather than a flat load.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(1))) u32x4_t* gptr_u4;
__device__ __forceinline__ uint4 gload16(const void* p) {
  const u32x4_t v = *(gptr_u4)(p);
  uint4 o;
  o.x = v.x;
  o.y = v.y;
  o.z = v.z;
  o.w = v.w;
  return o;
}

// Accumulator layout of v_mfma_f32_32x32x16_bf16: lane l, register r holds
// column l % 32 and row 8 * (r / 4) + 4 * (l / 32) + r % 4.
__device__ __forceinline__ int c_row(int lane, int r) {
  return ((r >> 2) << 3) + ((lane >> 5) << 2) + (r & 3);
}

__device__ __forceinline__ int find_group(const int32_t* t0s, int G, int tile) {
  int lo = 0, hi = G;  // t0s[lo] <= tile < t0s[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (t0s[mid] <= tile)
      lo = mid;
    else
      hi = mid;
  }
  return lo;
}

__device__ __forceinline__ uint4 widen_fp8_lo(uint4 v) {  // bytes 0..7 -> 8 bf16
  uint4 o;
  o.x = e4m3_to_bf16_bits(v.x & 0xff) | (e4m3_to_bf16_bits((v.x >> 8) & 0xff) << 16);
  o.y = e4m3_to_bf16_bits((v.x >> 16) & 0xff) | (e4m3_to_bf16_bits(v.x >> 24) << 16);
  o.z = e4m3_to_bf16_bits(v.y & 0xff) | (e4m3_to_bf16_bits((v.y >> 8) & 0xff) << 16);
  o.w = e4m3_to_bf16_bits((v.y >> 16) & 0xff) | (e4m3_to_bf16_bits(v.y >> 24) << 16);
  return o;
}

constexpr int kStage = (kBM + kBN) * kLds;  // bf16 elements per LDS stage (A tile then B tile)
constexpr int kEpiLd = 128 + 8;             // epilogue staging row stride (bf16), 272 bytes

template <bool GATED, bool FP8>
__global__ __launch_bounds__(256, 1) void ffn_mfma_kernel(const FfnParams p) {
  // Two LDS stages (double buffer) of A and B tiles; reused to stage the
  // output tile for 16-byte coalesced stores.
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * kStage];
  __shared__ int32_t t0s[kMaxGroups + 1];

  constexpr int kBChunks = FP8 ? 4 : 8;  // 16-byte global chunks of B per thread per K step
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int G = p.G;
  const int total = p.tile_totals[GATED ? 0 : 1];
  for (int g = tid; g < G; g += 256) t0s[g] = GATED ? p.groups[g].tile0_gu : p.groups[g].tile0_dn;
  if (tid == 0) t0s[G] = total;
  __syncthreads();

  const int nwg = gridDim.x;
  const int slot = (blockIdx.x & 7) * (nwg >> 3) + (blockIdx.x >> 3);
  const int K = p.K, KT = K / kBK, n_out = p.n_out;
  const uint16_t* A = reinterpret_cast<const uint16_t*>(p.a);
  uint16_t* O = reinterpret_cast<uint16_t*>(p.out);

  for (int tile = slot; tile < total; tile += nwg) {
    const int g = find_group(t0s, G, tile);
    const GroupDesc gd = p.groups[g];
    const WeightDesc wd = p.wtab[g];
    const int local = tile - t0s[g];
    const int nti = local / gd.mt;
    const int m0 = (local - nti * gd.mt) * kBM;
    const int arow0 = GATED ? gd.x_row0 : gd.y_row0;

    // Global sources of this thread's 16-byte chunks: a uniform 64-bit base
    // per operand plus 32-bit element offsets.  Rows beyond the group and
    // columns beyond the matrix are clamped onto its last row/column, so every
    // load is in bounds; those rows/columns are never stored.
    const uint16_t* abase = A + (int64_t)(arow0 + m0) * K;
    const int alast = gd.n - 1 - m0;
    uint32_t aoff[8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
      aoff[i] = (uint32_t)(min((tid >> 3) + 32 * i, alast) * K + (tid & 7) * 8);
    // B rows of chunk i: bf16 -> tile row (tid >> 3) + 32 i, fp8 -> (tid >> 2) + 64 i.
    // Gate/up tiles: tile rows [128 w, 128 w + 64) are gate features and
    // [128 w + 64, 128 w + 128) the same up features (w = wave column), so
    // the matrix a chunk comes from is fixed by i at compile time.
    const char* bgate = reinterpret_cast<const char*>(GATED ? wd.gate : wd.down);
    const char* bup = reinterpret_cast<const char*>(GATED ? wd.up : wd.down);
    uint32_t boff[kBChunks];
#pragma unroll
    for (int i = 0; i < kBChunks; ++i) {
      int c;
      if (GATED)
        c = FP8 ? nti * (kBN / 2) + (i >> 1) * 64 + (tid >> 2)
                : nti * (kBN / 2) + (i >> 2) * 64 + (i & 1) * 32 + (tid >> 3);
      else
        c = FP8 ? nti * kBN + 64 * i + (tid >> 2) : nti * kBN + 32 * i + (tid >> 3);
      c = min(c, n_out - 1);
      boff[i] = FP8 ? (uint32_t)(c * K + (tid & 3) * 16) : (uint32_t)(c * K + (tid & 7) * 8);
    }

    uint4 ra[8], rb[kBChunks];
#define AEP_GLOAD(kt)                                                                            \
  do {                                                                                           \
    _Pragma("unroll") for (int i = 0; i < 8; ++i) ra[i] = gload16(abase + aoff[i] + (kt) * kBK); \
    _Pragma("unroll") for (int i = 0; i < kBChunks; ++i) {                                       \
      const bool up_ = GATED && (FP8 ? (i & 1) : ((i >> 1) & 1));                                \
      rb[i] = gload16((up_ ? bup : bgate) + ((size_t)boff[i] + (size_t)(kt) * kBK) * (FP8 ? 1 : 2)); \
    }                                                                                            \
  } while (0)
#define AEP_LSTORE(st)                                                                           \
  do {                                                                                           \
    uint16_t* As_ = smem + (st) * kStage;                                                        \
    uint16_t* Bs_ = As_ + kBM * kLds;                                                            \
    _Pragma("unroll") for (int i = 0; i < 8; ++i)                                                \
        *reinterpret_cast<uint4*>(&As_[((tid >> 3) + 32 * i) * kLds + (tid & 7) * 8]) = ra[i];    \
    if constexpr (FP8) {                                                                         \
      _Pragma("unroll") for (int i = 0; i < kBChunks; ++i) {                                     \
        uint16_t* dst_ = &Bs_[((tid >> 2) + 64 * i) * kLds + (tid & 3) * 16];                    \
        uint4 hi_;                                                                               \
        hi_.x = rb[i].z;                                                                         \
        hi_.y = rb[i].w;                                                                         \
        hi_.z = 0;                                                                               \
        hi_.w = 0;                                                                               \
        *reinterpret_cast<uint4*>(dst_) = widen_fp8_lo(rb[i]);                                   \
        *reinterpret_cast<uint4*>(dst_ + 8) = widen_fp8_lo(hi_);                                 \
      }                                                                                          \
    } else {                                                                                     \
      _Pragma("unroll") for (int i = 0; i < kBChunks; ++i)                                       \
          *reinterpret_cast<uint4*>(&Bs_[((tid >> 3) + 32 * i) * kLds + (tid & 7) * 8]) = rb[i];  \
    }                                                                                            \
  } while (0)

    f32x16_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    AEP_GLOAD(0);
    __syncthreads();  // every wave is done with the previous tile's LDS
    AEP_LSTORE(0);
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
      // Prefetch of step kt + 1 (the last step reloads itself: the loads and
      // the LDS store stay unconditional, which keeps them in registers).
      const int kn = min(kt + 1, KT - 1);
      AEP_GLOAD(kn);
      const uint16_t* As = smem + (kt & 1) * kStage;
      const uint16_t* Bs = As + kBM * kLds;
#pragma unroll
      for (int ks = 0; ks < kBK / 16; ++ks) {
        bf16x8_t a[4], b[4];
        const int kof = ks * 16 + (lane >> 5) * 8;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          a[i] = *reinterpret_cast<const bf16x8_t*>(&As[(wm * 128 + i * 32 + (lane & 31)) * kLds + kof]);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          b[j] = *reinterpret_cast<const bf16x8_t*>(&Bs[(wn * 128 + j * 32 + (lane & 31)) * kLds + kof]);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
      }
      // The other stage was last read in step kt - 1, which every wave
      // finished before the barrier that ended that step.
      AEP_LSTORE((kt + 1) & 1);
      __syncthreads();
    }
#undef AEP_GLOAD
#undef AEP_LSTORE

    // Epilogue: stage bf16 results in LDS ([256][128 + 8]), then write
    // 16-byte chunks of whole rows.  Gate/up tiles produce 128 features in
    // one pass; down tiles produce 256 columns in two passes of 128 (column
    // blocks j = 0, 1 then j = 2, 3 of every wave).
    uint16_t* Cs = smem;
    constexpr int kPasses = GATED ? 1 : 2;
#pragma unroll
    for (int pass = 0; pass < kPasses; ++pass) {
      if (pass) __syncthreads();  // previous pass's reads are done
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const int j = GATED ? jj : 2 * pass + jj;
        const int cl = wn * 64 + jj * 32 + (lane & 31);  // column inside the staged 128
        float sg = 1.f, su = 1.f;
        if constexpr (FP8) {
          if constexpr (GATED) {
            const int fc = min(nti * (kBN / 2) + cl, n_out - 1);
            sg = __uint_as_float((uint32_t)wd.s_gu[fc] << 16);
            su = __uint_as_float((uint32_t)wd.s_gu[n_out + fc] << 16);
          } else {
            const int cc = min(nti * kBN + wn * 128 + j * 32 + (lane & 31), n_out - 1);
            sg = __uint_as_float((uint32_t)wd.s_down[cc] << 16);
          }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int rl = wm * 128 + i * 32 + c_row(lane, r);
            float v;
            if constexpr (GATED) {
              const float gv = acc[i][j][r] * sg;
              const float uv = acc[i][j + 2][r] * su;
              v = gv / (1.f + __expf(-gv)) * uv;
            } else {
              v = acc[i][j][r] * sg;
            }
            Cs[rl * kEpiLd + cl] = (uint16_t)f32_to_bf16_rne(v);
          }
        }
      }
      __syncthreads();
      // 256 rows x 16 chunks of 8 columns; chunk c < 8 is wave column 0's
      // block, c >= 8 wave column 1's.
#pragma unroll 4
      for (int it = 0; it < 16; ++it) {
        const int q = tid + 256 * it;
        const int rl = q >> 4, c16 = q & 15;
        const int row = m0 + rl;
        int col;
        if (GATED)
          col = nti * (kBN / 2) + c16 * 8;
        else
          col = nti * kBN + (c16 >> 3) * 128 + pass * 64 + (c16 & 7) * 8;
        if (row < gd.n && col < n_out) {
          const uint4 v = *reinterpret_cast<const uint4*>(&Cs[rl * kEpiLd + c16 * 8]);
          *reinterpret_cast<uint4*>(O + (int64_t)(gd.y_row0 + row) * n_out + col) = v;
        }
      }
    }
  }
}

// ---------------------------------------------------------------- f32 path
template <bool GATED>
__global__ __launch_bounds__(256) void ffn_f32_kernel(const FfnParams p) {
  constexpr int BM = kBM32, BN = kBN32, BK = 16, LD = BN + 4;
  __shared__ __attribute__((aligned(16))) float As[BK][LD];
  __shared__ __attribute__((aligned(16))) float Bg[BK][LD];
  __shared__ __attribute__((aligned(16))) float Bu[GATED ? BK : 1][LD];
  __shared__ int32_t t0s[kMaxGroups + 1];
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  const int G = p.G;
  const int total = p.tile_totals[GATED ? 0 : 1];
  for (int g = tid; g < G; g += 256) t0s[g] = GATED ? p.groups[g].tile0_gu : p.groups[g].tile0_dn;
  if (tid == 0) t0s[G] = total;
  __syncthreads();
  const int K = p.K, n_out = p.n_out;
  const float* A = reinterpret_cast<const float*>(p.a);
  float* O = reinterpret_cast<float*>(p.out);

  for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
    const int g = find_group(t0s, G, tile);
    const GroupDesc gd = p.groups[g];
    const WeightDesc wd = p.wtab[g];
    const int local = tile - t0s[g];
    const int nti = local / gd.mt;
    const int m0 = (local - nti * gd.mt) * BM;
    const int arow0 = GATED ? gd.x_row0 : gd.y_row0;
    const int lr = tid >> 2, lk = (tid & 3) * 4;
    const float* asrc = A + (int64_t)(arow0 + min(m0 + lr, gd.n - 1)) * K + lk;
    const int bc = min(nti * BN + lr, n_out - 1);
    const float* gsrc = reinterpret_cast<const float*>(GATED ? wd.gate : wd.down) + (int64_t)bc * K + lk;
    const float* usrc = GATED ? reinterpret_cast<const float*>(wd.up) + (int64_t)bc * K + lk : nullptr;

    float ag[4][4], au[4][4];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int c = 0; c < 4; ++c) ag[r][c] = au[r][c] = 0.f;

    for (int k0 = 0; k0 < K; k0 += BK) {
      const float4 va = *reinterpret_cast<const float4*>(asrc + k0);
      const float4 vg = *reinterpret_cast<const float4*>(gsrc + k0);
      As[lk + 0][lr] = va.x;
      As[lk + 1][lr] = va.y;
      As[lk + 2][lr] = va.z;
      As[lk + 3][lr] = va.w;
      Bg[lk + 0][lr] = vg.x;
      Bg[lk + 1][lr] = vg.y;
      Bg[lk + 2][lr] = vg.z;
      Bg[lk + 3][lr] = vg.w;
      if constexpr (GATED) {
        const float4 vu = *reinterpret_cast<const float4*>(usrc + k0);
        Bu[lk + 0][lr] = vu.x;
        Bu[lk + 1][lr] = vu.y;
        Bu[lk + 2][lr] = vu.z;
        Bu[lk + 3][lr] = vu.w;
      }
      __syncthreads();
#pragma unroll
      for (int kk = 0; kk < BK; ++kk) {
        const float4 a = *reinterpret_cast<const float4*>(&As[kk][ty * 4]);
        const float4 b = *reinterpret_cast<const float4*>(&Bg[kk][tx * 4]);
        const float av[4] = {a.x, a.y, a.z, a.w}, bv[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int c = 0; c < 4; ++c) ag[r][c] = fmaf(av[r], bv[c], ag[r][c]);
        if constexpr (GATED) {
          const float4 u = *reinterpret_cast<const float4*>(&Bu[kk][tx * 4]);
          const float uv[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
          for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int c = 0; c < 4; ++c) au[r][c] = fmaf(av[r], uv[c], au[r][c]);
        }
      }
      __syncthreads();
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = m0 + ty * 4 + r;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int col = nti * BN + tx * 4 + c;
        if (row < gd.n && col < n_out) {
          float v = ag[r][c];
          if constexpr (GATED) v = v / (1.f + expf(-v)) * au[r][c];
          O[(int64_t)(gd.y_row0 + row) * n_out + col] = v;
        }
      }
    }
  }
}

static int grid_for(int max_tiles, int cap) {
  int g = max_tiles < cap ? max_tiles : cap;
  g = (g + 7) & ~7;  // the XCD slot map needs a multiple of 8
  return g < 8 ? 8 : g;
}

hipError_t launch_ffn(int stage, int act_dtype, int w_dtype, const GroupDesc* groups,
                      const WeightDesc* wtab, int G, const int32_t* tile_totals, int max_tiles,
                      const void* xp, void* h, void* y, int d, int f, int num_cu, hipStream_t s) {
  if (max_tiles <= 0) return hipSuccess;
  const FfnParams p = stage == 0 ? FfnParams{groups, wtab, tile_totals, xp, h, G, d, f}
                                 : FfnParams{groups, wtab, tile_totals, h, y, G, f, d};
  if (act_dtype == 0) {
    const int grid = grid_for(max_tiles, 4 * num_cu);
    if (stage == 0)
      ffn_f32_kernel<true><<<grid, 256, 0, s>>>(p);
    else
      ffn_f32_kernel<false><<<grid, 256, 0, s>>>(p);
    return hipGetLastError();
  }
  const int grid = grid_for(max_tiles, num_cu);  // one 256-thread workgroup per CU (LDS, registers)
  if (w_dtype == 2) {
    if (stage == 0)
      ffn_mfma_kernel<true, true><<<grid, 256, 0, s>>>(p);
    else
      ffn_mfma_kernel<false, true><<<grid, 256, 0, s>>>(p);
  } else {
    if (stage == 0)
      ffn_mfma_kernel<true, false><<<grid, 256, 0, s>>>(p);
    else
      ffn_mfma_kernel<false, false><<<grid, 256, 0, s>>>(p);
  }
  return hipGetLastError();
}

}  // namespace aep
