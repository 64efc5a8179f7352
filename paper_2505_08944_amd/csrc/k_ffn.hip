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

// Tile order inside one group's nrow x ncol grid of big tiles: panels of
// kPanel column tiles, row tiles one after another inside a panel, the
// columns of a row tile adjacent.  The persistent grids hand each XCD runs of
// consecutive tile ids (32 for 256 workgroups), so an XCD works on a 4 x 8
// block of tiles: per K step its L2 sees 4 row bands of A and 8 column bands
// of B instead of every row band of the group against one column band.
constexpr int kPanel = 8;
__device__ __forceinline__ void panel_decode(int local, int nrow, int ncol, int& rt, int& ct) {
  const int per = kPanel * nrow;
  const int pi = local / per;
  const int within = local - pi * per;
  const int w = min(kPanel, ncol - pi * kPanel);  // the last panel may be narrower
  rt = within / w;
  ct = pi * kPanel + (within - rt * w);
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

// 16 fp8 codes -> 16 bf16 (two 16-byte chunks, lowest k first)
__device__ __forceinline__ void widen_fp8(uint4 v, uint4& lo, uint4& hi) {
  const uint2 a = e4m3x4_to_bf16x4(v.x), b = e4m3x4_to_bf16x4(v.y);
  const uint2 c = e4m3x4_to_bf16x4(v.z), d = e4m3x4_to_bf16x4(v.w);
  lo = make_uint4(a.x, a.y, b.x, b.y);
  hi = make_uint4(c.x, c.y, d.x, d.y);
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
  const int total = p.tile_totals[GATED ? 0 : 2];
  for (int g = tid; g < G; g += 256) t0s[g] = p.groups[g].t0[GATED ? 0 : 2];
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
    int rt, nti;
    panel_decode(local, gd.nbig, GATED ? (n_out + kBN / 2 - 1) / (kBN / 2) : (n_out + kBN - 1) / kBN, rt,
                 nti);
    const int m0 = rt * kBM;
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

    // Two register sets of global-load staging: the loads of step kt + 2
    // are issued at the start of step kt, so every load has a full K step to
    // arrive before its data is written to LDS during step kt + 1.
    uint4 ra0[8], rb0[kBChunks], ra1[8], rb1[kBChunks];
#define AEP_GLOAD(RA, RB, kt)                                                                    \
  do {                                                                                           \
    _Pragma("unroll") for (int i = 0; i < 8; ++i) RA[i] = gload16(abase + aoff[i] + (kt) * kBK); \
    _Pragma("unroll") for (int i = 0; i < kBChunks; ++i) {                                       \
      const bool up_ = GATED && (FP8 ? (i & 1) : ((i >> 1) & 1));                                \
      RB[i] = gload16((up_ ? bup : bgate) + ((size_t)boff[i] + (size_t)(kt) * kBK) * (FP8 ? 1 : 2)); \
    }                                                                                            \
  } while (0)
#define AEP_LSTORE(RA, RB, st)                                                                   \
  do {                                                                                           \
    uint16_t* As_ = smem + (st) * kStage;                                                        \
    uint16_t* Bs_ = As_ + kBM * kLds;                                                            \
    _Pragma("unroll") for (int i = 0; i < 8; ++i)                                                \
        *reinterpret_cast<uint4*>(&As_[((tid >> 3) + 32 * i) * kLds + (tid & 7) * 8]) = RA[i];    \
    if constexpr (FP8) {                                                                         \
      _Pragma("unroll") for (int i = 0; i < kBChunks; ++i) {                                     \
        uint16_t* dst_ = &Bs_[((tid >> 2) + 64 * i) * kLds + (tid & 3) * 16];                    \
        uint4 lo_, hi_;                                                                          \
        widen_fp8(RB[i], lo_, hi_);                                                              \
        *reinterpret_cast<uint4*>(dst_) = lo_;                                                   \
        *reinterpret_cast<uint4*>(dst_ + 8) = hi_;                                               \
      }                                                                                          \
    } else {                                                                                     \
      _Pragma("unroll") for (int i = 0; i < kBChunks; ++i)                                       \
          *reinterpret_cast<uint4*>(&Bs_[((tid >> 3) + 32 * i) * kLds + (tid & 7) * 8]) = RB[i];  \
    }                                                                                            \
  } while (0)
  constexpr int kStores = 8 + (FP8 ? 2 * kBChunks : kBChunks);  // LDS writes per thread per step

    f32x16_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

#define AEP_READ(Abuf, ks_, A_, B_)                                                              \
  do {                                                                                           \
    const uint16_t* As_ = (Abuf);                                                                \
    const uint16_t* Bs_ = As_ + kBM * kLds;                                                      \
    const int kof_ = (ks_) * 16 + (lane >> 5) * 8;                                               \
    _Pragma("unroll") for (int i = 0; i < 4; ++i) A_[i] =                                        \
        *reinterpret_cast<const bf16x8_t*>(&As_[(wm * 128 + i * 32 + (lane & 31)) * kLds + kof_]); \
    _Pragma("unroll") for (int j = 0; j < 4; ++j) B_[j] =                                        \
        *reinterpret_cast<const bf16x8_t*>(&Bs_[(wn * 128 + j * 32 + (lane & 31)) * kLds + kof_]); \
  } while (0)
#define AEP_MMA(A_, B_)                                                                          \
  do {                                                                                           \
    _Pragma("unroll") for (int i = 0; i < 4; ++i) _Pragma("unroll") for (int j = 0; j < 4; ++j)  \
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A_[i], B_[j], acc[i][j], 0, 0, 0);   \
  } while (0)
// One software-pipeline group: read the operands of the next 16-wide k slice
// (8 LDS reads) while the 16 MFMAs of the current slice run.  Reads are
// spread two per four MFMAs: bunching them costs MFMA issue slots (measured
// on gfx950: 8 reads then 16 MFMAs runs ~10% slower than 2 : 4).
#define AEP_GROUP(Abuf, ks_, An, Bn, Ac, Bc)                                                     \
  do {                                                                                           \
    AEP_READ(Abuf, ks_, An, Bn);                                                                 \
    AEP_MMA(Ac, Bc);                                                                             \
    _Pragma("unroll") for (int q_ = 0; q_ < 4; ++q_) {                                           \
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);                                         \
      __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);                                         \
    }                                                                                            \
    __builtin_amdgcn_sched_barrier(0);                                                           \
  } while (0)
// The same, with the global loads of step kt + 2 spread between the MFMAs.
#define AEP_GROUP_LD(Abuf, ks_, An, Bn, Ac, Bc, RA, RB, kl)                                      \
  do {                                                                                           \
    AEP_GLOAD(RA, RB, kl);                                                                       \
    AEP_READ(Abuf, ks_, An, Bn);                                                                 \
    AEP_MMA(Ac, Bc);                                                                             \
    _Pragma("unroll") for (int q_ = 0; q_ < 4; ++q_) {                                           \
      __builtin_amdgcn_sched_group_barrier(0x020, (8 + kBChunks) / 4, 0);                        \
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);                                         \
      __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);                                         \
    }                                                                                            \
    __builtin_amdgcn_sched_barrier(0);                                                           \
  } while (0)
// The same, with the LDS writes of the next step's tile spread between the MFMAs.
#define AEP_GROUP_ST(Abuf, ks_, An, Bn, Ac, Bc, RA, RB, st)                                      \
  do {                                                                                           \
    AEP_READ(Abuf, ks_, An, Bn);                                                                 \
    AEP_LSTORE(RA, RB, st);                                                                      \
    AEP_MMA(Ac, Bc);                                                                             \
    _Pragma("unroll") for (int q_ = 0; q_ < 4; ++q_) {                                           \
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);                                         \
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                                         \
      __builtin_amdgcn_sched_group_barrier(0x200, kStores / 16, 0);                              \
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                                         \
      __builtin_amdgcn_sched_group_barrier(0x200, kStores / 16, 0);                              \
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                                         \
      __builtin_amdgcn_sched_group_barrier(0x200, kStores / 16, 0);                              \
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                                         \
      __builtin_amdgcn_sched_group_barrier(0x200, kStores / 16, 0);                              \
    }                                                                                            \
    __builtin_amdgcn_sched_barrier(0);                                                           \
  } while (0)
// One K step (64 deep = four 16-wide slices) over LDS stage kt & 1:
//   issue the global loads of step kt + 2; slice 0 runs while slice 1 is
//   read; slice 1 runs while slice 2 is read and the tile of step kt + 1
//   (loaded during step kt - 1) is written to the other LDS stage; slice 2
//   runs while slice 3 is read; barrier; slice 3 runs while slice 0 of the
//   next stage is read.  The other stage was last read during step kt - 1,
//   before that step's barrier.  Past the last step, loads and stores repeat
//   the last step's data (kept unconditional so they stay in registers).
#define AEP_STEP(kt_, RLa, RLb, RSa, RSb)                                                        \
  do {                                                                                           \
    const uint16_t* cur_ = smem + ((kt_) & 1) * kStage;                                          \
    const uint16_t* nxt_ = smem + (((kt_) + 1) & 1) * kStage;                                    \
    AEP_GROUP_LD(cur_, 1, a1, b1, a0, b0, RLa, RLb, min((kt_) + 2, KT - 1));                     \
    AEP_GROUP_ST(cur_, 2, a0, b0, a1, b1, RSa, RSb, ((kt_) + 1) & 1);                            \
    AEP_GROUP(cur_, 3, a1, b1, a0, b0);                                                          \
    __syncthreads();                                                                             \
    AEP_GROUP(nxt_, 0, a0, b0, a1, b1);                                                          \
  } while (0)

    bf16x8_t a0[4], b0[4], a1[4], b1[4];
    AEP_GLOAD(ra0, rb0, 0);
    AEP_GLOAD(ra1, rb1, min(1, KT - 1));
    __syncthreads();  // every wave is done with the previous tile's LDS
    AEP_LSTORE(ra0, rb0, 0);
    __syncthreads();
    AEP_READ(smem, 0, a0, b0);
    int kt = 0;
    for (; kt + 1 < KT; kt += 2) {
      AEP_STEP(kt, ra0, rb0, ra1, rb1);
      AEP_STEP(kt + 1, ra1, rb1, ra0, rb0);
    }
    if (kt < KT) AEP_STEP(kt, ra0, rb0, ra1, rb1);
#undef AEP_STEP
#undef AEP_GROUP_ST
#undef AEP_GROUP_LD
#undef AEP_GROUP
#undef AEP_MMA
#undef AEP_READ
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
              v = __fdividef(gv, 1.f + __expf(-gv)) * uv;
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

// ------------------------------------------------- bf16 weights: direct-to-LDS
// The same 256 x 256 tiles and quadrant MFMA work, but tiles move from global
// memory straight into LDS (global_load_lds_dwordx4: 64 lanes x 16 bytes into
// 1 KB of consecutive LDS, no staging registers), through a ring of STAGES
// LDS buffers with a prefetch distance of STAGES - 1 K steps of BKS.  LDS
// rows are not padded; a 16-byte chunk c of tile row r sits at position
// c ^ s(r), where s spreads the 8 rows read together by one fragment read
// over distinct banks (s(r) = r % 8 for 128-byte rows, (r / 2) % 4 for
// 64-byte rows).  Each lane picks the global chunk that belongs at its fixed
// LDS position, so the swizzle costs nothing at load time.
typedef __attribute__((address_space(3))) void* lds_vptr;
typedef const __attribute__((address_space(1))) void* glb_vptr;

// One direct global -> LDS load: 64 lanes x 16 bytes to lds_addr + 16 * lane.
// Issued through inline asm so that the compiler does not see an LDS write
// it cannot disambiguate (it would otherwise wait for every outstanding load
// before each LDS read); the kernel orders these loads itself with
// wait_vmcnt + barriers.  M0 holds the LDS destination.
__device__ __forceinline__ void dload16(const void* gptr, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(gptr),
               "s"(__builtin_amdgcn_readfirstlane(lds_addr))
               : "memory", "m0");
}

// s_waitcnt with only vmcnt constrained (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xf) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
}

// One output tile of BM rows x BN columns (gate/up: BN/2 features of gate and
// the same BN/2 of up) at row m0 of group gd, column tile nti.  Four waves in
// a 2 x 2 grid, each owning a (BM/2) x (BN/2) block of 32 x 32 MFMA
// fragments.  STAGES LDS buffers of (BM + BN) x 128 bytes form the ring
// (prefetch distance STAGES - 1 K steps of 64).
template <bool GATED, int BM, int BN, int STAGES>
__device__ __forceinline__ void dl_tile(const FfnParams& p, unsigned char* smem, uint32_t lds_base,
                                        const GroupDesc& gd, const WeightDesc& wd, int nti, int m0) {
  constexpr int BKS = kBK;
  constexpr int kRowB = BKS * 2;              // 128 bytes: one tile row of one K step
  constexpr int TM = BM / 2, TN = BN / 2;     // wave tile
  constexpr int MI = TM / 32, NI = TN / 32;   // 32 x 32 fragments per wave
  constexpr int kNA = BM / 8 / 4;             // direct loads per wave per K step: A (8 rows each)
  constexpr int kNB = BN / 8 / 4;             // ... and B
  constexpr int kTileA = BM * kRowB, kStageB = (BM + BN) * kRowB;
  constexpr int kDist = STAGES - 1;
  constexpr int kPerStep = kNA + kNB;
  constexpr int kLd = BN / 2 + 8;             // epilogue staging row stride (bf16)
  static_assert(MI >= 1 && NI >= 2 && NI % 2 == 0, "wave tile");
  static_assert(STAGES * kStageB <= 2 * (kBM + kBN) * kRowB, "ring must fit the shared buffer");
  static_assert(BM * kLd * 2 <= 2 * (kBM + kBN) * kRowB, "epilogue staging must fit");

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int K = p.K, KT = K / BKS, n_out = p.n_out;
  const uint16_t* A = reinterpret_cast<const uint16_t*>(p.a);
  uint16_t* O = reinterpret_cast<uint16_t*>(p.out);
  // loader: lane l fills LDS position l % 8 of row l / 8 of an 8-row block with
  // the k chunk that belongs there, (l % 8) ^ (row % 8)
  const int ld_row = lane >> 3;
  const int ld_c = (lane & 7) ^ (lane >> 3);
  // reader: fragment row and its swizzle
  const int rd_row = lane & 31;
  const int rd_s = rd_row & 7;

  const int arow0 = GATED ? gd.x_row0 : gd.y_row0;
  const uint16_t* abase = A + (int64_t)(arow0 + m0) * K;
  const int alast = gd.n - 1 - m0;
  uint32_t aoff[kNA], boff[kNB];
#pragma unroll
  for (int i = 0; i < kNA; ++i) aoff[i] = (uint32_t)(min((wave * kNA + i) * 8 + ld_row, alast) * K + ld_c * 8);
  // B rows: a wave column's TN rows are TN/2 gate features then the same TN/2
  // up features; an 8-row load block never straddles the two halves.
  const uint16_t* bsrc[kNB];
#pragma unroll
  for (int i = 0; i < kNB; ++i) {
    const int br = (wave * kNB + i) * 8 + ld_row;
    int c;
    bool up = false;
    if (GATED) {
      const int within = br % TN;
      up = within >= TN / 2;
      c = nti * (BN / 2) + (br / TN) * (TN / 2) + within % (TN / 2);
    } else {
      c = nti * BN + br;
    }
    c = min(c, n_out - 1);
    boff[i] = (uint32_t)(c * K + ld_c * 8);
    bsrc[i] = reinterpret_cast<const uint16_t*>(GATED ? (up ? wd.up : wd.gate) : wd.down);
  }

#define DL_LOAD(kt_, st_)                                                                        \
  do {                                                                                           \
    const uint32_t sa_ = lds_base + (st_) * kStageB + wave * kNA * 1024;                          \
    const uint32_t sb_ = lds_base + (st_) * kStageB + kTileA + wave * kNB * 1024;                 \
    _Pragma("unroll") for (int i = 0; i < kNA; ++i)                                              \
        dload16(abase + aoff[i] + (kt_) * BKS, sa_ + i * 1024);                                  \
    _Pragma("unroll") for (int i = 0; i < kNB; ++i)                                              \
        dload16(bsrc[i] + boff[i] + (kt_) * BKS, sb_ + i * 1024);                                \
  } while (0)
#define DL_READ(st_, ks_, A_, B_)                                                                \
  do {                                                                                           \
    const unsigned char* ab_ = smem + (st_) * kStageB;                                           \
    const int ro_ = rd_row * kRowB + (((2 * (ks_) + (lane >> 5)) ^ rd_s) << 4);                  \
    _Pragma("unroll") for (int i = 0; i < MI; ++i) A_[i] =                                       \
        *reinterpret_cast<const bf16x8_t*>(ab_ + (wm * TM + i * 32) * kRowB + ro_);              \
    _Pragma("unroll") for (int j = 0; j < NI; ++j) B_[j] =                                       \
        *reinterpret_cast<const bf16x8_t*>(ab_ + kTileA + (wn * TN + j * 32) * kRowB + ro_);     \
  } while (0)
#define DL_MMA(A_, B_)                                                                           \
  do {                                                                                           \
    _Pragma("unroll") for (int i = 0; i < MI; ++i) _Pragma("unroll") for (int j = 0; j < NI; ++j) \
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A_[i], B_[j], acc[i][j], 0, 0, 0);   \
  } while (0)
  // operand reads spread between the MFMAs
  constexpr int kQ = MI * NI >= 4 ? 4 : MI * NI;
#define DL_GROUP(st_, ks_, An, Bn, Ac, Bc)                                                       \
  do {                                                                                           \
    DL_READ(st_, ks_, An, Bn);                                                                   \
    DL_MMA(Ac, Bc);                                                                              \
    _Pragma("unroll") for (int q_ = 0; q_ < kQ; ++q_) {                                          \
      __builtin_amdgcn_sched_group_barrier(0x100, (MI + NI + kQ - 1) / kQ, 0);                   \
      __builtin_amdgcn_sched_group_barrier(0x008, MI * NI / kQ, 0);                              \
    }                                                                                            \
    __builtin_amdgcn_sched_barrier(0);                                                           \
  } while (0)

  f32x16_t acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  bf16x8_t a0[MI], b0[NI], a1[MI], b1[NI];
  // Nothing of this wave may still be in flight when the ring is refilled
  // (the wait counter is in issue order, so earlier stores of the previous
  // tile's epilogue would otherwise blur the counts below).
  wait_vmcnt<0>();
  __syncthreads();  // every wave is done with the previous tile's LDS
#pragma unroll
  for (int s = 0; s < kDist; ++s) DL_LOAD(min(s, KT - 1), s);
  wait_vmcnt<(kDist - 1) * kPerStep>();  // step 0 has landed (this wave's part)
  __syncthreads();                       // ... and every wave's part
  DL_READ(0, 0, a0, b0);
  // Step kt computes stage kt % STAGES and refills the stage read in step
  // kt - 1 (every wave passed that step's barrier) with step kt + kDist.
  // Past the last step the loads repeat the last step (never read).
  int st = 0;
  for (int kt = 0; kt < KT; ++kt) {
    const int nst = st + 1 == STAGES ? 0 : st + 1;
    const int fst = st + kDist >= STAGES ? st + kDist - STAGES : st + kDist;
    DL_LOAD(min(kt + kDist, KT - 1), fst);
    __builtin_amdgcn_sched_barrier(0);
    DL_GROUP(st, 1, a1, b1, a0, b0);
    DL_GROUP(st, 2, a0, b0, a1, b1);
    DL_GROUP(st, 3, a1, b1, a0, b0);
    wait_vmcnt<(kDist - 1) * kPerStep>();  // step kt + 1 has landed
    __syncthreads();
    DL_GROUP(nst, 0, a0, b0, a1, b1);
    st = nst;
  }
#undef DL_GROUP
#undef DL_MMA
#undef DL_READ
#undef DL_LOAD

  // Epilogue: stage bf16 results in LDS ([BM][BN/2 + 8]) and write 16-byte
  // chunks of whole rows.  Gate/up: one pass, feature fragment j pairs with
  // up fragment j + NI/2.  Down: two passes of BN/2 columns (each wave
  // contributes column fragments pass * NI/2 .. pass * NI/2 + NI/2 - 1).
  // The loads issued past the last step target the ring this reuses: let
  // them land first.
  wait_vmcnt<0>();
  uint16_t* Cs = reinterpret_cast<uint16_t*>(smem);
  constexpr int kPasses = GATED ? 1 : 2;
  constexpr int kChunks = BN / 16;  // 16-byte chunks per staged row
#pragma unroll
  for (int pass = 0; pass < kPasses; ++pass) {
    __syncthreads();  // LDS reads of the K loop / previous pass are done
#pragma unroll
    for (int jj = 0; jj < NI / 2; ++jj) {
      const int j = GATED ? jj : pass * (NI / 2) + jj;
      const int cl = wn * (TN / 2) + jj * 32 + (lane & 31);
#pragma unroll
      for (int i = 0; i < MI; ++i) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int rl = wm * TM + i * 32 + c_row(lane, r);
          float v;
          if constexpr (GATED) {
            const float gv = acc[i][j][r];
            v = __fdividef(gv, 1.f + __expf(-gv)) * acc[i][j + NI / 2][r];
          } else {
            v = acc[i][j][r];
          }
          Cs[rl * kLd + cl] = (uint16_t)f32_to_bf16_rne(v);
        }
      }
    }
    __syncthreads();
#pragma unroll 4
    for (int it = 0; it < BM * kChunks / 256; ++it) {
      const int q = tid + 256 * it;
      const int rl = q / kChunks, cc = q % kChunks;
      const int row = m0 + rl;
      const int sc = cc * 8;  // staged column
      const int col = GATED ? nti * (BN / 2) + sc
                            : nti * BN + (sc / (TN / 2)) * TN + pass * (TN / 2) + sc % (TN / 2);
      if (row < gd.n && col < n_out) {
        const uint4 v = *reinterpret_cast<const uint4*>(&Cs[rl * kLd + sc]);
        *reinterpret_cast<uint4*>(O + (int64_t)(gd.y_row0 + row) * n_out + col) = v;
      }
    }
  }
}

// bf16-weight FFN launch: every tile of the big family (256 rows), then every
// tile of the small family (64 rows: cold experts and the ragged tails of hot
// ones), in one persistent grid.  Small tiles come last, so they also fill
// the tail of the big ones.  Small tiles are 64 rows x 128 columns: cold
// experts are weight-streaming bound, and narrower tiles spread each expert's
// weights over more CUs.
template <bool GATED>
__global__ __launch_bounds__(256, 1) void ffn_dlds_kernel(const FfnParams p) {
  __shared__ __attribute__((aligned(1024))) unsigned char smem[2 * (kBM + kBN) * kBK * 2];
  __shared__ int32_t t0b[kMaxGroups + 1], t0s[kMaxGroups + 1];
  const int tid = threadIdx.x;
  const int G = p.G;
  const int big_total = p.tile_totals[GATED ? 0 : 2];
  const int small_total = p.tile_totals[GATED ? 1 : 3];
  for (int g = tid; g < G; g += 256) {
    t0b[g] = p.groups[g].t0[GATED ? 0 : 2];
    t0s[g] = p.groups[g].t0[GATED ? 1 : 3];
  }
  if (tid == 0) {
    t0b[G] = big_total;
    t0s[G] = small_total;
  }
  __syncthreads();
  const uint32_t lds_base = (uint32_t)(uintptr_t)(lds_vptr)smem;
  const int nwg = gridDim.x;
  const int slot = (blockIdx.x & 7) * (nwg >> 3) + (blockIdx.x >> 3);
  const int ncol_big = GATED ? (p.n_out + kBN / 2 - 1) / (kBN / 2) : (p.n_out + kBN - 1) / kBN;
  for (int tile = slot; tile < big_total + small_total; tile += nwg) {
    if (tile < big_total) {
      const int g = find_group(t0b, G, tile);
      const GroupDesc gd = p.groups[g];
      const int local = tile - t0b[g];
      int rt, nti;
      panel_decode(local, gd.nbig, ncol_big, rt, nti);
      dl_tile<GATED, kBM, kBN, 2>(p, smem, lds_base, gd, p.wtab[g], nti, rt * kBM);
    } else {
      const int t = tile - big_total;
      const int g = find_group(t0s, G, t);
      const GroupDesc gd = p.groups[g];
      const int local = t - t0s[g];
      const int nti = local / gd.nsmall;
      dl_tile<GATED, kSmallBM, kSmallBN, 4>(p, smem, lds_base, gd, p.wtab[g], nti,
                                  gd.small_row0 + (local - nti * gd.nsmall) * kSmallBM);
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
  const int total = p.tile_totals[GATED ? 0 : 2];
  for (int g = tid; g < G; g += 256) t0s[g] = p.groups[g].t0[GATED ? 0 : 2];
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
    const int nti = local / gd.nbig;
    const int m0 = (local - nti * gd.nbig) * BM;
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
      ffn_dlds_kernel<true><<<grid, 256, 0, s>>>(p);
    else
      ffn_dlds_kernel<false><<<grid, 256, 0, s>>>(p);
  }
  return hipGetLastError();
}

}  // namespace aep
