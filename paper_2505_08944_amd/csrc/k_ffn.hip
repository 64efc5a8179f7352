// Ragged grouped SwiGLU expert FFN (the contraction hot spot of a drained
// layer).  Two persistent launches per batch:
//
//   gate/up:  h[r, c] = silu(x_r . W_gate[c]) * (x_r . W_up[c])   (K = d)
//   down:     y[r, c] = h_r . W_down[c]                            (K = f)
//
// The plan kernel laid the tiles of all groups (experts) end to end in three
// row-tile families, split per stage: 256 x 256 tiles for the full 256-row
// blocks of an expert (and for a remainder above 128 rows, unless that would
// start another round of the grid in a short stage), then 128 x 128 medium
// tiles (256 x 128 tall ones for a cold batch's remainders above 128 rows)
// and 64 x 128 small tiles (64 x 256 with fp8 weights) for the ragged row
// tails and cold experts.  One launch covers a whole skewed batch, from a
// 1-row expert to the hottest one:
// every big tile first, then the smaller ones, which also fill the tail of
// the big family.  The workgroup -> tile map is XCD aware: hardware
// dispatches workgroups round robin over the 8 XCDs, so workgroup w works on
// slot (w % 8) * (grid / 8) + w / 8, giving each XCD (and its L2) a
// contiguous run of tiles, and the big tiles of a group are ordered in panels
// of 8 column tiles (4 in the down launch) so that such a run is a compact
// block of row and column tiles.
//
// bf16 / fp8-weight path: 256-thread workgroups, K step 64, four waves each
// owning a quadrant of the tile computed with v_mfma_f32_32x32x16_bf16 (f32
// accumulate).  Tiles move from global memory straight into LDS (no staging
// registers) through a ring of stages; the loads of later K steps are in
// flight while the current one is multiplied, and the refill of a freed
// stage is spread over the MFMAs that follow instead of issued as a block.  Gate/up tiles hold BN/2
// features of W_gate and the same BN/2 of W_up, interleaved per wave quadrant,
// so each lane finds the gate and up accumulator of the same (row, feature)
// in its own registers and applies the SiLU-and-multiply epilogue without any
// exchange.  fp8 (OCP e4m3fn) weights stay fp8 in LDS and are widened to bf16
// exactly when read into MFMA operands; the per-channel scale multiplies the
// f32 accumulator in the epilogue.
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
  const int32_t* tile_group;  // group of each tile of this launch (written by the plan)
  float* split_slots;         // split-K partial sums (nullptr: no split)
  int32_t* split_cnt;         // pieces finished per tile (zero between launches)
  int64_t split_bytes;        // size of split_slots
  const void* a;  // x_perm (gate/up) or h (down)
  void* out;      // h (gate/up) or y (down)
  int G;
  int K;      // reduction length: d (gate/up) or f (down)
  int n_out;  // output columns: f (gate/up) or d (down)
  unsigned long long* clk;  // clock probe (nullptr: off)
  int clk_n;
};

// Accumulator layout of v_mfma_f32_32x32x16_bf16: lane l, register r holds
// column l % 32 and row 8 * (r / 4) + 4 * (l / 32) + r % 4.
__device__ __forceinline__ int c_row(int lane, int r) {
  return ((r >> 2) << 3) + ((lane >> 5) << 2) + (r & 3);
}

// Tile order inside one group's nrow x ncol grid of big tiles: panels of
// PANEL column tiles, row tiles one after another inside a panel, the
// columns of a row tile adjacent.  The persistent grids hand each XCD runs of
// consecutive tile ids (32 for 256 workgroups), so an XCD works on a compact
// block of tiles (4 x 8 for gate/up, 8 x 4 for down): per K step its L2 sees
// a few row bands of A and column bands of B instead of every row band of the
// group against one column band.  Down launches have few column tiles
// (d / 256) and long K; panels of 4 measured 1-4% faster there, panels of 8
// faster for gate/up on single experts.
template <int PANEL>
__device__ __forceinline__ void panel_decode(int local, int nrow, int ncol, int& rt, int& ct) {
  const int per = PANEL * nrow;
  const int pi = local / per;
  const int within = local - pi * per;
  const int w = min(PANEL, ncol - pi * PANEL);  // the last panel may be narrower
  rt = within / w;
  ct = pi * PANEL + (within - rt * w);
}

// ------------------------------------------------- direct-to-LDS MFMA tiles
// Tiles move from global memory straight into LDS (buffer_load_dwordx4 with
// the lds bit: 64 lanes x 16 bytes into 1 KB of consecutive LDS, no staging
// registers),
// through a ring of STAGES LDS buffers with a prefetch distance of
// STAGES - 1 K steps.  LDS rows are not padded; a 16-byte chunk c of tile row r sits at position
// c ^ s(r), where s spreads the 8 rows read together by one fragment read
// over distinct banks (s(r) = r % 8 for 128-byte rows, (r / 2) % 4 for
// 64-byte rows).  Each lane picks the global chunk that belongs at its fixed
// LDS position, so the swizzle costs nothing at load time.
typedef __attribute__((address_space(3))) void* lds_vptr;
typedef const __attribute__((address_space(1))) void* glb_vptr;

// A raw buffer resource over [base, base + bytes): stride 0, 32-bit data
// format, every access bounds-checked against bytes (an access past the end
// reads zeros and writes nothing).  The fields are uniform (SGPRs).
typedef int i32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ i32x4_t make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = (uint64_t)(uintptr_t)base;
  i32x4_t r;
  r.x = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r.y = __builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xFFFFu));
  r.z = __builtin_amdgcn_readfirstlane((int)bytes);
  r.w = 0x00020000;  // data format 32
  return r;
}

// One direct buffer -> LDS load: lane l reads the 16 bytes at byte offset
// voff + soff of the resource and writes them to lds_addr + 16 * l (M0 holds
// lds_addr).  The per-step K offset rides in the scalar soff, so a load costs
// no vector address arithmetic.  Issued through inline asm so that the
// compiler does not see an LDS write it cannot disambiguate (it would
// otherwise wait for every outstanding load before each LDS read); the
// kernel orders these loads itself with wait_vmcnt + barriers.
__device__ __forceinline__ void dload16(i32x4_t rsrc, uint32_t voff, uint32_t soff, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %3\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds" ::"v"(voff), "s"(rsrc),
               "s"(soff), "s"(__builtin_amdgcn_readfirstlane(lds_addr))
               : "memory", "m0");
}

// s_waitcnt with only vmcnt constrained (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xf) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
}

// Wait until at most MUL * per loads are outstanding, per in [LO, HI] (the
// wave's loads per K step; the immediate must be a constant, hence the
// uniform branch ladder).
template <int MUL, int LO, int HI>
__device__ __forceinline__ void wait_steps(int per) {
  if constexpr (MUL == 0 || LO == HI) {
    wait_vmcnt<MUL * LO>();
  } else {
    if (per <= LO)
      wait_vmcnt<MUL * LO>();
    else
      wait_steps<MUL, LO + 1, HI>(per);
  }
}

// One output tile of BM rows x BN columns (gate/up: BN/2 features of gate and
// the same BN/2 of up) at row m0 of group gd, column tile nti.  Four waves in
// a 2 x 2 grid, each owning a (BM/2) x (BN/2) block of 32 x 32 MFMA
// fragments.  STAGES LDS buffers form the ring (prefetch distance STAGES - 1
// K steps of 64); a stage holds the A tile (BM rows x 128 bytes, bf16) and
// the B tile (BN rows x 128 bytes for bf16 weights, x 64 bytes for fp8).
//
// fp8 weights (FP8): B stays e4m3 in LDS.  One 16-byte read gives a lane 16
// consecutive k of its row; lanes 0-31 read k-chunk 2m, lanes 32-63 chunk
// 2m + 1 (K elements 32m .. 32m + 31), and the two halves of the read feed
// two MFMAs after an exact e4m3 -> bf16 conversion.  The A reads follow the
// same assignment of k to lanes (bf16 chunks 4m + 2h and 4m + 2h + 1 for
// lane half h), so every MFMA still pairs equal k; per-channel scales are
// applied in the epilogue.
template <bool GATED, bool FP8, int BM, int BN, int STAGES, int BSTAGES, int CAP>
__device__ __forceinline__ void dl_tile(const FfnParams& p, unsigned char* smem, uint32_t lds_base,
                                        const GroupDesc& gd, const WeightDesc& wd, int nti, int m0,
                                        int rot_seed, int n_split = 1, int piece = 0, float* slot = nullptr,
                                        int32_t* cnt = nullptr) {
  constexpr int BKS = kBK;
  constexpr int kRowA = BKS * 2;              // 128 bytes: one A row of one K step
  constexpr int kRowB = FP8 ? BKS : BKS * 2;  // one B row of one K step
  constexpr int kRplA = 1024 / kRowA;         // rows per direct load (8)
  constexpr int kRplB = 1024 / kRowB;         // 8, or 16 for fp8
  constexpr int kChB = kRowB / 16;            // 16-byte chunks per B row (8 or 4)
  constexpr int TM = BM / 2, TN = BN / 2;     // wave tile
  constexpr int MI = TM / 32, NI = TN / 32;   // 32 x 32 fragments per wave
  constexpr int kNA = BM / kRplA / 4;         // direct loads per wave per K step: A
  constexpr int kNB = BN / kRplB / 4;         // ... and B
  constexpr int kTileA = BM * kRowA, kTileB = BN * kRowB, kStageB = kTileA + kTileB;
  constexpr int kPerStep = kNA + kNB;
  // Ring layout.  One ring (BSTAGES == STAGES): stage s holds A then B at
  // s * kStageB.  Split rings (BSTAGES > STAGES, bf16 big tiles): STAGES A
  // stages first, then BSTAGES B stages, so the weight tiles are prefetched
  // further ahead than the activation tiles.
  constexpr bool kSplit = BSTAGES != STAGES;
  constexpr int kAStride = kSplit ? kTileA : kStageB;
  constexpr int kBBase = kSplit ? STAGES * kTileA : kTileA;
  constexpr int kBStride = kSplit ? kTileB : kStageB;
  static_assert(!kSplit || (!FP8 && STAGES == 2 && BSTAGES == 3), "split rings: bf16, 2 A + 3 B stages");
  constexpr int kLd = BN / 2 + 8;             // epilogue staging row stride (bf16)
  static_assert(MI >= 1 && NI >= 2 && NI % 2 == 0, "wave tile");
  static_assert(kNA >= 1 && kNB >= 1, "loads per wave");
  static_assert(!GATED || kNB * kRplB == TN / 2, "a wave's B rows are all gate or all up rows");
  static_assert(STAGES * kTileA + BSTAGES * kTileB <= CAP, "ring must fit the shared buffer");
  static_assert(BM * kLd * 2 <= CAP, "epilogue staging must fit");
  static_assert((STAGES - 1) * kPerStep < 64, "vmcnt range");

  // The thread index goes through an empty asm so that the per-lane offsets
  // derived from it are computed per tile instead of being hoisted out of the
  // tile loop, where they would stay live across the K loop and be spilled.
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int K = p.K, KT0 = K / BKS, n_out = p.n_out;
  // K steps of this work item: all of them, or piece `piece` of n_split
  // (split-K): steps [k0, k0 + KT).
  const int k0 = piece * KT0 / n_split, KT = (piece + 1) * KT0 / n_split - k0;
  // K rotation: the tile walks its K steps starting at step rot and wrapping
  // round (step j of the loop loads K step krot(j)).  Tiles that run at the
  // same time start at different steps, so their weight streams do not hit
  // the same DRAM channels in lockstep (a load-only probe of the cold-tile
  // pattern: 0.68 -> 0.79 of peak HBM bandwidth).  rot_seed < 0: no rotation.
  const int rot = rot_seed < 0 ? 0 : (int)((7u * (unsigned)rot_seed) % (unsigned)KT);
  auto krot = [&](int j) { return k0 + (j + rot < KT ? j + rot : j + rot - KT); };
  const uint16_t* A = reinterpret_cast<const uint16_t*>(p.a);
  uint16_t* O = reinterpret_cast<uint16_t*>(p.out);
  // chunk swizzles: spread the 8 rows one 128-byte bank window sees over
  // distinct banks (r % 8 for 128-byte rows, (r / 2) % 4 for 64-byte rows)
  auto swz_b = [](int r) { return kChB == 8 ? (r & 7) : ((r >> 1) & 3); };
  // loaders: lane l fills chunk position l % chunks-per-row of row
  // l / chunks-per-row of a load block with the global chunk that belongs
  // there (load blocks start at multiples of 8 or 16 rows)
  const int lda_row = lane >> 3;
  const int lda_c = (lane & 7) ^ lda_row;
  const int ldb_row = lane / kChB;
  const int ldb_c = (lane % kChB) ^ swz_b(ldb_row);
  // readers: fragment row and its swizzle
  const int rd_row = lane & 31;
  const int rd_sa = rd_row & 7;
  const int rd_sb = swz_b(rd_row);

  const int arow0 = GATED ? gd.x_row0 : gd.y_row0;
  const uint16_t* abase = A + (int64_t)(arow0 + m0) * K;
  const int alast = gd.n - 1 - m0;
  // A load blocks of this wave that hold rows of the group: blocks past the
  // group's end are not loaded (their LDS rows hold stale data, their outputs
  // are never stored), which saves the activation traffic of ragged and cold
  // tiles.  Every K step of the tile issues the same number of loads per wave.
  // Big bf16 tiles (two-stage ring) load every block: rows past the end
  // repeat the last row, and the refill carries no per-load branches.
  constexpr bool kAllA = !FP8 && STAGES == 2;
  const int na_eff = kAllA ? kNA : __builtin_amdgcn_readfirstlane(
      max(0, min(kNA, (alast + 1 - wave * kNA * kRplA + kRplA - 1) / kRplA)));
  const int per_step = na_eff + kNB;
  uint32_t aoff[kNA], boff[kNB];  // byte offsets into the two resources
#pragma unroll
  for (int i = 0; i < kNA; ++i)
    aoff[i] = (uint32_t)(min((wave * kNA + i) * kRplA + lda_row, alast) * K + lda_c * 8) * 2u;
  // B rows: a wave column's TN rows are TN/2 gate features then the same TN/2
  // up features; a wave's B rows lie in one of the two halves.
  const unsigned char* bmat;
  {
    const int br0 = wave * kNB * kRplB;
    const bool up = GATED && (br0 % TN) >= TN / 2;
    bmat = reinterpret_cast<const unsigned char*>(GATED ? (up ? wd.up : wd.gate) : wd.down);
  }
  // the group's rows from row m0 on, and the weight matrix (the host bounds
  // both below 4 GiB)
  const i32x4_t rsA = make_rsrc(abase, (uint32_t)(alast + 1) * (uint32_t)K * 2u);
  const i32x4_t rsB = make_rsrc(bmat, (uint32_t)n_out * (uint32_t)K * (FP8 ? 1u : 2u));
#pragma unroll
  for (int i = 0; i < kNB; ++i) {
    const int br = (wave * kNB + i) * kRplB + ldb_row;
    int c = GATED ? nti * (BN / 2) + (br / TN) * (TN / 2) + (br % TN) % (TN / 2) : nti * BN + br;
    c = min(c, n_out - 1);
    boff[i] = (uint32_t)(c * K * (FP8 ? 1 : 2) + ldb_c * 16);
  }

#define DL_LOAD(kt_, st_)                                                                        \
  do {                                                                                           \
    const uint32_t sa_ = lds_base + (st_) * kAStride + wave * kNA * 1024;                         \
    const uint32_t sb_ = lds_base + kBBase + (st_) * kBStride + wave * kNB * 1024;                \
    _Pragma("unroll") for (int i = 0; i < kNA; ++i)                                              \
        if (i < na_eff) dload16(rsA, aoff[i], (kt_) * kRowA, sa_ + i * 1024);                    \
    _Pragma("unroll") for (int i = 0; i < kNB; ++i)                                              \
        dload16(rsB, boff[i], (kt_) * kRowB, sb_ + i * 1024);                                    \
  } while (0)
  // bf16 weights: k-slice ks (16 k) of every fragment
#define DL_READ(sa_, sb_, ks_, A_, B_)                                                           \
  do {                                                                                           \
    const unsigned char* aa_ = smem + (sa_) * kAStride;                                          \
    const unsigned char* bb_ = smem + kBBase + (sb_) * kBStride;                                 \
    const int ro_ = rd_row * kRowA + (((2 * (ks_) + (lane >> 5)) ^ rd_sa) << 4);                 \
    _Pragma("unroll") for (int i = 0; i < MI; ++i) A_[i] =                                       \
        *reinterpret_cast<const bf16x8_t*>(aa_ + (wm * TM + i * 32) * kRowA + ro_);              \
    _Pragma("unroll") for (int j = 0; j < NI; ++j) B_[j] =                                       \
        *reinterpret_cast<const bf16x8_t*>(bb_ + (wn * TN + j * 32) * kRowB + ro_);              \
  } while (0)
  // fp8 weights: half-step m (32 k): A for both MFMAs, raw e4m3 B
#define DL_READ8(st_, m_, A1_, A2_, R_)                                                          \
  do {                                                                                           \
    const unsigned char* ab_ = smem + (st_) * kStageB; /* one ring */                            \
    const int ca_ = 4 * (m_) + 2 * (lane >> 5);                                                  \
    const int ra1_ = rd_row * kRowA + ((ca_ ^ rd_sa) << 4);                                      \
    const int ra2_ = rd_row * kRowA + (((ca_ + 1) ^ rd_sa) << 4);                                \
    const int rb_ = rd_row * kRowB + (((2 * (m_) + (lane >> 5)) ^ rd_sb) << 4);                  \
    _Pragma("unroll") for (int j = 0; j < NI; ++j) R_[j] =                                       \
        *reinterpret_cast<const uint4*>(ab_ + kTileA + (wn * TN + j * 32) * kRowB + rb_);        \
    _Pragma("unroll") for (int i = 0; i < MI; ++i) {                                             \
      A1_[i] = *reinterpret_cast<const bf16x8_t*>(ab_ + (wm * TM + i * 32) * kRowA + ra1_);      \
      A2_[i] = *reinterpret_cast<const bf16x8_t*>(ab_ + (wm * TM + i * 32) * kRowA + ra2_);      \
    }                                                                                            \
  } while (0)
  // e4m3 x 16 -> two bf16 x 8 operands (exact)
#define DL_WIDEN(R_, B1_, B2_)                                                                   \
  do {                                                                                           \
    _Pragma("unroll") for (int j = 0; j < NI; ++j) {                                             \
      const uint2 w0_ = e4m3x4_to_bf16x4(R_[j].x), w1_ = e4m3x4_to_bf16x4(R_[j].y);              \
      const uint2 w2_ = e4m3x4_to_bf16x4(R_[j].z), w3_ = e4m3x4_to_bf16x4(R_[j].w);              \
      B1_[j] = __builtin_bit_cast(bf16x8_t, make_uint4(w0_.x, w0_.y, w1_.x, w1_.y));             \
      B2_[j] = __builtin_bit_cast(bf16x8_t, make_uint4(w2_.x, w2_.y, w3_.x, w3_.y));             \
    }                                                                                            \
  } while (0)
#define DL_MMA(A_, B_)                                                                           \
  do {                                                                                           \
    _Pragma("unroll") for (int i = 0; i < MI; ++i) _Pragma("unroll") for (int j = 0; j < NI; ++j) \
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A_[i], B_[j], acc[i][j], 0, 0, 0);   \
  } while (0)
  // operand reads spread between the MFMAs
  constexpr int kQ = MI * NI >= 4 ? 4 : MI * NI;
#define DL_GROUP(sa_, sb_, ks_, An, Bn, Ac, Bc)                                                  \
  do {                                                                                           \
    DL_READ(sa_, sb_, ks_, An, Bn);                                                              \
    DL_MMA(Ac, Bc);                                                                              \
    _Pragma("unroll") for (int q_ = 0; q_ < kQ; ++q_) {                                          \
      __builtin_amdgcn_sched_group_barrier(0x100, (MI + NI + kQ - 1) / kQ, 0);                   \
      __builtin_amdgcn_sched_group_barrier(0x008, MI * NI / kQ, 0);                              \
    }                                                                                            \
    __builtin_amdgcn_sched_barrier(0);                                                           \
  } while (0)
  // fp8: one operand fragment of half-step m (index < NI: raw B, then A1, A2)
#define DL_READ8_1(st_, m_, A1_, A2_, R_, idx_)                                                  \
  do {                                                                                           \
    const unsigned char* ab_ = smem + (st_) * kStageB;                                           \
    const int ca_ = 4 * (m_) + 2 * (lane >> 5);                                                  \
    if ((idx_) < NI) {                                                                           \
      const int rb_ = rd_row * kRowB + (((2 * (m_) + (lane >> 5)) ^ rd_sb) << 4);                \
      R_[(idx_)] = *reinterpret_cast<const uint4*>(ab_ + kTileA + (wn * TN + (idx_) * 32) * kRowB + rb_); \
    } else if ((idx_) < NI + MI) {                                                               \
      const int ra1_ = rd_row * kRowA + ((ca_ ^ rd_sa) << 4);                                    \
      A1_[(idx_) - NI] = *reinterpret_cast<const bf16x8_t*>(ab_ + (wm * TM + ((idx_) - NI) * 32) * kRowA + ra1_); \
    } else {                                                                                     \
      const int ra2_ = rd_row * kRowA + (((ca_ + 1) ^ rd_sa) << 4);                              \
      A2_[(idx_) - NI - MI] = *reinterpret_cast<const bf16x8_t*>(ab_ + (wm * TM + ((idx_) - NI - MI) * 32) * kRowA + ra2_); \
    }                                                                                            \
  } while (0)
  // fp8: widen the raw B read in the previous group, then read the next
  // half-step while the 2 * MI * NI MFMAs of this one run; the refill is
  // spread over the step's MFMAs as in the deeper bf16 rings (DL_GROUP_S).
#define DL_GROUP8_S(st_, m_, A1n, A2n, Rn, A1c, A2c, Rc, LK, LST, GB)                             \
  do {                                                                                           \
    constexpr int MN_ = MI * NI, M2_ = 2 * MI * NI, MT_ = 4 * MI * NI, LT_ = kNA + kNB,          \
                  R_ = 2 * MI + NI;                                                              \
    const uint32_t sa_ = lds_base + (LST) * kStageB + wave * kNA * 1024;                          \
    const uint32_t sb_ = lds_base + (LST) * kStageB + kTileA + wave * kNB * 1024;                 \
    DL_WIDEN(Rc, b1, b2);                                                                        \
    __builtin_amdgcn_sched_barrier(0);                                                           \
    _Pragma("unroll") for (int q_ = 0; q_ < M2_; ++q_) {                                         \
      _Pragma("unroll") for (int r_ = q_ * R_ / M2_; r_ < (q_ + 1) * R_ / M2_; ++r_)             \
          DL_READ8_1(st_, m_, A1n, A2n, Rn, r_);                                                 \
      __builtin_amdgcn_sched_barrier(0);                                                         \
      if (q_ < MN_)                                                                              \
        acc[q_ / NI][q_ % NI] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(                         \
            A1c[q_ / NI], b1[q_ % NI], acc[q_ / NI][q_ % NI], 0, 0, 0);                          \
      else                                                                                       \
        acc[(q_ - MN_) / NI][(q_ - MN_) % NI] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(         \
            A2c[(q_ - MN_) / NI], b2[(q_ - MN_) % NI], acc[(q_ - MN_) / NI][(q_ - MN_) % NI], 0, 0, 0); \
      __builtin_amdgcn_sched_barrier(0);                                                         \
      _Pragma("unroll") for (int l_ = 0; l_ < LT_; ++l_) {                                       \
        if ((l_ * MT_) / LT_ == (GB) + q_) {                                                     \
          const bool isa_ = l_ < 2 * kMinAB ? (l_ % 2 == 0) : (kNA > kNB);                       \
          const int ix_ = l_ < 2 * kMinAB ? l_ / 2 : kMinAB + (l_ - 2 * kMinAB);                 \
          if (isa_) {                                                                            \
            if (ix_ < na_eff) dload16(rsA, aoff[ix_], (LK) * kRowA, sa_ + ix_ * 1024);           \
          } else {                                                                               \
            dload16(rsB, boff[ix_], (LK) * kRowB, sb_ + ix_ * 1024);                             \
          }                                                                                      \
        }                                                                                        \
      }                                                                                          \
      __builtin_amdgcn_sched_barrier(0);                                                         \
    }                                                                                            \
  } while (0)

  // Two-stage rings (bf16 big tiles): the refill of the stage freed by a
  // barrier (kNA + kNB loads per wave, the kNB weight blocks first, which
  // measured 2-4% faster than alternating A and B blocks) goes out one load
  // after every second MFMA of the 32 MFMAs that follow the barrier, i.e.
  // over the first two operand groups of the step.
  // Loads bunched after the barrier queue up at the address unit (four waves
  // issue theirs at once) and stall the issuing wave, and with it its matrix
  // pipe; spread this way they leave 32 MFMAs for the last load to land.
  // The group's own operand reads (next slice) go out one per MFMA over its
  // first MI + NI MFMAs.  GB: index of the group's first MFMA counted from
  // the barrier.
#define DL_READ1(sa_, sb_, ks_, A_, B_, idx_)                                                    \
  do {                                                                                           \
    const int ro_ = rd_row * kRowA + (((2 * (ks_) + (lane >> 5)) ^ rd_sa) << 4);                 \
    if ((idx_) < MI)                                                                             \
      A_[(idx_)] = *reinterpret_cast<const bf16x8_t*>(smem + (sa_) * kAStride +                  \
                                                      (wm * TM + (idx_) * 32) * kRowA + ro_);    \
    else                                                                                         \
      B_[(idx_) - MI] = *reinterpret_cast<const bf16x8_t*>(                                      \
          smem + kBBase + (sb_) * kBStride + (wn * TN + ((idx_) - MI) * 32) * kRowB + ro_);      \
  } while (0)
  // Deeper rings (the medium, small and tall families, fp8 big tiles): the
  // refill of a freed stage is spread evenly over all MFMAs of the next step
  // (refill list entry l, A and B blocks alternating while both remain, goes
  // out after MFMA (l * MT) / LT of the step: MT MFMAs, LT loads), and the
  // group's operand reads over its MFMAs.  Against one block of loads after
  // the barrier: EP-share cold experts -10% (bf16 and fp8), fp8 4096-row
  // expert -6..-11%.
  constexpr int kMinAB = kNA < kNB ? kNA : kNB;
#define DL_GROUP_S(st_, ks_, An, Bn, Ac, Bc, LK, LST, GB)                                        \
  do {                                                                                           \
    constexpr int MN_ = MI * NI, MT_ = 4 * MI * NI, LT_ = kNA + kNB, R_ = MI + NI;               \
    const uint32_t sa_ = lds_base + (LST) * kAStride + wave * kNA * 1024;                         \
    const uint32_t sb_ = lds_base + kBBase + (LST) * kBStride + wave * kNB * 1024;                \
    _Pragma("unroll") for (int m_ = 0; m_ < MN_; ++m_) {                                         \
      _Pragma("unroll") for (int r_ = m_ * R_ / MN_; r_ < (m_ + 1) * R_ / MN_; ++r_)             \
          DL_READ1(st_, st_, ks_, An, Bn, r_);                                                   \
      __builtin_amdgcn_sched_barrier(0);                                                         \
      acc[m_ / NI][m_ % NI] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(                           \
          Ac[m_ / NI], Bc[m_ % NI], acc[m_ / NI][m_ % NI], 0, 0, 0);                             \
      __builtin_amdgcn_sched_barrier(0);                                                         \
      _Pragma("unroll") for (int l_ = 0; l_ < LT_; ++l_) {                                       \
        if ((l_ * MT_) / LT_ == (GB) + m_) {                                                     \
          const bool isa_ = l_ < 2 * kMinAB ? (l_ % 2 == 0) : (kNA > kNB);                       \
          const int ix_ = l_ < 2 * kMinAB ? l_ / 2 : kMinAB + (l_ - 2 * kMinAB);                 \
          if (isa_) {                                                                            \
            if (ix_ < na_eff) dload16(rsA, aoff[ix_], (LK) * kRowA, sa_ + ix_ * 1024);           \
          } else {                                                                               \
            dload16(rsB, boff[ix_], (LK) * kRowB, sb_ + ix_ * 1024);                             \
          }                                                                                      \
        }                                                                                        \
      }                                                                                          \
      __builtin_amdgcn_sched_barrier(0);                                                         \
    }                                                                                            \
  } while (0)
  // Two-deep A ring (bf16 big tiles): the refill after the barrier that ends
  // step kt goes out one load after every second MFMA of the 32 MFMAs that
  // follow the barrier.  Split rings: the A blocks of step kt + 2 in the first
  // group (the wait that ends the next step needs them), then the B blocks
  // of step kt + 3.  One ring: the B blocks of step kt + 2 first, then its A
  // blocks (weight-first measured 2-4% faster there).  GB: index of the
  // group's first MFMA counted from the barrier.
#define DL_GROUP_R(sa_, sb_, ks_, An, Bn, Ac, Bc, LKA, LSTA, LKB, LSTB, GB)                      \
  do {                                                                                           \
    static_assert(kNA == kNB && kNA + kNB == MI * NI, "one load per two MFMAs of two groups"); \
    const uint32_t la_ = lds_base + (LSTA) * kAStride + wave * kNA * 1024;                        \
    const uint32_t lb_ = lds_base + kBBase + (LSTB) * kBStride + wave * kNB * 1024;               \
    _Pragma("unroll") for (int m_ = 0; m_ < MI * NI; ++m_) {                                     \
      if (m_ < MI + NI) DL_READ1(sa_, sb_, ks_, An, Bn, m_);                                     \
      __builtin_amdgcn_sched_barrier(0);                                                         \
      acc[m_ / NI][m_ % NI] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(                           \
          Ac[m_ / NI], Bc[m_ % NI], acc[m_ / NI][m_ % NI], 0, 0, 0);                             \
      __builtin_amdgcn_sched_barrier(0);                                                         \
      if (m_ % 2 == 1) {                                                                         \
        const int l_ = ((GB) + m_) / 2;                                                          \
        if (kSplit ? l_ < kNA : l_ >= kNB) {                                                     \
          const int i_ = kSplit ? l_ : l_ - kNB;                                                 \
          dload16(rsA, aoff[i_], (LKA) * kRowA, la_ + i_ * 1024);                                \
        } else {                                                                                 \
          const int i_ = kSplit ? l_ - kNA : l_;                                                 \
          dload16(rsB, boff[i_], (LKB) * kRowB, lb_ + i_ * 1024);                                \
        }                                                                                        \
      }                                                                                          \
      __builtin_amdgcn_sched_barrier(0);                                                         \
    }                                                                                            \
  } while (0)

  f32x16_t acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // The previous tile's epilogue stores may still be in flight: the ring
  // waits below count this tile's loads only, and since loads complete in
  // issue order, older outstanding stores can only make those waits
  // stricter (not waiting for the stores here: fine-grained layer gate/up
  // -3%).
  __syncthreads();  // every wave is done with the previous tile's LDS
  if constexpr (kSplit) {
    // Split rings: A(0), B(0), B(1), A(1); B(2) goes out with step 0's
    // first operand group.  Step 0 has landed once only B(1) and A(1) are
    // outstanding.
    const uint32_t la_ = lds_base + wave * kNA * 1024;
    const uint32_t lb_ = lds_base + kBBase + wave * kNB * 1024;
    const int k0 = krot(0), k1 = krot(min(1, KT - 1));
#pragma unroll
    for (int i = 0; i < kNA; ++i) dload16(rsA, aoff[i], k0 * kRowA, la_ + i * 1024);
#pragma unroll
    for (int i = 0; i < kNB; ++i) dload16(rsB, boff[i], k0 * kRowB, lb_ + i * 1024);
#pragma unroll
    for (int i = 0; i < kNB; ++i) dload16(rsB, boff[i], k1 * kRowB, lb_ + kBStride + i * 1024);
#pragma unroll
    for (int i = 0; i < kNA; ++i) dload16(rsA, aoff[i], k1 * kRowA, la_ + kAStride + i * 1024);
    wait_vmcnt<kNA + kNB>();
  } else {
#pragma unroll
    for (int s = 0; s < STAGES; ++s) DL_LOAD(krot(min(s, KT - 1)), s);
    wait_steps<STAGES - 1, kNB, kPerStep>(per_step);  // step 0 has landed (this wave's part)
  }
  __syncthreads();  // ... and every wave's part
  // Step kt computes stage kt % STAGES.  Its last operand reads come before
  // the barrier that ends the step, so right after that barrier the stage
  // is refilled with step kt + STAGES: a step's loads have STAGES - 1 whole
  // steps of MFMA work to land.  Past the last step the loads repeat the
  // last step (never read).
  if constexpr (kSplit) {
    // A in 2 stages, B in 3: after the barrier that ends step kt, A(kt + 2)
    // refills A stage kt % 2 (spread over the first group of step kt + 1)
    // and B(kt + 3) refills B stage kt % 3 (over its second group).  The
    // wait that ends step kt + 1 needs steps kt + 2 complete, so B(kt + 3)
    // -- the last kNB loads issued -- may still be in flight: each weight
    // tile has two steps of MFMAs to land, each activation tile one.
    bf16x8_t a0[MI], b0[NI], a1[MI], b1[NI];
    DL_READ(0, 0, 0, a0, b0);
    int sa = 0, sb = 0;
    int lka = krot(min(1, KT - 1)), lsta = 1;  // A refill in flight (issued by the prologue)
    int lkb = krot(min(2, KT - 1)), lstb = 2;  // B refill issued by step 0's first group
    for (int kt = 0; kt < KT; ++kt) {
      const int nsa = sa ^ 1, nsb = sb == 2 ? 0 : sb + 1;
      DL_GROUP_R(sa, sb, 1, a1, b1, a0, b0, lka, lsta, lkb, lstb, MI * NI);
      DL_GROUP(sa, sb, 2, a0, b0, a1, b1);
      DL_GROUP(sa, sb, 3, a1, b1, a0, b0);
      wait_vmcnt<kNB>();  // step kt + 1 has landed (this wave's part)
      __syncthreads();    // ... and every wave's; A stage sa and B stage sb are free
      lka = krot(min(kt + 2, KT - 1));
      lsta = sa;
      lkb = krot(min(kt + 3, KT - 1));
      lstb = sb;
      DL_GROUP_R(nsa, nsb, 0, a0, b0, a1, b1, lka, lsta, lkb, lstb, 0);
      sa = nsa;
      sb = nsb;
    }
  } else if constexpr (!FP8 && STAGES == 2) {
    // The refill of step kt + 2 into stage st starts after the barrier that
    // ends step kt (in the group computing its last slice) and ends in the
    // first group of step kt + 1.  That group's first pass repeats half of
    // the prologue's loads of step 1 (same bytes, same place; they land
    // before the barrier that ends step 0).
    bf16x8_t a0[MI], b0[NI], a1[MI], b1[NI];
    DL_READ(0, 0, 0, a0, b0);
    int st = 0;
    int lk = krot(min(1, KT - 1)), lst = 1;  // the refill in flight: its K step and stage
    for (int kt = 0; kt < KT; ++kt) {
      const int nst = st ^ 1;
      DL_GROUP_R(st, st, 1, a1, b1, a0, b0, lk, lst, lk, lst, MI * NI);
      DL_GROUP(st, st, 2, a0, b0, a1, b1);
      DL_GROUP(st, st, 3, a1, b1, a0, b0);
      wait_vmcnt<0>();  // step kt + 1 has landed (this wave's part)
      __syncthreads();  // ... and every wave's; stage st is free
      lk = krot(min(kt + STAGES, KT - 1));
      lst = st;
      DL_GROUP_R(nst, nst, 0, a0, b0, a1, b1, lk, lst, lk, lst, 0);
      st = nst;
    }
  } else if constexpr (!FP8) {
    // Deeper rings: the refill of step kt + STAGES into stage st is spread
    // over the four operand groups of step kt + 1 (it has STAGES - 2 more
    // steps to land).  The first pass repeats loads of the prologue's last
    // step (same bytes, same place).
    bf16x8_t a0[MI], b0[NI], a1[MI], b1[NI];
    DL_READ(0, 0, 0, a0, b0);
    int st = 0;
    int lk = krot(min(STAGES - 1, KT - 1)), lst = STAGES - 1;  // the refill in flight
    for (int kt = 0; kt < KT; ++kt) {
      const int nst = st + 1 == STAGES ? 0 : st + 1;
      DL_GROUP_S(st, 1, a1, b1, a0, b0, lk, lst, MI * NI);
      DL_GROUP_S(st, 2, a0, b0, a1, b1, lk, lst, 2 * MI * NI);
      DL_GROUP_S(st, 3, a1, b1, a0, b0, lk, lst, 3 * MI * NI);
      wait_steps<STAGES - 2, kNB, kPerStep>(per_step);  // step kt + 1 has landed
      __syncthreads();
      lk = krot(min(kt + STAGES, KT - 1));
      lst = st;
      DL_GROUP_S(nst, 0, a0, b0, a1, b1, lk, lst, 0);
      st = nst;
    }
  } else {
    bf16x8_t a10[MI], a20[MI], a11[MI], a21[MI], b1[NI], b2[NI];
    uint4 r0[NI], r1[NI];
    DL_READ8(0, 0, a10, a20, r0);
    int st = 0;
    int lk = krot(min(STAGES - 1, KT - 1)), lst = STAGES - 1;  // the refill in flight
    for (int kt = 0; kt < KT; ++kt) {
      const int nst = st + 1 == STAGES ? 0 : st + 1;
      DL_GROUP8_S(st, 1, a11, a21, r1, a10, a20, r0, lk, lst, 2 * MI * NI);
      wait_steps<STAGES - 2, kNB, kPerStep>(per_step);  // step kt + 1 has landed
      __syncthreads();
      lk = krot(min(kt + STAGES, KT - 1));
      lst = st;
      DL_GROUP8_S(nst, 0, a10, a20, r0, a11, a21, r1, lk, lst, 0);
      st = nst;
    }
  }
#undef DL_GROUP_R
#undef DL_GROUP_S
#undef DL_READ1
#undef DL_GROUP8_S
#undef DL_READ8_1
#undef DL_GROUP
#undef DL_MMA
#undef DL_WIDEN
#undef DL_READ8
#undef DL_READ
#undef DL_LOAD

  // Split-K: every piece stores its f32 partial sums in its part of the
  // tile's slot, then counts itself finished; the piece that counts last
  // adds the parts in piece order -- the same order whichever piece that is,
  // so results are reproducible run to run -- and runs the epilogue.
  // Ordering: parts and counter are accessed only with agent-scope atomics,
  // which the hardware performs at the level that is coherent across the
  // XCDs' L2 caches; every wave waits for its part stores to be acknowledged
  // (vmcnt 0) and the workgroup barrier orders that before the counter
  // increment; the finisher issues its part loads only after the increment
  // that returned n_split - 1 (the result reaches them through LDS and a
  // barrier).  So each part is complete at the coherent level before any
  // load of it is issued.  The atomics are relaxed (no release/acquire
  // fences): at agent scope those write back and invalidate the whole L2,
  // which made the pieces slower than no split.
  if (n_split > 1) {
    // part layout [wave][fragment][register][lane]: 16 stores 256 bytes apart
    constexpr int kPart = BM * BN;  // floats
    float* mine = slot + (int64_t)piece * kPart + wave * (MI * NI * 16 * 64) + lane;
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NI; ++j) {
        float* dst = mine + (i * NI + j) * (16 * 64);
#pragma unroll
        for (int r = 0; r < 16; ++r)
          __hip_atomic_store(dst + r * 64, acc[i][j][r], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __builtin_amdgcn_sched_barrier(0);
      }
    wait_vmcnt<0>();  // every store of this wave has completed
    __syncthreads();  // ... of every wave; the ring is free
    volatile int* flag = reinterpret_cast<volatile int*>(smem);
    if (tid == 0)
      flag[0] = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == n_split - 1;
    __syncthreads();
    const bool last = flag[0] != 0;
    __syncthreads();  // the flag is read before the epilogue reuses the LDS
    if (!last) return;
    if (tid == 0) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);  // next launch
  }

  // Epilogue: stage bf16 results in LDS ([BM][BN/2 + 8]) and write 16-byte
  // chunks of whole rows.  Gate/up: one pass, feature fragment j pairs with
  // up fragment j + NI/2.  Down: two passes of BN/2 columns (each wave
  // contributes column fragments pass * NI/2 .. pass * NI/2 + NI/2 - 1).
  // fp8 weights: the per-channel scales multiply the accumulators here.
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
      float sg = 1.f, su = 1.f;
      if constexpr (FP8) {
        if constexpr (GATED) {
          const int fc = min(nti * (BN / 2) + cl, n_out - 1);
          sg = __uint_as_float((uint32_t)wd.s_gu[fc] << 16);
          su = __uint_as_float((uint32_t)wd.s_gu[n_out + fc] << 16);
        } else {
          const int cc = min(nti * BN + wn * TN + j * 32 + (lane & 31), n_out - 1);
          sg = __uint_as_float((uint32_t)wd.s_down[cc] << 16);
        }
      }
#pragma unroll
      for (int i = 0; i < MI; ++i) {
        // the fragment's values (and its up partner's): the accumulators, or
        // for a split tile the sum of its pieces' parts in piece order
        float f0[16], f1[GATED ? 16 : 1];
        if (n_split > 1) {
          // every piece's part of the fragment (and of its partner) is
          // loaded before any is added: one memory round trip, not one per
          // piece; then the sum in piece order
          float t0[kMaxSplit][16], t1[kMaxSplit][GATED ? 16 : 1];
          float* pp = slot + wave * (MI * NI * 16 * 64) + lane + (i * NI + j) * (16 * 64);
#pragma unroll
          for (int q = 0; q < kMaxSplit; ++q) {
            if (q < n_split) {
              float* p0 = pp + (int64_t)q * (BM * BN);
#pragma unroll
              for (int r = 0; r < 16; ++r)
                t0[q][r] = __hip_atomic_load(p0 + r * 64, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              if constexpr (GATED) {
                float* p1 = p0 + (NI / 2) * (16 * 64);
#pragma unroll
                for (int r = 0; r < 16; ++r)
                  t1[q][r] = __hip_atomic_load(p1 + r * 64, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              }
            }
          }
#pragma unroll
          for (int r = 0; r < 16; ++r) f0[r] = 0.f;
#pragma unroll
          for (int r = 0; r < (GATED ? 16 : 1); ++r) f1[r] = 0.f;
#pragma unroll
          for (int q = 0; q < kMaxSplit; ++q) {
            if (q < n_split) {
#pragma unroll
              for (int r = 0; r < 16; ++r) f0[r] += t0[q][r];
              if constexpr (GATED)
#pragma unroll
                for (int r = 0; r < 16; ++r) f1[r] += t1[q][r];
            }
          }
        } else {
#pragma unroll
          for (int r = 0; r < 16; ++r) f0[r] = acc[i][j][r];
          if constexpr (GATED)
#pragma unroll
            for (int r = 0; r < 16; ++r) f1[r] = acc[i][j + NI / 2][r];
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int rl = wm * TM + i * 32 + c_row(lane, r);
          float v;
          if constexpr (GATED) {
            const float gv = FP8 ? f0[r] * sg : f0[r];
            const float uv = FP8 ? f1[r] * su : f1[r];
            v = gv * __builtin_amdgcn_rcpf(1.f + __expf(-gv)) * uv;
          } else {
            v = FP8 ? f0[r] * sg : f0[r];
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

// The FFN launch for bf16 or fp8 weights: every tile of the big family (256
// rows), then the medium (128 rows; 256 for a cold expert's remainder above
// 128 rows) and small (64 rows) tiles of the row remainders and of cold
// experts, in one persistent grid.  The smaller families come last, so they
// also fill the tail of the big one; cold
// experts are weight-streaming bound, and narrow tiles spread each expert's
// weights over more CUs.  bf16 big tiles keep 2 activation stages and 3
// weight stages (all 160 KB of LDS; the plan's tile -> group map replaces a
// group table in LDS).  fp8 stages are smaller (e4m3 B tiles), so their
// rings are deeper: 3 big / 6 medium and small stages instead of 2 / 4.
template <bool FP8>
constexpr int ring_bytes(int a_stages, int b_stages, int bm, int bn) {
  return a_stages * bm * kBK * 2 + b_stages * bn * kBK * (FP8 ? 1 : 2);
}
constexpr int cmax(int a, int b) { return a > b ? a : b; }
template <bool GATED, bool FP8>
__global__ __launch_bounds__(256, 1) void ffn_dlds_kernel(const FfnParams p) {
  // fp8 small tiles are twice as wide: per K step they read as many weight
  // bytes as bf16 ones and half the activation bytes per weight byte
  constexpr int kSBN = FP8 ? kSmallBN8 : kSmallBN;
  constexpr int kBigStages = FP8 ? 3 : 2, kBigBStages = FP8 ? 3 : 3, kSmallStages = FP8 ? 6 : 4,
                kTallStages = 3;
  constexpr int kRing = cmax(cmax(ring_bytes<FP8>(kBigStages, kBigBStages, kBM, kBN),
                                  ring_bytes<FP8>(kTallStages, kTallStages, kTallBM, kMedBN)),
                             cmax(ring_bytes<FP8>(kSmallStages, kSmallStages, kMedBM, kMedBN),
                                  ring_bytes<FP8>(kSmallStages, kSmallStages, kSmallBM, kSBN)));
  __shared__ __attribute__((aligned(1024))) unsigned char smem[kRing];
  const bool probe = p.clk != nullptr && (int)blockIdx.x < p.clk_n;
  unsigned long long clk0 = 0, rt0 = 0;
  if (probe) {
    clk0 = __builtin_amdgcn_s_memtime();
    rt0 = __builtin_amdgcn_s_memrealtime();
  }
  const int stage = GATED ? 0 : 1, st3 = 3 * stage;
  const int tot0 = p.tile_totals[st3], tot1 = p.tile_totals[st3 + 1], tot2 = p.tile_totals[st3 + 2];
  const uint32_t lds_base = (uint32_t)(uintptr_t)(lds_vptr)smem;
  const int nwg = gridDim.x;
  const int ncol_big = GATED ? (p.n_out + kBN / 2 - 1) / (kBN / 2) : (p.n_out + kBN - 1) / kBN;
  // The weight-streaming families (medium, tall, small) rotate their K walk
  // by tile; big tiles share activation and weight bands with the tiles next
  // to them in an XCD's L2, which a rotation would pull apart.
  constexpr bool kRotateBig = false;
  const int total = tot0 + tot1 + tot2;
  // Split-K: a launch of at most half a grid of tiles cuts each tile into
  // n_split pieces of consecutive K steps (at least kMinSplitSteps each), so
  // that more CUs stream its weights; the partial sums of a tile's pieces
  // take n_split parts of its slot (big tiles first, then family 1, then
  // small, each slot sized for its family).
  int n_split = 1;
  int64_t slot1 = 0, slot2 = 0;  // float offsets of the family 1 and small slots
  if (p.split_slots != nullptr && total > 0 && 2 * total <= nwg && total <= kSplitCounters) {
    n_split = max(1, min(min(kMaxSplit, nwg / total), p.K / (kBK * kMinSplitSteps)));
    const int64_t per = (int64_t)tot0 * (kBM * kBN) + (int64_t)tot1 * (kTallBM * kMedBN) +
                        (int64_t)tot2 * (kSmallBM * kSBN);  // floats per piece
    while (n_split > 1 && (int64_t)n_split * per * 4 > p.split_bytes) --n_split;
    slot1 = (int64_t)n_split * tot0 * (kBM * kBN);
    slot2 = slot1 + (int64_t)n_split * tot1 * (kTallBM * kMedBN);
  }
  const int items = total * n_split;  // work item = tile * n_split + piece
  // Work items go round by round: a full round of the grid gives each XCD
  // (the hardware deals workgroups round robin over the 8 XCDs) a run of
  // nwg / 8 consecutive items; a partial round gives each XCD a run of
  // ceil(count / 8), so a launch with fewer items than workgroups still
  // uses every XCD's L2 and memory path.
  const int xcd = blockIdx.x & 7, xj = blockIdx.x >> 3;
  for (int base = 0; base < items; base += nwg) {
    const int cnt = min(nwg, items - base);
    const int q = cnt == nwg ? (nwg >> 3) : ((cnt + 7) >> 3);
    const int idx = xcd * q + xj;
    if (xj >= q || idx >= cnt) continue;
    const int item = base + idx;
    const int tile = item / n_split, piece = item - tile * n_split;
    const int g = p.tile_group[tile];
    const GroupDesc gd = p.groups[g];
    if (tile < tot0) {
      const int local = tile - gd.t0[st3];
      int rt, nti;
      panel_decode<GATED ? 8 : 4>(local, gd.nrt[stage][0], ncol_big, rt, nti);
      dl_tile<GATED, FP8, kBM, kBN, kBigStages, kBigBStages, kRing>(
          p, smem, lds_base, gd, p.wtab[g], nti, rt * kBM, kRotateBig ? tile : -1, n_split, piece,
          n_split > 1 ? p.split_slots + (int64_t)tile * n_split * (kBM * kBN) : nullptr, p.split_cnt + tile);
    } else {
      // medium or small: the row tiles of one column tile are consecutive
      const bool med = tile < tot0 + tot1;
      const int f = med ? 1 : 2;
      const int local = tile - (med ? tot0 : tot0 + tot1) - gd.t0[st3 + f];
      const int nti = local / gd.nrt[stage][f];
      const int ri = local - nti * gd.nrt[stage][f];
      float* sl = n_split == 1 ? nullptr
                  : med ? p.split_slots + slot1 + (int64_t)(tile - tot0) * n_split * (kTallBM * kMedBN)
                        : p.split_slots + slot2 + (int64_t)(tile - tot0 - tot1) * n_split * (kSmallBM * kSBN);
      if (med && gd.h1[stage] == kTallBM)
        dl_tile<GATED, FP8, kTallBM, kMedBN, kTallStages, kTallStages, kRing>(
            p, smem, lds_base, gd, p.wtab[g], nti, gd.row1[stage] + ri * kTallBM, tile, n_split, piece, sl,
            p.split_cnt + tile);
      else if (med)
        dl_tile<GATED, FP8, kMedBM, kMedBN, kSmallStages, kSmallStages, kRing>(
            p, smem, lds_base, gd, p.wtab[g], nti, gd.row1[stage] + ri * kMedBM, tile, n_split, piece, sl,
            p.split_cnt + tile);
      else
        dl_tile<GATED, FP8, kSmallBM, kSBN, kSmallStages, kSmallStages, kRing>(
            p, smem, lds_base, gd, p.wtab[g], nti, gd.row2[stage] + ri * kSmallBM, tile, n_split, piece, sl,
            p.split_cnt + tile);
    }
  }
  if (probe) {
    const unsigned long long clk1 = __builtin_amdgcn_s_memtime(), rt1 = __builtin_amdgcn_s_memrealtime();
    if (threadIdx.x == 0) {
      p.clk[2 * blockIdx.x] = clk1 - clk0;
      p.clk[2 * blockIdx.x + 1] = rt1 - rt0;
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
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  const int total = p.tile_totals[GATED ? 0 : 3];
  const int K = p.K, n_out = p.n_out;
  const float* A = reinterpret_cast<const float*>(p.a);
  float* O = reinterpret_cast<float*>(p.out);

  for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
    const int g = p.tile_group[tile];
    const GroupDesc gd = p.groups[g];
    const WeightDesc wd = p.wtab[g];
    const int local = tile - gd.t0[GATED ? 0 : 3];
    const int nti = local / gd.nrt[GATED ? 0 : 1][0];
    const int m0 = (local - nti * gd.nrt[GATED ? 0 : 1][0]) * BM;
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
                      const WeightDesc* wtab, int G, const int32_t* tile_totals,
                      const int32_t* tile_group, float* split_slots, int32_t* split_cnt,
                      int64_t split_bytes, int max_tiles,
                      const void* xp, void* h, void* y, int d, int f, int num_cu,
                      unsigned long long* clk, int clk_n, hipStream_t s) {
  if (max_tiles <= 0) return hipSuccess;
  const FfnParams p = stage == 0 ? FfnParams{groups, wtab, tile_totals, tile_group, split_slots, split_cnt,
                                             split_bytes, xp, h, G, d, f, clk, clk_n}
                                 : FfnParams{groups, wtab, tile_totals, tile_group, split_slots, split_cnt,
                                             split_bytes, h, y, G, f, d, clk, clk_n};
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
      ffn_dlds_kernel<true, true><<<grid, 256, 0, s>>>(p);
    else
      ffn_dlds_kernel<false, true><<<grid, 256, 0, s>>>(p);
  } else {
    if (stage == 0)
      ffn_dlds_kernel<true, false><<<grid, 256, 0, s>>>(p);
    else
      ffn_dlds_kernel<false, false><<<grid, 256, 0, s>>>(p);
  }
  return hipGetLastError();
}

}  // namespace aep
