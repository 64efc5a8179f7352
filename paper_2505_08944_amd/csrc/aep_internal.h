// Internal definitions shared by libaep's host code and its gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace aep {

// One mu-queue entry (16 bytes): the row it refers to (the token's tensor
// stays where it arrived, as the paper's token metadata refers to GPU-resident
// input tensors), the layer-local token id and top-k slot, and the gate weight.
struct QEntry {
  const void* row;
  int32_t token_slot;  // token | slot << 24
  float w;
};
static_assert(sizeof(QEntry) == 16, "QEntry must be 16 bytes");

constexpr int kTokenBits = 24;
constexpr int32_t kTokenMask = (1 << kTokenBits) - 1;

// Weights of one expert (device pointers) -- the per-layer table the FFN
// kernels read.
struct WeightDesc {
  const void* gate;
  const void* up;
  const void* down;
  const uint16_t* s_gu;    // fp8 only: [2f] bf16 scales
  const uint16_t* s_down;  // fp8 only: [d]  bf16 scales
  const void* pad;
};
static_assert(sizeof(WeightDesc) == 48, "WeightDesc layout");

// One FFN group of a drained batch, written by the plan kernel.  A group's
// rows are covered by up to three row-tile families (bf16 / fp8 weights),
// chosen per FFN stage (0: gate/up, 1: down): "big" 256-row tiles over the
// full 256-row blocks, plus one more for a remainder above 128 rows (above
// 192 rows in a stage where the extra big tiles would start another round
// of the grid and that has fewer than 4 rounds; never in a cold batch), then
// "medium" 128-row tiles and at most one "small" 64-row tile over the
// remainder.  In a cold batch a remainder above 128 rows takes one "tall"
// 256-row tile (kTallBM) in family 1 instead (h1 = kTallBM), so a cold
// expert's weights are streamed once.  f32 weights use the big family alone,
// with 64-row tiles.  In stage s, family 0 covers rows [0, nrt[s][0] * 256),
// family 1 [row1[s], row1[s] + nrt[s][1] * h1[s]) and family 2 [row2[s],
// row2[s] + nrt[s][2] * 64), clamped to n.  t0[s * 3 + f] is the group's first
// tile id in family f of stage s.
struct GroupDesc {
  int32_t n;          // rows
  int32_t x_row0;     // first row in x_perm
  int32_t y_row0;     // first row in h and y
  int32_t t0[6];      // first tile id per (stage, family)
  int32_t nrt[2][3];  // row tiles per (stage, family): big, medium (or tall), small
  int32_t row1[2];    // first row of family 1 per stage (family 0 starts at row 0)
  int32_t row2[2];    // first row of family 2 per stage
  int32_t h1[2];      // rows per family-1 tile per stage: kMedBM, or kTallBM in a cold batch
  int32_t pad[3];
};
static_assert(sizeof(GroupDesc) == 96, "GroupDesc layout");

// Device error flag bits.
constexpr int32_t kErrNonFinite = 1;
constexpr int32_t kErrTokenRange = 2;
constexpr int32_t kErrSlotRange = 4;
constexpr int32_t kErrCollision = 8;

constexpr int kRouteThreads = 256;
constexpr int kRouteLanes = 8;                              // lanes per token in the router
constexpr int kRouteTokens = kRouteThreads / kRouteLanes;   // tokens per router workgroup
constexpr int kMaxRouteExperts = 64;
constexpr int kDirectPrefixBlocks = 64;  // router workgroups whose appends sum earlier counts directly
constexpr int kMaxTopK = 8;
constexpr int kMaxGroups = 1024;

// FFN tiling (bf16 / fp8 weights): tiles of BM rows x BN columns; gate/up
// tiles cover BN/2 features of gate and the same BN/2 of up.
constexpr int kBM = 256;
constexpr int kBN = 256;
constexpr int kBK = 64;
constexpr int kSmallBM = 64;            // small-family tiles: 64 rows ...
constexpr int kSmallBN = 128;           // ... x 128 columns (gate/up: 64 features)
constexpr int kSmallBN8 = 256;          // ... x 256 columns with fp8 weights
constexpr int kMedBM = 128;             // medium-family tiles: 128 rows ...
constexpr int kMedBN = 128;             // ... x 128 columns
constexpr int kTallBM = 256;            // family 1 of a cold batch: 256 rows x kMedBN columns
// Split-K of an FFN launch with at most half a grid of tiles: up to kMaxSplit
// pieces of at least kMinSplitSteps K steps each per tile, for launches of at
// most kSplitCounters tiles; kSplitPartBytes is one piece's partial sums of a
// big tile (the largest family).
constexpr int kMaxSplit = 4;
constexpr int kMinSplitSteps = 8;
constexpr int kSplitCounters = 1024;
constexpr int64_t kSplitPartBytes = (int64_t)kBM * kBN * 4;
// The partial sums' area of a context: 128 big-tile pieces (a launch of 64
// big tiles splits in 2, one of 128 small tiles in 2, 32 big tiles in 4;
// the kernel lowers n_split until a launch's pieces fit).
constexpr int64_t kSplitBytes = 128 * kSplitPartBytes;
// f32 path
constexpr int kBM32 = 64;
constexpr int kBN32 = 64;

// Layer-granularity pick (host): the block to drain next from per-block
// totals R[nb] under an aep_policy (defrag: R[b] + sum_{i=1..lookahead}
// R[(b + i) mod nb] * delta^i).  Ties go to the lowest block; false when every
// block is empty.  Defined with the host scheduler (sched.hip).
bool pick_block(const int64_t* R, int nb, int policy, double delta, int lookahead, int* pb);

// ---------------------------------------------------------------- launchers
// Each returns hipGetLastError() after the launch.
// Routes T tokens; blockcnt [ceil(T / kRouteTokens)][E] receives each router
// workgroup's row count per expert.  Above kDirectPrefixBlocks workgroups the
// launch then rewrites them into each workgroup's first queue slot and writes
// depth_nxt (depth_cur + this fragment's counts); below, append does both.
// done: a launch counter that must be 0 before the launch (the kernel leaves
// it 0).
hipError_t launch_route(const float* logits, int T, int E, int k, int renorm, int32_t* r_idx,
                        float* r_w, int32_t* r_rank, int32_t* blockcnt, int32_t* idx_out,
                        float* w_out, const int32_t* depth_cur, int32_t* depth_nxt, int32_t* done,
                        int32_t* err, hipStream_t s);
// token_ids == nullptr: token t of the fragment is token_base + t.  Else its
// id is token_ids[t] (< n_ids) and it claims pool entry live[id] / pend[id].
hipError_t launch_append(const int32_t* r_idx, const float* r_w, const int32_t* r_rank,
                         const int32_t* first_slot, int T, int E, int k, const char* x,
                         int64_t row_bytes, int32_t token_base, const int32_t* depth_cur,
                         int32_t* depth_nxt, QEntry* q, int64_t q_stride, const void** tok_row,
                         const int32_t* token_ids, int n_ids, int32_t* live, int32_t* pend,
                         int32_t* err, hipStream_t s);
// Rows of several experts in one launch: rows [pre[e], pre[e+1]) to queue e
// (pre: device, E + 1 entries, exclusive prefix of the per-expert counts).
hipError_t launch_enqueue_grouped(const char* rows, int64_t row_bytes, const int32_t* token_ids,
                                  const int32_t* slots, const float* gate_w, int n, int n_tokens, int k, int E,
                                  const int32_t* pre, const int32_t* depth_cur, int32_t* depth_nxt, QEntry* q,
                                  int64_t q_stride, int32_t* err, hipStream_t s);
hipError_t launch_enqueue_rows(const char* rows, int64_t row_bytes, const int32_t* token_ids,
                               const int32_t* slots, const float* gate_w, int n, int n_tokens,
                               int k, int expert, int E, const int32_t* depth_cur,
                               int32_t* depth_nxt, QEntry* q, int64_t q_stride, int32_t* err,
                               hipStream_t s);
// tile_totals[6] and nt[6] (column tiles per row tile), index stage * 3 +
// family (stage 0 gate/up, 1 down; family 0 big, 1 medium, 2 small).
// med_bm = small_bm = 0 disables the two smaller families (every row in big
// tiles of big_bm).  num_cu: a batch with fewer full big gate/up tiles than
// CUs puts no remainder in a big tile.
// only_expert >= 0: drain that expert's queue alone (every other group gets
// 0 rows and keeps its queue).  depth is the current half of the layer's
// depth ping-pong, depth_other the other one; both are cleared for the
// drained experts.
// tile_group [2][tile_cap]: the group of each tile of the gate/up (row 0) and
// down (row 1) launch, tiles numbered big family first, then medium, small;
// tile_cap bounds either launch's tile count.
hipError_t launch_plan(int E, int S, int n_tokens, int k, int only_expert, int32_t* depth,
                       int32_t* depth_other, int32_t* counts, int32_t* offsets, GroupDesc* groups,
                       int32_t* tile_totals, const int* nt, int big_bm, int med_bm, int small_bm,
                       int num_cu, int32_t* tile_group, int64_t tile_cap, int32_t* pos, float* posw,
                       hipStream_t s);
// N bounds the routed rows (the exact count is offsets[E] on the device);
// pos == nullptr skips the (token, slot) -> row map.
hipError_t launch_gather(const QEntry* q, int64_t q_stride, const int32_t* offsets, int E,
                         int64_t N, int n_tokens, int shared, const void* const* tok_row,
                         char* xp, int64_t row_bytes, int32_t* row_token, float* row_w,
                         int32_t* pos, float* posw, int k, int32_t* err, hipStream_t s);
// token pool: rows [0, offsets[E]) of a batch (N bounds them) are merged into
// pool[row_token[r]]; release writes out / ready for completed ids.
hipError_t launch_pool_accumulate(int act_dtype, const void* y, int64_t N, const int32_t* offsets,
                                  int E, const int32_t* row_token, const float* row_w, float* pool,
                                  int32_t* pend, int d, hipStream_t s);
hipError_t launch_pool_release(int act_dtype, float* pool, int32_t* live, int32_t* pend, int n_ids,
                               void* out, int32_t* ready, int d, hipStream_t s);
// stage 0: gate/up (xp -> h), stage 1: down (h -> y); max_tiles bounds the
// stage's tile count (the exact count is on the device); tile_group is that
// stage's row of the plan's tile -> group map.  split_slots (split_bytes
// bytes) holds the split-K partial sums and split_cnt [kSplitCounters] the
// pieces finished per tile, zero before the launch and left zero (bf16 / fp8
// weights; split_slots == nullptr: no split).
// clk != nullptr: workgroup w < clk_n writes its elapsed (s_memtime,
// s_memrealtime) ticks to clk[2w], clk[2w + 1] (bf16 / fp8 weights only).
hipError_t launch_ffn(int stage, int act_dtype, int w_dtype, const GroupDesc* groups,
                      const WeightDesc* wtab, int G, const int32_t* tile_totals,
                      const int32_t* tile_group, float* split_slots, int32_t* split_cnt,
                      int64_t split_bytes, int max_tiles,
                      const void* xp, void* h, void* y, int d, int f, int num_cu,
                      unsigned long long* clk, int clk_n, hipStream_t s);
hipError_t launch_combine(int act_dtype, const void* y, int64_t N, int n_tokens, int S, int k,
                          const int32_t* pos, const float* posw, void* out, int d, hipStream_t s);
hipError_t launch_fp8_to_bf16(const uint8_t* codes, uint16_t* out, int64_t n, hipStream_t s);

}  // namespace aep
