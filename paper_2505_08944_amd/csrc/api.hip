// libaep host side: the C ABI declared in include/aep.h.
//
// Host state per layer holds what the host can know without a device sync --
// tokens and rows queued, an upper bound of every expert's queue depth (for
// capacity checks), which half of the device depth ping-pong is current --
// while the queue entries themselves, the per-expert depths and everything
// derived from them live in the caller's device workspace.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "aep.h"
#include "aep_internal.h"

using namespace aep;

namespace {

struct LayerState {
  int32_t tokens = 0;          // layer-local token ids handed out / declared
  int64_t rows = 0;            // queued rows (an upper bound in pool mode)
  std::vector<int64_t> bound;  // per expert, an upper bound of its queue depth
  bool pool = false;           // fed by aep_route_enqueue_ids (token-pool mode)
  int cur = 0;                 // current half of the depth ping-pong
  std::vector<uint8_t> have_w; // weights registered, per group

  void clear() {
    tokens = 0;
    rows = 0;
    pool = false;
    std::fill(bound.begin(), bound.end(), 0);
  }
};

}  // namespace

// The opaque context of include/aep.h.
struct aep_ctx {
  aep_config cfg{};
  int G = 0;
  int esz = 0;  // bytes per activation element
  // workspace layout (byte offsets)
  size_t off_err = 0, off_depth = 0, off_q = 0, off_tokrow = 0, off_wtab = 0;
  size_t off_ridx = 0, off_rw = 0, off_rrank = 0, off_blockcnt = 0;
  size_t off_counts = 0, off_offsets = 0, off_groups = 0, off_tiles = 0, off_tilegrp = 0;
  int64_t tile_cap = 0;  // entries per FFN launch in the tile -> group map
  size_t off_xp = 0, off_rowtok = 0, off_roww = 0, off_pos = 0, off_posw = 0, off_h = 0;
  size_t off_pool = 0, off_live = 0, off_pend = 0;  // token pools (cfg.token_pool)
  // split-K of the FFN launches (bf16 activations): per-tile piece counters
  // (cleared with the depth counters at binding) and the partial sums
  size_t off_splitcnt = 0, off_split = 0, split_bytes = 0;
  size_t off_grppre = 0;  // aep_enqueue_rows_grouped: prefix of the per-expert counts
  size_t ws_need = 0;
  char* ws = nullptr;
  bool ws_static = false;   // ws is the library's static workspace (aep_bind_static_workspace)
  uint64_t static_gen = 0;  // ... bound in this generation of that device's binding
  int device = -1;
  int num_cu = 0;
  std::vector<LayerState> layers;
  std::vector<WeightDesc> wtab_host;  // [layer][group]
  unsigned long long* clk = nullptr;  // clock probe (aep_set_clock_probe)
  int clk_n = 0;
  bool batch_out = false;
  bool batch_expert = false;  // the outstanding batch is a single-expert drain
  uint64_t epoch = 0;
  int32_t batch_layer = -1;

  int64_t tmax() const { return cfg.max_tokens_per_layer; }
  int64_t row_cap() const { return tmax() * cfg.top_k; }
  int32_t* err() const { return reinterpret_cast<int32_t*>(ws + off_err); }
  // router launch counter (last-workgroup scan), in the error-flag block
  int32_t* route_done() const { return reinterpret_cast<int32_t*>(ws + off_err) + 16; }
  int32_t* depth(int layer, int half) const {
    return reinterpret_cast<int32_t*>(ws + off_depth) + ((int64_t)layer * 2 + half) * cfg.n_experts;
  }
  QEntry* q(int layer) const {
    return reinterpret_cast<QEntry*>(ws + off_q) + (int64_t)layer * cfg.n_experts * tmax();
  }
  const void** tokrow(int layer) const {
    return reinterpret_cast<const void**>(ws + off_tokrow) + (int64_t)layer * tmax();
  }
  WeightDesc* wtab(int layer) const {
    return reinterpret_cast<WeightDesc*>(ws + off_wtab) + (int64_t)layer * G;
  }
  float* pool(int layer) const {
    return reinterpret_cast<float*>(ws + off_pool) + (int64_t)layer * tmax() * cfg.d_model;
  }
  int32_t* live(int layer) const { return reinterpret_cast<int32_t*>(ws + off_live) + (int64_t)layer * tmax(); }
  int32_t* pend(int layer) const { return reinterpret_cast<int32_t*>(ws + off_pend) + (int64_t)layer * tmax(); }
  template <typename T>
  T* at(size_t off) const {
    return reinterpret_cast<T*>(ws + off);
  }
};

namespace {

using Ctx = aep_ctx;

// Tiling of the FFN launches: nt[6] = column tiles per row tile, index
// stage * 3 + family (stage 0 gate/up, 1 down; family big, medium, small),
// and the row-tile heights.  f32 uses 64 x 64 tiles only; bf16 and fp8
// weights use 256 x 256 big tiles, 128 x 128 medium and 64 x 128 small ones
// (64 x 256 with fp8 weights).
void tiling(const Ctx& c, int nt[6], int* big_bm, int* med_bm, int* small_bm) {
  const int d = c.cfg.d_model, f = c.cfg.d_ffn;
  auto cdiv = [](int a, int b) { return (a + b - 1) / b; };
  if (c.cfg.act_dtype == AEP_F32) {
    nt[0] = nt[1] = nt[2] = cdiv(f, kBN32);
    nt[3] = nt[4] = nt[5] = cdiv(d, kBN32);
    *big_bm = kBM32;
    *med_bm = *small_bm = 0;
  } else {
    nt[0] = cdiv(f, kBN / 2);
    nt[1] = cdiv(f, kMedBN / 2);
    const int sbn = c.cfg.w_dtype == AEP_FP8_E4M3 ? kSmallBN8 : kSmallBN;
    nt[2] = cdiv(f, sbn / 2);
    nt[3] = cdiv(d, kBN);
    nt[4] = cdiv(d, kMedBN);
    nt[5] = cdiv(d, sbn);
    *big_bm = kBM;
    *med_bm = kMedBM;
    *small_bm = kSmallBM;
  }
}

// Upper bound of one FFN launch's tiles for a batch of N routed rows and T
// tokens: every group's rows in big tiles (one partial big row tile per
// non-empty group), plus at most 2 medium and 1 small row tiles per group.
int64_t tile_bound(const Ctx& c, int stage, int64_t N, int64_t T) {
  int nt[6], big_bm, med_bm, small_bm;
  tiling(c, nt, &big_bm, &med_bm, &small_bm);
  const int64_t E = c.cfg.n_experts, S = c.cfg.n_shared, G = E + S;
  const int64_t big_rows = N / big_bm + std::min<int64_t>(E, N) + S * ((T + big_bm - 1) / big_bm);
  const int* ns = nt + 3 * stage;
  return big_rows * ns[0] + (small_bm ? G * (2 * (int64_t)ns[1] + ns[2]) : 0);
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

bool layout(Ctx& c) {
  const aep_config& g = c.cfg;
  const int64_t L = g.n_layers, E = g.n_experts, S = g.n_shared, T = g.max_tokens_per_layer,
                k = g.top_k, d = g.d_model, f = g.d_ffn;
  const int64_t N = T * k;
  const int64_t xrows = N + (S ? T : 0);
  const int64_t hrows = N + S * T;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align256(o + bytes);
    return at;
  };
  c.off_err = take(256);
  c.off_depth = take(sizeof(int32_t) * L * 2 * E);
  if (g.act_dtype == AEP_BF16) c.off_splitcnt = take(sizeof(int32_t) * kSplitCounters);
  c.off_grppre = take(sizeof(int32_t) * (E + 1));
  c.off_q = take(sizeof(QEntry) * L * E * T);
  c.off_tokrow = take(sizeof(void*) * L * T);
  c.off_wtab = take(sizeof(WeightDesc) * L * c.G);
  c.off_ridx = take(sizeof(int32_t) * N);
  c.off_rw = take(sizeof(float) * N);
  c.off_rrank = take(sizeof(int32_t) * N);
  c.off_blockcnt = take(sizeof(int32_t) * ((T + kRouteTokens - 1) / kRouteTokens) * E);
  c.off_counts = take(sizeof(int32_t) * c.G);
  c.off_offsets = take(sizeof(int32_t) * (c.G + 1));
  c.off_groups = take(sizeof(GroupDesc) * c.G);
  c.off_tiles = take(sizeof(int32_t) * 6);
  c.tile_cap = std::max(tile_bound(c, 0, N, T), tile_bound(c, 1, N, T));
  c.off_tilegrp = take(sizeof(int32_t) * 2 * c.tile_cap);
  c.off_xp = take((size_t)xrows * d * c.esz);
  c.off_rowtok = take(sizeof(int32_t) * N);
  c.off_roww = take(sizeof(float) * N);
  c.off_pos = take(sizeof(int32_t) * N);
  c.off_posw = take(sizeof(float) * N);
  c.off_h = take((size_t)hrows * f * c.esz);
  if (g.act_dtype == AEP_BF16) {
    c.split_bytes = kSplitBytes;
    c.off_split = take(c.split_bytes);
  }
  if (g.token_pool) {
    c.off_pool = take(sizeof(float) * L * T * d);
    c.off_live = take(sizeof(int32_t) * L * T);
    c.off_pend = take(sizeof(int32_t) * L * T);
  }
  c.ws_need = o;
  return true;
}

Ctx* as_ctx(aep_ctx* p) { return p; }
const Ctx* as_ctx(const aep_ctx* p) { return p; }
hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

aep_status dev(hipError_t e) { return e == hipSuccess ? AEP_OK : AEP_ERR_DEVICE; }

// The workspace of aep_bind_static_workspace: one array per GPU, allocated
// with the code object and held until the process ends.  In host code its
// name is only a stand-in; its device address comes from hipGetSymbolAddress
// (looked up once per device, with that device current) and is the only
// handle host code ever passes on.
static __device__ __align__(256) unsigned char scratch[AEP_STATIC_WORKSPACE_BYTES];

struct StaticScratch {
  std::mutex mu;
  std::vector<char*> ptr;     // per device: address of `scratch` there (nullptr: not looked up yet)
  std::vector<uint64_t> gen;  // per device: incremented by every binding
};
StaticScratch& static_scratch() {
  static StaticScratch s;
  return s;
}

// A workspace is bound, and, if it is the static one, no other context has
// bound it since.
bool ws_bound(const Ctx* c) {
  if (!c->ws) return false;
  if (!c->ws_static) return true;
  StaticScratch& s = static_scratch();
  std::lock_guard<std::mutex> g(s.mu);
  return (size_t)c->device < s.gen.size() && s.gen[c->device] == c->static_gen;
}

// Initialise ws (the caller's allocation or the static array) on stream s and
// reset every queue of c.
aep_status bind(Ctx* c, char* ws, int devid, hipStream_t s) {
  int ncu = 0;
  if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, devid) != hipSuccess)
    return AEP_ERR_DEVICE;
  // clear the error flag and launch counter, every depth counter and the weight tables
  if (hipMemsetAsync(ws + c->off_err, 0, c->off_q - c->off_err, s) != hipSuccess) return AEP_ERR_DEVICE;
  if (hipMemsetAsync(ws + c->off_wtab, 0, sizeof(WeightDesc) * c->cfg.n_layers * c->G, s) != hipSuccess)
    return AEP_ERR_DEVICE;
  if (c->cfg.token_pool && hipMemsetAsync(ws + c->off_pool, 0, c->ws_need - c->off_pool, s) != hipSuccess)
    return AEP_ERR_DEVICE;
  if (hipStreamSynchronize(s) != hipSuccess) return AEP_ERR_DEVICE;
  c->ws = ws;
  c->ws_static = false;
  c->device = devid;
  c->num_cu = ncu > 0 ? ncu : 1;
  for (auto& l : c->layers) {
    l.clear();
    l.cur = 0;
    std::fill(l.have_w.begin(), l.have_w.end(), 0);
  }
  c->batch_out = false;
  c->batch_expert = false;
  std::fill(c->wtab_host.begin(), c->wtab_host.end(), WeightDesc{});
  return AEP_OK;
}


}  // namespace

extern "C" {

const char* aep_status_string(aep_status s) {
  switch (s) {
    case AEP_OK: return "AEP_OK";
    case AEP_ERR_INVALID_ARG: return "AEP_ERR_INVALID_ARG";
    case AEP_ERR_CAPACITY: return "AEP_ERR_CAPACITY";
    case AEP_ERR_EMPTY: return "AEP_ERR_EMPTY";
    case AEP_ERR_STATE: return "AEP_ERR_STATE";
    case AEP_ERR_DEVICE: return "AEP_ERR_DEVICE";
    case AEP_ERR_UNSUPPORTED: return "AEP_ERR_UNSUPPORTED";
  }
  return "AEP_ERR_UNKNOWN";
}

aep_status aep_create(const aep_config* cfg, aep_ctx** out) {
  if (!cfg || !out) return AEP_ERR_INVALID_ARG;
  const aep_config& g = *cfg;
  if (g.n_layers < 1 || g.n_experts < 1 || g.n_shared < 0 ||
      g.n_experts + g.n_shared > kMaxGroups)
    return AEP_ERR_INVALID_ARG;
  if (g.d_model < 64 || g.d_ffn < 64 || g.d_model % 64 || g.d_ffn % 64) return AEP_ERR_UNSUPPORTED;
  if (g.top_k < 1 || g.top_k > g.n_experts || g.top_k > kMaxTopK) return AEP_ERR_INVALID_ARG;
  if (g.renorm != 0 && g.renorm != 1) return AEP_ERR_INVALID_ARG;
  if (g.max_tokens_per_layer < 1 || g.max_tokens_per_layer > kTokenMask) return AEP_ERR_INVALID_ARG;
  if (g.token_pool != 0 && g.token_pool != 1) return AEP_ERR_INVALID_ARG;
  if (g.token_pool && g.n_shared > 0) return AEP_ERR_UNSUPPORTED;
  const bool f32 = g.act_dtype == AEP_F32 && g.w_dtype == AEP_F32;
  const bool bf = g.act_dtype == AEP_BF16 && (g.w_dtype == AEP_BF16 || g.w_dtype == AEP_FP8_E4M3);
  if (!f32 && !bf) {
    const bool known = (g.act_dtype >= 0 && g.act_dtype <= 2) && (g.w_dtype >= 0 && g.w_dtype <= 2);
    return known ? AEP_ERR_UNSUPPORTED : AEP_ERR_INVALID_ARG;
  }
  // The bf16 / fp8 FFN kernels address one group's activation rows (at most
  // max_tokens_per_layer rows of d or f elements) and one weight matrix
  // through buffer resources: 32-bit byte offsets and sizes.
  if (bf) {
    const uint64_t lim = 1ull << 32;
    const uint64_t kmax = (uint64_t)std::max(g.d_model, g.d_ffn);
    if ((uint64_t)g.max_tokens_per_layer * kmax * 2 >= lim || (uint64_t)g.d_model * g.d_ffn * 2 >= lim)
      return AEP_ERR_UNSUPPORTED;
  }
  Ctx* c = new (std::nothrow) Ctx();
  if (!c) return AEP_ERR_CAPACITY;
  c->cfg = g;
  c->G = g.n_experts + g.n_shared;
  c->esz = g.act_dtype == AEP_F32 ? 4 : 2;
  layout(*c);
  c->layers.resize(g.n_layers);
  for (auto& l : c->layers) {
    l.bound.assign(g.n_experts, 0);
    l.have_w.assign(c->G, 0);
  }
  c->wtab_host.assign((size_t)g.n_layers * c->G, WeightDesc{});
  *out = c;
  return AEP_OK;
}

aep_status aep_destroy(aep_ctx* ctx) {
  delete as_ctx(ctx);
  return AEP_OK;
}

aep_status aep_workspace_size(const aep_ctx* ctx, size_t* bytes) {
  if (!ctx || !bytes) return AEP_ERR_INVALID_ARG;
  *bytes = as_ctx(ctx)->ws_need;
  return AEP_OK;
}

aep_status aep_bind_workspace(aep_ctx* ctx, void* d_ws, size_t bytes, void* stream) {
  Ctx* c = as_ctx(ctx);
  if (!c || !d_ws) return AEP_ERR_INVALID_ARG;
  if (reinterpret_cast<uintptr_t>(d_ws) & 255) return AEP_ERR_INVALID_ARG;
  if (bytes < c->ws_need) return AEP_ERR_CAPACITY;
  if (c->batch_out && ws_bound(c)) return AEP_ERR_STATE;
  int devid = -1;
  if (hipGetDevice(&devid) != hipSuccess) return AEP_ERR_DEVICE;
  return bind(c, reinterpret_cast<char*>(d_ws), devid, as_stream(stream));
}

aep_status aep_bind_static_workspace(aep_ctx* ctx, void* stream) {
  Ctx* c = as_ctx(ctx);
  if (!c) return AEP_ERR_INVALID_ARG;
  if (c->ws_need > AEP_STATIC_WORKSPACE_BYTES) return AEP_ERR_CAPACITY;
  if (c->batch_out && ws_bound(c)) return AEP_ERR_STATE;
  int devid = -1;
  if (hipGetDevice(&devid) != hipSuccess || devid < 0) return AEP_ERR_DEVICE;
  StaticScratch& ss = static_scratch();
  char* base = nullptr;
  {
    std::lock_guard<std::mutex> g(ss.mu);
    if ((size_t)devid >= ss.ptr.size()) {
      ss.ptr.resize((size_t)devid + 1, nullptr);
      ss.gen.resize((size_t)devid + 1, 0);
    }
    if (!ss.ptr[devid]) {
      void* p = nullptr;
      if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return AEP_ERR_DEVICE;
      ss.ptr[devid] = reinterpret_cast<char*>(p);
    }
    base = ss.ptr[devid];
  }
  const aep_status st = bind(c, base, devid, as_stream(stream));
  if (st != AEP_OK) return st;
  std::lock_guard<std::mutex> g(ss.mu);
  c->ws_static = true;
  c->static_gen = ++ss.gen[devid];
  return AEP_OK;
}

aep_status aep_set_expert_weights(aep_ctx* ctx, int32_t layer, int32_t expert, const void* w_gate,
                                  const void* w_up, const void* w_down, const void* scale_gate_up,
                                  const void* scale_down, void* stream) {
  Ctx* c = as_ctx(ctx);
  if (!c) return AEP_ERR_INVALID_ARG;
  if (!ws_bound(c)) return AEP_ERR_STATE;
  if (layer < 0 || layer >= c->cfg.n_layers || expert < 0 || expert >= c->G) return AEP_ERR_INVALID_ARG;
  if (!w_gate || !w_up || !w_down) return AEP_ERR_INVALID_ARG;
  const bool fp8 = c->cfg.w_dtype == AEP_FP8_E4M3;
  if (fp8 != (scale_gate_up != nullptr) || fp8 != (scale_down != nullptr)) return AEP_ERR_INVALID_ARG;
  WeightDesc& w = c->wtab_host[(size_t)layer * c->G + expert];
  w.gate = w_gate;
  w.up = w_up;
  w.down = w_down;
  w.s_gu = reinterpret_cast<const uint16_t*>(scale_gate_up);
  w.s_down = reinterpret_cast<const uint16_t*>(scale_down);
  w.pad = nullptr;
  hipStream_t s = as_stream(stream);
  if (hipMemcpyAsync(c->wtab(layer) + expert, &w, sizeof(WeightDesc), hipMemcpyHostToDevice, s) != hipSuccess)
    return AEP_ERR_DEVICE;
  if (hipStreamSynchronize(s) != hipSuccess) return AEP_ERR_DEVICE;
  c->layers[layer].have_w[expert] = 1;
  return AEP_OK;
}

static aep_status route_common(Ctx* c, int32_t layer, const void* x, const float* logits, int32_t T,
                               const int32_t* token_ids, int32_t* idx_out, float* w_out, void* stream) {
  if (!c) return AEP_ERR_INVALID_ARG;
  if (!ws_bound(c)) return AEP_ERR_STATE;
  if (layer < 0 || layer >= c->cfg.n_layers || T < 0) return AEP_ERR_INVALID_ARG;
  if (token_ids && !c->cfg.token_pool) return AEP_ERR_UNSUPPORTED;
  LayerState& L = c->layers[layer];
  const bool want_pool = token_ids != nullptr;
  if (L.rows > 0 && L.pool != want_pool) return AEP_ERR_STATE;
  if (T == 0) return AEP_OK;
  if (!x || !logits) return AEP_ERR_INVALID_ARG;
  const int E = c->cfg.n_experts, k = c->cfg.top_k;
  if (E > kMaxRouteExperts) return AEP_ERR_UNSUPPORTED;
  int64_t ub = 0;
  for (int e = 0; e < E; ++e) ub = std::max(ub, L.bound[e]);
  if (ub + T > c->tmax() || L.rows + (int64_t)T * k > c->row_cap()) return AEP_ERR_CAPACITY;
  if (!want_pool && (int64_t)L.tokens + T > c->tmax()) return AEP_ERR_CAPACITY;
  hipStream_t s = as_stream(stream);
  int32_t* ridx = c->at<int32_t>(c->off_ridx);
  float* rw = c->at<float>(c->off_rw);
  int32_t* rrank = c->at<int32_t>(c->off_rrank);
  int32_t* bcnt = c->at<int32_t>(c->off_blockcnt);
  hipError_t e1 = launch_route(logits, T, E, k, c->cfg.renorm, ridx, rw, rrank, bcnt, idx_out, w_out,
                               c->depth(layer, L.cur), c->depth(layer, L.cur ^ 1), c->route_done(), c->err(), s);
  if (e1 != hipSuccess) return AEP_ERR_DEVICE;
  const int64_t row_bytes = (int64_t)c->cfg.d_model * c->esz;
  hipError_t e2 = launch_append(ridx, rw, rrank, bcnt, T, E, k, reinterpret_cast<const char*>(x), row_bytes,
                                want_pool ? 0 : L.tokens, c->depth(layer, L.cur), c->depth(layer, L.cur ^ 1),
                                c->q(layer), c->tmax(), c->tokrow(layer), token_ids,
                                (int)c->tmax(), want_pool ? c->live(layer) : nullptr,
                                want_pool ? c->pend(layer) : nullptr, c->err(), s);
  if (e2 != hipSuccess) return AEP_ERR_DEVICE;
  L.cur ^= 1;
  if (!want_pool) L.tokens += T;
  L.pool = want_pool;
  L.rows += (int64_t)T * k;
  for (int e = 0; e < E; ++e) L.bound[e] += T;
  return AEP_OK;
}

aep_status aep_route_enqueue(aep_ctx* ctx, int32_t layer, const void* x, const float* logits, int32_t T,
                             int32_t* idx_out, float* w_out, void* stream) {
  return route_common(as_ctx(ctx), layer, x, logits, T, nullptr, idx_out, w_out, stream);
}

aep_status aep_route_enqueue_ids(aep_ctx* ctx, int32_t layer, const void* x, const float* logits,
                                 int32_t T, const int32_t* token_ids, int32_t* idx_out, float* w_out,
                                 void* stream) {
  if (T > 0 && !token_ids) return AEP_ERR_INVALID_ARG;
  Ctx* c = as_ctx(ctx);
  if (c && T == 0 && !c->cfg.token_pool) return AEP_ERR_UNSUPPORTED;
  return route_common(c, layer, x, logits, T, T > 0 ? token_ids : nullptr, idx_out, w_out, stream);
}

aep_status aep_enqueue_rows(aep_ctx* ctx, int32_t layer, int32_t expert, const void* rows,
                            const int32_t* token_ids, const int32_t* slots, const float* gate_w,
                            int32_t n, int32_t n_tokens, void* stream) {
  Ctx* c = as_ctx(ctx);
  if (!c) return AEP_ERR_INVALID_ARG;
  if (!ws_bound(c)) return AEP_ERR_STATE;
  if (layer < 0 || layer >= c->cfg.n_layers || expert < 0 || expert >= c->cfg.n_experts || n < 0)
    return AEP_ERR_INVALID_ARG;
  if (c->cfg.n_shared > 0) return AEP_ERR_UNSUPPORTED;
  LayerState& L = c->layers[layer];
  if (L.rows > 0 && L.pool) return AEP_ERR_STATE;
  if (n == 0) return AEP_OK;
  if (!rows || !token_ids || !gate_w || n_tokens < 1) return AEP_ERR_INVALID_ARG;
  if ((int64_t)n_tokens > c->tmax() || L.bound[expert] + n > c->tmax() || L.rows + n > c->row_cap())
    return AEP_ERR_CAPACITY;
  hipStream_t s = as_stream(stream);
  const int64_t row_bytes = (int64_t)c->cfg.d_model * c->esz;
  hipError_t e = launch_enqueue_rows(reinterpret_cast<const char*>(rows), row_bytes, token_ids, slots,
                                     gate_w, n, n_tokens, c->cfg.top_k, expert, c->cfg.n_experts,
                                     c->depth(layer, L.cur), c->depth(layer, L.cur ^ 1), c->q(layer),
                                     c->tmax(), c->err(), s);
  if (e != hipSuccess) return AEP_ERR_DEVICE;
  L.cur ^= 1;
  L.pool = false;
  L.tokens = std::max(L.tokens, n_tokens);
  L.rows += n;
  L.bound[expert] += n;
  return AEP_OK;
}

aep_status aep_enqueue_rows_grouped(aep_ctx* ctx, int32_t layer, const int32_t* h_counts, const void* rows,
                                    const int32_t* token_ids, const int32_t* slots, const float* gate_w,
                                    int32_t n_tokens, void* stream) {
  Ctx* c = as_ctx(ctx);
  if (!c || !h_counts) return AEP_ERR_INVALID_ARG;
  if (!ws_bound(c)) return AEP_ERR_STATE;
  if (layer < 0 || layer >= c->cfg.n_layers) return AEP_ERR_INVALID_ARG;
  if (c->cfg.n_shared > 0) return AEP_ERR_UNSUPPORTED;
  const int E = c->cfg.n_experts;
  std::vector<int32_t> pre(E + 1, 0);
  int64_t total = 0;
  for (int e = 0; e < E; ++e) {
    if (h_counts[e] < 0) return AEP_ERR_INVALID_ARG;
    total += h_counts[e];
    if (total > INT32_MAX) return AEP_ERR_CAPACITY;
    pre[e + 1] = (int32_t)total;
  }
  LayerState& L = c->layers[layer];
  if (L.rows > 0 && L.pool) return AEP_ERR_STATE;
  if (total == 0) return AEP_OK;
  if (!rows || !token_ids || !gate_w || n_tokens < 1) return AEP_ERR_INVALID_ARG;
  if ((int64_t)n_tokens > c->tmax() || L.rows + total > c->row_cap()) return AEP_ERR_CAPACITY;
  for (int e = 0; e < E; ++e)
    if (L.bound[e] + h_counts[e] > c->tmax()) return AEP_ERR_CAPACITY;
  hipStream_t s = as_stream(stream);
  int32_t* dpre = c->at<int32_t>(c->off_grppre);
  if (hipMemcpyAsync(dpre, pre.data(), sizeof(int32_t) * (E + 1), hipMemcpyHostToDevice, s) != hipSuccess)
    return AEP_ERR_DEVICE;
  const int64_t row_bytes = (int64_t)c->cfg.d_model * c->esz;
  hipError_t e = launch_enqueue_grouped(reinterpret_cast<const char*>(rows), row_bytes, token_ids, slots, gate_w,
                                        (int)total, n_tokens, c->cfg.top_k, E, dpre, c->depth(layer, L.cur),
                                        c->depth(layer, L.cur ^ 1), c->q(layer), c->tmax(), c->err(), s);
  if (e != hipSuccess) return AEP_ERR_DEVICE;
  L.cur ^= 1;
  L.pool = false;
  L.tokens = std::max(L.tokens, n_tokens);
  L.rows += total;
  for (int ex = 0; ex < E; ++ex) L.bound[ex] += h_counts[ex];
  return AEP_OK;
}

aep_status aep_queue_depth(const aep_ctx* ctx, int32_t layer, int64_t* tokens, int64_t* rows) {
  const Ctx* c = as_ctx(ctx);
  if (!c || layer < 0 || layer >= c->cfg.n_layers) return AEP_ERR_INVALID_ARG;
  if (tokens) *tokens = c->layers[layer].tokens;
  if (rows) *rows = c->layers[layer].rows;
  return AEP_OK;
}

aep_status aep_expert_counts(aep_ctx* ctx, int32_t layer, int32_t* h_counts, void* stream) {
  Ctx* c = as_ctx(ctx);
  if (!c || !h_counts || layer < 0 || layer >= c->cfg.n_layers) return AEP_ERR_INVALID_ARG;
  if (!ws_bound(c)) return AEP_ERR_STATE;
  hipStream_t s = as_stream(stream);
  if (hipMemcpyAsync(h_counts, c->depth(layer, c->layers[layer].cur), sizeof(int32_t) * c->cfg.n_experts,
                     hipMemcpyDeviceToHost, s) != hipSuccess)
    return AEP_ERR_DEVICE;
  return dev(hipStreamSynchronize(s));
}

aep_status aep_pick_layer(const aep_ctx* ctx, int32_t policy, double delta, int32_t lookahead,
                          int32_t* layer) {
  const Ctx* c = as_ctx(ctx);
  if (!c || !layer) return AEP_ERR_INVALID_ARG;
  if (policy < AEP_POLICY_MTFS || policy > AEP_POLICY_DEFRAG) return AEP_ERR_INVALID_ARG;
  if (policy == AEP_POLICY_DEFRAG && (lookahead < 0 || !(delta >= 0.0) || !std::isfinite(delta)))
    return AEP_ERR_INVALID_ARG;
  std::vector<int64_t> rows(c->layers.size());
  for (size_t b = 0; b < rows.size(); ++b) rows[b] = c->layers[b].rows;
  int pb = -1;
  if (!pick_block(rows.data(), (int)rows.size(), policy, delta, lookahead, &pb)) return AEP_ERR_EMPTY;
  *layer = pb;
  return AEP_OK;
}

aep_status aep_rebatch(aep_ctx* ctx, int32_t layer, aep_batch* out, void* stream) {
  Ctx* c = as_ctx(ctx);
  if (!c || !out || layer < 0 || layer >= c->cfg.n_layers) return AEP_ERR_INVALID_ARG;
  if (!ws_bound(c) || c->batch_out) return AEP_ERR_STATE;
  LayerState& L = c->layers[layer];
  if (L.rows > 0 && L.pool) return AEP_ERR_STATE;  // pool-mode layers drain one expert at a time
  if (L.rows == 0 && !(c->cfg.n_shared > 0 && L.tokens > 0)) return AEP_ERR_EMPTY;
  for (int g = 0; g < c->G; ++g)
    if (!L.have_w[g]) return AEP_ERR_STATE;
  int nt[6], big_bm, med_bm, small_bm;
  tiling(*c, nt, &big_bm, &med_bm, &small_bm);
  hipStream_t s = as_stream(stream);
  const int E = c->cfg.n_experts, S = c->cfg.n_shared, k = c->cfg.top_k;
  int32_t* counts = c->at<int32_t>(c->off_counts);
  int32_t* offsets = c->at<int32_t>(c->off_offsets);
  int32_t* pos = c->at<int32_t>(c->off_pos);
  float* posw = c->at<float>(c->off_posw);
  if (launch_plan(E, S, L.tokens, k, -1, c->depth(layer, L.cur), c->depth(layer, L.cur ^ 1), counts, offsets,
                  c->at<GroupDesc>(c->off_groups), c->at<int32_t>(c->off_tiles), nt, big_bm, med_bm,
                  small_bm, c->num_cu, c->at<int32_t>(c->off_tilegrp), c->tile_cap, pos, posw, s) != hipSuccess)
    return AEP_ERR_DEVICE;
  const int64_t row_bytes = (int64_t)c->cfg.d_model * c->esz;
  if (launch_gather(c->q(layer), c->tmax(), offsets, E, L.rows, L.tokens, S > 0, c->tokrow(layer),
                    c->at<char>(c->off_xp), row_bytes, c->at<int32_t>(c->off_rowtok), c->at<float>(c->off_roww),
                    pos, posw, k, c->err(), s) != hipSuccess)
    return AEP_ERR_DEVICE;
  c->epoch += 1;
  c->batch_out = true;
  c->batch_expert = false;
  c->batch_layer = layer;
  out->layer = layer;
  out->n_tokens = L.tokens;
  out->n_routed = L.rows;
  out->n_rows = L.rows + (int64_t)S * L.tokens;
  out->epoch = c->epoch;
  out->x_perm = c->ws + c->off_xp;
  out->counts = counts;
  out->offsets = offsets;
  out->row_token = c->at<int32_t>(c->off_rowtok);
  out->row_weight = c->at<float>(c->off_roww);
  out->token_pos = pos;
  out->token_weight = posw;
  L.clear();
  return AEP_OK;
}

aep_status aep_rebatch_expert(aep_ctx* ctx, int32_t layer, int32_t expert, aep_batch* out, void* stream) {
  Ctx* c = as_ctx(ctx);
  if (!c || !out || layer < 0 || layer >= c->cfg.n_layers || expert < 0 || expert >= c->cfg.n_experts)
    return AEP_ERR_INVALID_ARG;
  if (!c->cfg.token_pool) return AEP_ERR_UNSUPPORTED;
  if (!ws_bound(c) || c->batch_out) return AEP_ERR_STATE;
  LayerState& L = c->layers[layer];
  if (L.rows > 0 && !L.pool) return AEP_ERR_STATE;
  const int64_t nb = std::min(L.bound[expert], L.rows);
  if (nb == 0) return AEP_ERR_EMPTY;
  if (!L.have_w[expert]) return AEP_ERR_STATE;
  int nt[6], big_bm, med_bm, small_bm;
  tiling(*c, nt, &big_bm, &med_bm, &small_bm);
  hipStream_t s = as_stream(stream);
  const int E = c->cfg.n_experts, k = c->cfg.top_k;
  int32_t* counts = c->at<int32_t>(c->off_counts);
  int32_t* offsets = c->at<int32_t>(c->off_offsets);
  if (launch_plan(E, 0, 0, k, expert, c->depth(layer, L.cur), c->depth(layer, L.cur ^ 1), counts, offsets,
                  c->at<GroupDesc>(c->off_groups),
                  c->at<int32_t>(c->off_tiles), nt, big_bm, med_bm, small_bm, c->num_cu,
                  c->at<int32_t>(c->off_tilegrp), c->tile_cap, nullptr, nullptr, s) != hipSuccess)
    return AEP_ERR_DEVICE;
  const int64_t row_bytes = (int64_t)c->cfg.d_model * c->esz;
  if (launch_gather(c->q(layer), c->tmax(), offsets, E, nb, 0, 0, c->tokrow(layer), c->at<char>(c->off_xp),
                    row_bytes, c->at<int32_t>(c->off_rowtok), c->at<float>(c->off_roww), nullptr, nullptr, k,
                    c->err(), s) != hipSuccess)
    return AEP_ERR_DEVICE;
  c->epoch += 1;
  c->batch_out = true;
  c->batch_expert = true;
  c->batch_layer = layer;
  out->layer = layer;
  out->n_tokens = 0;
  out->n_routed = nb;
  out->n_rows = nb;
  out->epoch = c->epoch;
  out->x_perm = c->ws + c->off_xp;
  out->counts = counts;
  out->offsets = offsets;
  out->row_token = c->at<int32_t>(c->off_rowtok);
  out->row_weight = c->at<float>(c->off_roww);
  out->token_pos = nullptr;
  out->token_weight = nullptr;
  L.bound[expert] = 0;
  int64_t sum = 0;
  for (int e = 0; e < E; ++e) sum += L.bound[e];
  L.rows = std::min(L.rows, sum);
  if (L.rows == 0) L.clear();
  return AEP_OK;
}

static aep_status check_batch(const Ctx* c, const aep_batch* b) {
  if (!c || !b) return AEP_ERR_INVALID_ARG;
  if (!ws_bound(c)) return AEP_ERR_STATE;
  if (!c->batch_out || b->epoch != c->epoch || b->layer != c->batch_layer) return AEP_ERR_STATE;
  return AEP_OK;
}

static aep_status ffn_stage(Ctx* c, const aep_batch* batch, int stage, void* y, void* stream) {
  aep_status st = check_batch(c, batch);
  if (st != AEP_OK) return st;
  if (stage == 1 && !y) return AEP_ERR_INVALID_ARG;
  const int64_t mt = tile_bound(*c, stage, batch->n_routed, batch->n_tokens);
  if (mt > INT32_MAX || mt > c->tile_cap) return AEP_ERR_UNSUPPORTED;
  return dev(launch_ffn(stage, c->cfg.act_dtype, c->cfg.w_dtype, c->at<GroupDesc>(c->off_groups),
                        c->wtab(batch->layer), c->G, c->at<int32_t>(c->off_tiles),
                        c->at<int32_t>(c->off_tilegrp) + stage * c->tile_cap,
                        c->split_bytes ? c->at<float>(c->off_split) : nullptr,
                        c->split_bytes ? c->at<int32_t>(c->off_splitcnt) : nullptr, (int64_t)c->split_bytes, (int)mt,
                        c->ws + c->off_xp, c->ws + c->off_h, y, c->cfg.d_model, c->cfg.d_ffn, c->num_cu,
                        c->clk, c->clk_n, as_stream(stream)));
}

aep_status aep_set_clock_probe(aep_ctx* ctx, uint64_t* d_buf, int32_t n_pairs) {
  Ctx* c = as_ctx(ctx);
  if (!c) return AEP_ERR_INVALID_ARG;
  const bool on = d_buf != nullptr && n_pairs > 0;
  c->clk = on ? reinterpret_cast<unsigned long long*>(d_buf) : nullptr;
  c->clk_n = on ? n_pairs : 0;
  return AEP_OK;
}

aep_status aep_expert_gate_up(aep_ctx* ctx, const aep_batch* batch, void* stream) {
  return ffn_stage(as_ctx(ctx), batch, 0, nullptr, stream);
}

aep_status aep_expert_down(aep_ctx* ctx, const aep_batch* batch, void* y, void* stream) {
  return ffn_stage(as_ctx(ctx), batch, 1, y, stream);
}

aep_status aep_expert_ffn(aep_ctx* ctx, const aep_batch* batch, void* y, void* stream) {
  if (!y) return check_batch(as_ctx(ctx), batch) == AEP_OK ? AEP_ERR_INVALID_ARG : check_batch(as_ctx(ctx), batch);
  aep_status st = ffn_stage(as_ctx(ctx), batch, 0, nullptr, stream);
  if (st != AEP_OK) return st;
  return ffn_stage(as_ctx(ctx), batch, 1, y, stream);
}

aep_status aep_combine(aep_ctx* ctx, const aep_batch* batch, const void* y, void* out, void* stream) {
  Ctx* c = as_ctx(ctx);
  aep_status st = check_batch(c, batch);
  if (st != AEP_OK) return st;
  if (c->batch_expert) return AEP_ERR_STATE;
  if (!y || !out) return AEP_ERR_INVALID_ARG;
  return dev(launch_combine(c->cfg.act_dtype, y, batch->n_routed, batch->n_tokens, c->cfg.n_shared,
                            c->cfg.top_k, batch->token_pos, batch->token_weight, out, c->cfg.d_model,
                            as_stream(stream)));
}

aep_status aep_pool_accumulate(aep_ctx* ctx, const aep_batch* batch, const void* y, void* stream) {
  Ctx* c = as_ctx(ctx);
  aep_status st = check_batch(c, batch);
  if (st != AEP_OK) return st;
  if (!c->batch_expert) return AEP_ERR_STATE;
  if (!y) return AEP_ERR_INVALID_ARG;
  return dev(launch_pool_accumulate(c->cfg.act_dtype, y, batch->n_routed, batch->offsets, c->cfg.n_experts,
                                    batch->row_token, batch->row_weight, c->pool(batch->layer),
                                    c->pend(batch->layer), c->cfg.d_model, as_stream(stream)));
}

aep_status aep_pool_release(aep_ctx* ctx, int32_t layer, void* out, int32_t* ready, void* stream) {
  Ctx* c = as_ctx(ctx);
  if (!c || layer < 0 || layer >= c->cfg.n_layers) return AEP_ERR_INVALID_ARG;
  if (!c->cfg.token_pool) return AEP_ERR_UNSUPPORTED;
  if (!ws_bound(c)) return AEP_ERR_STATE;
  if (!out) return AEP_ERR_INVALID_ARG;
  return dev(launch_pool_release(c->cfg.act_dtype, c->pool(layer), c->live(layer), c->pend(layer),
                                 (int)c->tmax(), out, ready, c->cfg.d_model, as_stream(stream)));
}

aep_status aep_release_batch(aep_ctx* ctx, aep_batch* batch) {
  Ctx* c = as_ctx(ctx);
  aep_status st = check_batch(c, batch);
  if (st != AEP_OK) return st;
  c->batch_out = false;
  c->batch_expert = false;
  c->batch_layer = -1;
  std::memset(batch, 0, sizeof(*batch));
  return AEP_OK;
}

aep_status aep_sync(aep_ctx* ctx, void* stream) {
  Ctx* c = as_ctx(ctx);
  if (!c) return AEP_ERR_INVALID_ARG;
  if (!ws_bound(c)) return AEP_ERR_STATE;
  if (hipStreamSynchronize(as_stream(stream)) != hipSuccess) return AEP_ERR_DEVICE;
  int32_t flag = 0;
  if (hipMemcpy(&flag, c->err(), sizeof(flag), hipMemcpyDeviceToHost) != hipSuccess) return AEP_ERR_DEVICE;
  if (flag != 0) {
    const int32_t zero = 0;
    if (hipMemcpy(c->err(), &zero, sizeof(zero), hipMemcpyHostToDevice) != hipSuccess) return AEP_ERR_DEVICE;
    return AEP_ERR_DEVICE;
  }
  return AEP_OK;
}

aep_status aep_fp8_e4m3_to_bf16(const uint8_t* codes, uint16_t* out, int64_t n, void* stream) {
  if (n < 0) return AEP_ERR_INVALID_ARG;
  if (n == 0) return AEP_OK;
  if (!codes || !out) return AEP_ERR_INVALID_ARG;
  return dev(launch_fp8_to_bf16(codes, out, n, as_stream(stream)));
}

}  // extern "C"
