/*
 * aep.h -- C ABI of libaep, the MI355X (gfx950) expert-layer hot path of
 * Asynchronous Expert Parallelism (AEP).
 *
 * The calls follow the paper's statement of the problem (Sec. 3.2, execution
 * engine): a receptor files arriving tokens under a LayerID = (block, expert)
 * queue (the "mu-queue"); when the GPU is free a scheduler picks a layer
 * (Sec. 3.4); the executor drains that layer's queues, merges the fragments
 * into one contiguous batch (re-batching), runs the experts, and the top-K
 * duplicates of each token are merged back with their gate weights (Sec. 3.2,
 * "Top-K support").  Token data stays on the GPU; queue metadata that the host
 * can know without a device sync (token and row totals) is kept on the host.
 *
 * Conventions for every entry point:
 *  - Every call returns an aep_status.  Argument, capacity and state errors
 *    are detected on the host before anything is launched and leave all state
 *    unchanged.  Launch failures return AEP_ERR_DEVICE.  Bad values that only
 *    the device can see (an out-of-range token id, a non-finite logit, two
 *    rows for one (token, slot)) set a device error flag and are reported as
 *    AEP_ERR_DEVICE by the next aep_sync; the offending value is clamped so
 *    that every memory access stays in bounds.  Nothing aborts or throws
 *    across the ABI.
 *  - "device pointer" arguments are HIP device allocations owned by the
 *    caller and only borrowed by the library; "host pointer" arguments are
 *    ordinary host memory.  All device work of a call is enqueued on the
 *    given stream (a hipStream_t; NULL is the legacy default stream), in
 *    stream order, and the call returns without waiting unless stated.
 *  - One host thread drives a context at a time.  Calls on one context must
 *    be ordered on one stream (or ordered by the caller across streams).
 *  - Matrices are row-major with the last dimension contiguous.  Weight
 *    matrices are stored out x in (the reduction dimension contiguous):
 *    W_gate, W_up [d_ffn][d_model], W_down [d_model][d_ffn].
 *  - Element formats: AEP_F32 = IEEE binary32; AEP_BF16 = bfloat16 (upper
 *    half of a binary32); AEP_FP8_E4M3 = OCP FP8 E4M3 ("e4m3fn": bias 7,
 *    largest finite 448, S.1111.111 is NaN, no infinities).
 */
#ifndef AEP_H_
#define AEP_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  AEP_OK = 0,
  AEP_ERR_INVALID_ARG = 1, /* a NULL/out-of-range argument or bad config      */
  AEP_ERR_CAPACITY = 2,    /* the queue or workspace cannot hold the request  */
  AEP_ERR_EMPTY = 3,       /* nothing queued (drain / pick)                   */
  AEP_ERR_STATE = 4,       /* call out of order (no workspace, stale batch...) */
  AEP_ERR_DEVICE = 5,      /* HIP error or device-detected bad input          */
  AEP_ERR_UNSUPPORTED = 6  /* valid but not implemented (shape, dtype combo)  */
} aep_status;

typedef enum { AEP_F32 = 0, AEP_BF16 = 1, AEP_FP8_E4M3 = 2 } aep_dtype;

/* Layer-pick policies (Sec. 3.4): most-tokens-first-serve, first-layer-first-
 * serve, and the defragging scheduler (Algorithm 1). */
typedef enum { AEP_POLICY_MTFS = 0, AEP_POLICY_FLFS = 1, AEP_POLICY_DEFRAG = 2 } aep_policy;

typedef struct {
  int32_t n_layers;    /* MoE layers (blocks) whose queues live in this context */
  int32_t n_experts;   /* routed experts per layer, E (routing needs E <= 64)   */
  int32_t n_shared;    /* shared experts per layer (see every token, weight 1)  */
  int32_t d_model;     /* d: multiple of 64                                      */
  int32_t d_ffn;       /* f: multiple of 64                                      */
  int32_t top_k;       /* k: slots per token, 1 <= k <= min(E, 8)               */
  int32_t renorm;      /* 1: gate weights renormalised over the k selected      */
  int32_t act_dtype;   /* aep_dtype of activations, H and outputs: F32 or BF16  */
  int32_t w_dtype;     /* aep_dtype of weights: F32 (with F32 act), BF16 or      */
                       /* FP8_E4M3 (with BF16 act)                               */
  int32_t max_tokens_per_layer; /* queue capacity: tokens a layer may hold     */
  int32_t token_pool;  /* 1: per-layer token pools for drains of single experts */
                       /* (aep_route_enqueue_ids ... aep_pool_release); adds    */
                       /* n_layers * max_tokens_per_layer * (4 d + 8) bytes of  */
                       /* workspace.  0: none.                                  */
} aep_config;

/* The library's context: one set of mu-queues (every layer), the expert
 * weight tables and the batch in flight.  Opaque; created by aep_create,
 * freed by aep_destroy, owned by the library. */
typedef struct aep_ctx aep_ctx;

/* A drained layer.  Filled by aep_rebatch; all pointers are device views into
 * the bound workspace and stay valid until aep_release_batch (or the next
 * aep_rebatch, which is refused while a batch is outstanding).
 *
 * Row space of the batch: rows [0, n_routed) are the routed rows, experts in
 * ascending id, each expert's queue in arrival order; when shared experts
 * exist, shared expert s owns rows [n_routed + s*n_tokens, ... + n_tokens),
 * one per token in id order.  n_rows = n_routed + n_shared * n_tokens. */
typedef struct {
  int32_t layer;
  int32_t n_tokens;          /* tokens of the layer (rows of the combine output)  */
  int64_t n_routed;          /* routed rows, sum of counts[0..E)                   */
  int64_t n_rows;            /* rows of y (routed + shared)                        */
  uint64_t epoch;            /* identifies the batch; stale handles are refused    */
  const void* x_perm;        /* [n_routed (+ n_tokens if shared)][d] act dtype:    */
                             /*   routed rows, then every token in id order       */
  const int32_t* counts;     /* [E + n_shared] rows per group                      */
  const int32_t* offsets;    /* [E + n_shared + 1] first row of each group         */
  const int32_t* row_token;  /* [n_routed] token id of each routed row             */
  const float* row_weight;   /* [n_routed] gate weight of each routed row          */
  const int32_t* token_pos;  /* [n_tokens][k] row of (token, slot), -1 if absent   */
  const float* token_weight; /* [n_tokens][k] gate weight of (token, slot), 0 if absent */
} aep_batch;

/* Human-readable name of a status (static string, never NULL). */
const char* aep_status_string(aep_status s);

/* Create a context for cfg (copied).  Validates the configuration; allocates
 * host state only.  *out receives the handle.  No device work.
 * AEP_ERR_UNSUPPORTED for a shape the kernels do not cover (d or f not a
 * multiple of 64; with BF16 activations, 2 * d * f bytes, or
 * 2 * max_tokens_per_layer * max(d, f) bytes, of 4 GiB or more). */
aep_status aep_create(const aep_config* cfg, aep_ctx** out);

/* Destroy a context (NULL is allowed).  Does not free the caller's workspace. */
aep_status aep_destroy(aep_ctx* ctx);

/* Bytes of device workspace this configuration needs (host only). */
aep_status aep_workspace_size(const aep_ctx* ctx, size_t* bytes);

/* Bind a caller-allocated device workspace of at least aep_workspace_size
 * bytes, 256-byte aligned, on the current HIP device.  Initialises it on
 * `stream` and waits for that.  Resets every queue.  The workspace holds the
 * mu-queues, weight tables, the batch buffers, the FFN intermediate and (bf16
 * activations) 32 MiB for the split-K partial sums of FFN launches with few
 * tiles. */
aep_status aep_bind_workspace(aep_ctx* ctx, void* d_ws, size_t bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): bind the
 * library's own static workspace instead of a caller allocation.  The array
 * holds AEP_STATIC_WORKSPACE_BYTES (96 MiB) on every GPU the library runs on,
 * comes with the code object and lives until the process ends; nothing is
 * allocated or freed by this call.  Otherwise as aep_bind_workspace: on the
 * current HIP device, initialised on `stream` (waits for it), every queue
 * reset, weights to be registered again.  AEP_ERR_CAPACITY (nothing changed)
 * if aep_workspace_size exceeds the maximum; AEP_ERR_STATE while a batch of
 * this context is outstanding.  All contexts bound this way on one GPU share
 * that GPU's array, which keeps what the last user left there: binding
 * another context takes the array over, and the earlier context's later
 * calls return AEP_ERR_STATE until it is bound again.  Work that two such
 * contexts enqueue so that it overlaps on the GPU (before the takeover, or
 * on different streams) races and corrupts both. */
#define AEP_STATIC_WORKSPACE_BYTES ((size_t)96 << 20)
aep_status aep_bind_static_workspace(aep_ctx* ctx, void* stream);

/* Register one expert's weights for a layer (pointers are borrowed and must
 * stay valid while the layer can run).  expert in [0, E) is routed; expert
 * in [E, E + n_shared) is shared expert expert - E.  Device pointers:
 *   w_gate, w_up [d_ffn][d_model], w_down [d_model][d_ffn] in w_dtype;
 *   for FP8 weights, scale_gate_up [2 * d_ffn] (gate channels, then up
 *   channels) and scale_down [d_model], bf16: W = code * scale per output
 *   channel.  Scales must be NULL for other weight types.
 * Copies the pointer table to the device on `stream` and waits for it. */
aep_status aep_set_expert_weights(aep_ctx* ctx, int32_t layer, int32_t expert, const void* w_gate,
                                  const void* w_up, const void* w_down, const void* scale_gate_up,
                                  const void* scale_down, void* stream);

/* Receptor + router for one arriving fragment of T tokens (Sec. 3.2):
 * routes each token on its gate logits (device, f32 [T][E]; top-k by logit,
 * larger first, equal logits -> lower expert id; weights = softmax
 * probabilities of the k selected, renormalised when cfg.renorm) and appends
 * one queue entry per (token, slot) to queue (layer, expert), in (token,
 * slot) order.  x (device, [T][d] act dtype) is NOT copied: entries refer to
 * its rows, so it must stay valid until this layer's aep_rebatch has run on
 * the stream.  Tokens get layer-local ids continuing the layer's count.
 * idx_out [T][k] int32 and w_out [T][k] f32 (device, may be NULL) receive
 * the routing.  T == 0 is a no-op.  AEP_ERR_CAPACITY if the layer could
 * exceed max_tokens_per_layer. */
aep_status aep_route_enqueue(aep_ctx* ctx, int32_t layer, const void* x, const float* logits, int32_t T,
                             int32_t* idx_out, float* w_out, void* stream);

/* Receptor for rows routed elsewhere: appends n rows to queue (layer,
 * expert) in order.  Device pointers: rows [n][d] act dtype (referenced,
 * not copied, as above), token_ids [n] int32 in [0, n_tokens), slots [n]
 * int32 in [0, k) (NULL: all 0), gate_w [n] f32.  The layer's token count
 * becomes max(current, n_tokens).  Not available on layers with shared
 * experts (AEP_ERR_UNSUPPORTED).  n == 0 is a no-op. */
aep_status aep_enqueue_rows(aep_ctx* ctx, int32_t layer, int32_t expert, const void* rows,
                            const int32_t* token_ids, const int32_t* slots, const float* gate_w,
                            int32_t n, int32_t n_tokens, void* stream);

/* Receptor for rows of several experts at once (e.g. one expert-parallel
 * receive buffer): rows [n][d] act dtype, grouped by expert in ascending
 * expert order, h_counts[e] (host, E entries, >= 0) of them for expert e,
 * n = sum of h_counts; token_ids, slots (NULL: all 0) and gate_w [n] as in
 * aep_enqueue_rows.  The queues end up exactly as after aep_enqueue_rows for
 * each expert in ascending order, in one launch.  The count prefix is copied
 * to the workspace from host memory (hipMemcpyAsync), so the call is not
 * meant for graph capture.  AEP_ERR_CAPACITY (nothing changed) if any
 * expert's queue or the layer would overflow; n == 0 is a no-op. */
aep_status aep_enqueue_rows_grouped(aep_ctx* ctx, int32_t layer, const int32_t* h_counts, const void* rows,
                                    const int32_t* token_ids, const int32_t* slots, const float* gate_w,
                                    int32_t n_tokens, void* stream);

/* Host-side queue totals of a layer (no device access). */
aep_status aep_queue_depth(const aep_ctx* ctx, int32_t layer, int64_t* tokens, int64_t* rows);

/* Per-expert queue depths of a layer copied to host memory h_counts [E];
 * synchronises `stream`. */
aep_status aep_expert_counts(aep_ctx* ctx, int32_t layer, int32_t* h_counts, void* stream);

/* Scheduler (Sec. 3.4): pick the next layer to drain from the host-side
 * queue totals rows(b) (no device access, no sync).  MTFS: most queued rows
 * (ties: lowest layer).  FLFS: lowest non-empty layer.  DEFRAG: Algorithm 1
 * at layer granularity -- a drain takes every expert of the layer and the
 * host knows only layer totals, so each queue of Algorithm 1 is replaced by
 * its layer's average rows(b) / n_experts and the score multiplied by
 * n_experts: score(b) = rows(b) + sum_{i=1..lookahead} rows((b+i) mod
 * n_layers) * delta^i over non-empty layers (ties: lowest).  delta >= 0 and
 * finite, lookahead >= 0 (AEP_ERR_INVALID_ARG otherwise).  AEP_ERR_EMPTY
 * (*layer untouched) when nothing is queued. */
aep_status aep_pick_layer(const aep_ctx* ctx, int32_t policy, double delta, int32_t lookahead,
                          int32_t* layer);

/* Scheduler over (block, expert) queues (Sec. 3.4, Algorithm 1), host only:
 * pick the queue to run next from a host table Q [n_blocks][n_experts] of
 * queued rows (row-major, every entry >= 0).
 *  MTFS:   the largest queue.
 *  FLFS:   the lowest block holding any row; its largest queue.
 *  DEFRAG: Algorithm 1: score(b, e) = Q[b][e] + sum_{i=1..lookahead}
 *          (sum_e' Q[(b+i) mod n_blocks][e'] / n_experts) * delta^i over the
 *          non-empty queues (delta >= 0, lookahead >= 0).
 * Ties go to the lowest (block, expert) in row-major order.  AEP_ERR_EMPTY
 * (outputs untouched) when every queue is empty. */
aep_status aep_sched_pick(const int64_t* Q, int32_t n_blocks, int32_t n_experts, int32_t policy,
                          double delta, int32_t lookahead, int32_t* block, int32_t* expert);

/* Discrete-event model of one expert runtime (Sec. 3.4 behaviour, Sec. 5
 * arrivals), host only.  One GPU hosts every expert of every block.  Request r
 * sends its first token to block 0 at arrival_us[r]; a token queued at block b
 * is routed to top_k distinct experts drawn from the integer popularity CDF
 * (one row per expert queue).  When the GPU is free and rows are queued (and
 * the time is before horizon_us) the policy picks one (block, expert) queue
 * (granularity 0, aep_sched_pick) or a whole block (granularity 1,
 * aep_pick_layer's scores over block totals) and drains it; the step takes
 * (non-empty experts) * cost_fixed_us + ceil(rows * cost_row_ns / 1000) us.
 * When it ends, each token whose last queued row of that block ran leaves:
 * the tokens that leave in one step are spread over n_frag attention ranks,
 * and each rank's fragment reaches the next block (after the last block:
 * block 0 with the request's next token, unless the request has produced
 * out_len[r] tokens and completes) attn_us + jitter later, jitter drawn in
 * [0, jitter_us].  Random choices use the SplitMix64 output function on
 * seed + stream * 0xD1B54A32D192ED03 + counter * 0x9E3779B97F4A7C15 (mod 2^64),
 * streams 1 routing (counter ((r * 2^20 + it) * 2^12 + block) * 2^12 + draw),
 * 2 fragment (counter (r * 2^20 + it) * 2^12 + block), 3 jitter (counter
 * step * 2^12 + rank); times are integer microseconds, so runs are exactly
 * reproducible.  All pointers are host memory owned by the caller. */
typedef struct {
  int32_t n_blocks;           /* N_B: 1..4096                                      */
  int32_t n_experts;          /* N_E experts per block: 1..4096                    */
  int32_t top_k;              /* 1..min(N_E, 64)                                   */
  int32_t n_frag;             /* attention ranks: 1..4096                          */
  int32_t granularity;        /* 0: (block, expert) queues; 1: whole blocks        */
  int32_t policy;             /* aep_policy                                        */
  double delta;               /* DEFRAG weight decay, >= 0                         */
  int32_t lookahead;          /* DEFRAG lookahead depth, >= 0                      */
  int32_t n_requests;         /* 0..2^20                                           */
  int64_t attn_us;            /* attention-stub latency, >= 1                      */
  int64_t jitter_us;          /* largest extra latency of a fragment, >= 0         */
  int64_t cost_fixed_us;      /* step cost per non-empty expert, >= 0              */
  int64_t cost_row_ns;        /* step cost per row, >= 0                           */
  int64_t horizon_us;         /* no step starts at or after this time              */
  uint64_t seed;
  const int64_t* arrival_us;  /* [n_requests], non-decreasing, >= 0                */
  const int32_t* out_len;     /* [n_requests], tokens per request, 1..2^20 - 1     */
  const int64_t* expert_cdf;  /* [n_experts], non-decreasing, last entry > 0       */
} aep_sim_config;

/* Optional per-step trace (arrays of `capacity` entries; steps beyond it are
 * counted in the summary but not recorded; block_rows_after may be NULL) and
 * per-request completion times (done_us [n_requests], -1 if not completed;
 * may be NULL). */
typedef struct {
  int64_t capacity;
  int64_t* t_start;            /* step start (us)                                 */
  int32_t* block;              /* block run                                       */
  int32_t* expert;             /* expert run, -1 when a whole block ran           */
  int64_t* rows;               /* rows drained                                    */
  int64_t* queued_after;       /* rows left in every queue after the drain        */
  int32_t* blocks_busy_after;  /* blocks holding any row after the drain          */
  int64_t* block_rows_after;   /* [capacity][n_blocks] rows queued per block after
                                  the drain (the queue-depth trace); may be NULL  */
  int64_t* done_us;
} aep_sim_trace;

typedef struct {
  int64_t steps;              /* expert steps run                                 */
  int64_t rows;               /* rows drained in total                            */
  int64_t busy_us;            /* sum of step durations                            */
  int64_t end_us;             /* time when the run stopped                        */
  int64_t token_passes;       /* (token, block) passes completed                  */
  int64_t requests_done;      /* requests that produced out_len tokens            */
  int64_t rows_queued_at_end; /* rows still queued when the run stopped           */
  int64_t recorded;           /* trace entries written                            */
} aep_sim_summary;

/* Run the model until no step can start (nothing queued and no arrival
 * pending, or the horizon reached).  trace may be NULL.  AEP_ERR_INVALID_ARG
 * on a bad config. */
aep_status aep_sim_run(const aep_sim_config* cfg, aep_sim_trace* trace, aep_sim_summary* out);

/* Executor, re-batch (Sec. 3.2): drain every queue of `layer` into one
 * contiguous batch -- per-expert counts and offsets, then a gather of every
 * queued row into x_perm (a bit copy) -- and empty the layer's queues.  Fills
 * *out (host struct).  AEP_ERR_EMPTY if nothing is queued, AEP_ERR_STATE if
 * a batch is still outstanding or weights of the layer are missing. */
aep_status aep_rebatch(aep_ctx* ctx, int32_t layer, aep_batch* out, void* stream);

/* Expert FFN of a batch: every group g computes, on its rows,
 * y = W_down (silu(W_gate x) * (W_up x)), silu(v) = v / (1 + e^-v), with
 * f32 accumulation; the intermediate h is rounded to the act dtype.
 * y: device [n_rows][d] act dtype, caller-owned.  A launch with few tiles
 * (bf16 and fp8 weights) splits its reduction into pieces whose f32 partial
 * sums are added in a fixed order, so results are reproducible run to run;
 * its per-tile counters live in the workspace, so FFN launches of one
 * context must not overlap on the GPU (issue them in stream order). */
aep_status aep_expert_ffn(aep_ctx* ctx, const aep_batch* batch, void* y, void* stream);

/* The two halves of aep_expert_ffn, for callers that schedule (or time) them
 * separately.  aep_expert_gate_up computes h = silu(W_gate x) * (W_up x) for
 * every row of the batch into the workspace; aep_expert_down then computes
 * y = W_down h.  aep_expert_down must follow aep_expert_gate_up of the same
 * batch in stream order (the library does not check this). */
aep_status aep_expert_gate_up(aep_ctx* ctx, const aep_batch* batch, void* stream);
aep_status aep_expert_down(aep_ctx* ctx, const aep_batch* batch, void* y, void* stream);

/* Top-K merge (Sec. 3.2): out[t] = sum_{j<k} token_weight[t][j] *
 * y[token_pos[t][j]] (slots ascending, absent slots skipped) + sum_s
 * y[n_routed + s*n_tokens + t], accumulated in f32 and rounded once.
 * out: device [n_tokens][d] act dtype, caller-owned. */
aep_status aep_combine(aep_ctx* ctx, const aep_batch* batch, const void* y, void* out, void* stream);

/* ---- Token pool: top-K merge across drains (Sec. 3.2, top-K support) ----
 * With single-expert drains a token's k rows run in different drains; its
 * outputs are merged in a per-layer pool keyed by a caller-chosen token id
 * (the request slot: the paper keys tokens by request and layer) and the
 * token is released when all k rows have been merged.  Requires
 * cfg.token_pool = 1 and n_shared = 0 (else AEP_ERR_UNSUPPORTED).  A layer
 * fed by aep_route_enqueue_ids is in pool mode until its queues are empty:
 * aep_route_enqueue, aep_enqueue_rows and aep_rebatch on it return
 * AEP_ERR_STATE, and aep_route_enqueue_ids on a layer holding rows of
 * aep_route_enqueue returns AEP_ERR_STATE.  Host-side totals of a pool-mode
 * layer (aep_queue_depth, aep_pick_layer) are upper bounds. */

/* As aep_route_enqueue, but token t of the fragment gets the caller's id
 * token_ids[t] (device int32 [T], each in [0, max_tokens_per_layer)) and
 * claims pool entry (layer, id) for its k rows.  An id whose entry is still
 * claimed (not yet released), or out of range, sets the device error flag
 * (reported by aep_sync).  Capacity: every expert queue of the layer must have
 * room for T more rows (AEP_ERR_CAPACITY otherwise, nothing launched). */
aep_status aep_route_enqueue_ids(aep_ctx* ctx, int32_t layer, const void* x, const float* logits,
                                 int32_t T, const int32_t* token_ids, int32_t* idx_out, float* w_out,
                                 void* stream);

/* Drain the queue of one expert of a pool-mode layer into a batch whose only
 * non-empty group is `expert` (counts/offsets of every other group are 0).
 * The exact row count is on the device (counts[expert]); n_routed = n_rows is
 * an upper bound known to the host (size y by it), n_tokens = 0 and
 * token_pos/token_weight are not filled.  Run the FFN as usual, then merge
 * with aep_pool_accumulate (aep_combine refuses such a batch).
 * AEP_ERR_EMPTY when the expert's queue is known to be empty, AEP_ERR_STATE as
 * for aep_rebatch. */
aep_status aep_rebatch_expert(aep_ctx* ctx, int32_t layer, int32_t expert, aep_batch* out, void* stream);

/* pool[layer][row_token[r]] += row_weight[r] * y[r] (f32 fused multiply-add)
 * for every row r of a single-expert batch, and one more of that token's k
 * rows is merged.  y: device [n_rows][d] act dtype. */
aep_status aep_pool_accumulate(aep_ctx* ctx, const aep_batch* batch, const void* y, void* stream);

/* Release every token of `layer` whose k rows have all been merged:
 * out[id] = the pool sum rounded once to the act dtype, the pool entry is
 * cleared and the id may be enqueued again; ready[id] = 1 for a released
 * token, 0 otherwise.  out: device [max_tokens_per_layer][d] act dtype (rows of
 * tokens not released are left untouched); ready: device int32
 * [max_tokens_per_layer] or NULL. */
aep_status aep_pool_release(aep_ctx* ctx, int32_t layer, void* out, int32_t* ready, void* stream);

/* Release a batch; its buffers may then be reused by the next aep_rebatch. */
aep_status aep_release_batch(aep_ctx* ctx, aep_batch* batch);

/* Wait for `stream`, then report (and clear) the device error flag. */
aep_status aep_sync(aep_ctx* ctx, void* stream);

/* Clock probe (instrumentation).  With d_buf a device array of 2 * n_pairs
 * uint64, every later bf16 / fp8-weight FFN launch of this context writes,
 * for each workgroup w < n_pairs, d_buf[2w] = shader-clock cycles
 * (s_memtime) and d_buf[2w+1] = ticks of the 100 MHz real-time counter
 * (s_memrealtime) elapsed in that workgroup; their ratio is the clock the
 * kernel ran at.  A launch overwrites the previous one's values; workgroups
 * of a launch are at most the CU count.  d_buf = NULL (or n_pairs <= 0)
 * turns the probe off (the default).  The f32 path records nothing.  The
 * buffer is borrowed and must stay valid while the probe is on. */
aep_status aep_set_clock_probe(aep_ctx* ctx, uint64_t* d_buf, int32_t n_pairs);

/* Utility: decode n OCP e4m3fn codes (device) to bf16 (device); exact. */
aep_status aep_fp8_e4m3_to_bf16(const uint8_t* codes, uint16_t* out, int64_t n, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* AEP_H_ */
