// Host-side scheduling over (block, expert) mu-queues and a discrete-event
// model of one expert runtime fed by an attention stub (Sec. 3.4, Algorithm 1;
// arrivals as in Sec. 5).  Host code only: no device work.
//
// aep_sched_pick: the three policies of Sec. 3.4 over a host table of queued
// rows Q[block][expert].
//
// aep_sim_run: one GPU that hosts every expert of every block, driven by a
// synthetic arrival process.  Requests arrive at block 0 at given times; a
// token queued at block b is routed to top_k distinct experts (one row per
// expert queue).  Whenever the GPU is free the policy picks what to run: one
// (block, expert) queue, or a whole block (every expert of it, one grouped
// launch).  When a step ends, a token whose top_k rows have all run leaves
// block b and goes through the attention stub: the tokens that left in one
// step are split over n_frag attention ranks and each rank's fragment arrives
// at block b + 1 after a latency plus a per-fragment jitter.  After the last
// block a token finishes one decode iteration; the request then sends its
// next token to block 0 the same way, or completes after out_len tokens.
//
// Every random choice (routing, fragment of a token, fragment jitter) comes
// from a counter-based generator: the SplitMix64 output function (Steele,
// Lea and Flood, "Fast splittable pseudorandom number generators", 2014)
// applied to seed + stream * 0xD1B54A32D192ED03 + counter * 0x9E3779B97F4A7C15
// (mod 2^64); the draw for a choice is a pure function of its key.  Times are
// integer microseconds, so a run is exactly reproducible.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <queue>
#include <unordered_map>
#include <vector>

#include "aep.h"
#include "aep_internal.h"

namespace {

constexpr uint64_t kStreamRoute = 1, kStreamFrag = 2, kStreamJitter = 3;

uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

uint64_t draw(uint64_t seed, uint64_t stream, uint64_t counter) {
  return mix64(seed + stream * 0xD1B54A32D192ED03ull + counter * 0x9E3779B97F4A7C15ull);
}

// Weights of the lookahead blocks: delta^1 .. delta^L, each the previous
// times delta.
std::vector<double> decay_weights(double delta, int lookahead) {
  std::vector<double> w((size_t)std::max(lookahead, 0));
  double pw = 1.0;
  for (auto& x : w) x = (pw *= delta);
  return w;
}

// Lookahead term of every block: the loads of the blocks after it (wrapping
// round), weighted by the decay of their distance, distances in ascending
// order.
std::vector<double> lookahead_terms(const std::vector<double>& load, double delta, int lookahead) {
  const int nb = (int)load.size();
  const std::vector<double> w = decay_weights(delta, lookahead);
  std::vector<double> look((size_t)nb, 0.0);
  for (int b = 0; b < nb; ++b)
    for (int i = 1; i <= lookahead; ++i) look[b] += load[(b + i) % nb] * w[i - 1];
  return look;
}

// Policy pick over a row-major table Q[nb][ne] of queued rows, evaluated one
// block at a time.  Every policy only ever runs the largest queue of some
// block (lowest expert on ties): MTFS compares those largest queues, FLFS takes
// the lowest non-empty block, and Algorithm 1 adds each block's lookahead term
// -- the average queue per expert of the blocks after it -- to its largest
// queue.  Blocks are compared with a strict "greater", so ties go to the lowest
// (block, expert).  Returns false when every queue is empty.
bool pick_queue(const int64_t* Q, int nb, int ne, int policy, double delta, int lookahead, int* pb,
                int* pe) {
  std::vector<int64_t> total((size_t)nb, 0), top_q((size_t)nb, 0);
  std::vector<int> top_e((size_t)nb, 0);
  for (int b = 0; b < nb; ++b) {
    const int64_t* row = Q + (size_t)b * ne;
    for (int e = 0; e < ne; ++e) {
      total[b] += row[e];
      if (row[e] > top_q[b]) top_q[b] = row[e], top_e[b] = e;
    }
  }
  std::vector<double> bonus((size_t)nb, 0.0);
  if (policy == AEP_POLICY_DEFRAG) {
    std::vector<double> avg((size_t)nb);
    for (int b = 0; b < nb; ++b) avg[b] = (double)total[b] / (double)ne;
    bonus = lookahead_terms(avg, delta, lookahead);
  }
  int bb = -1;
  double best = 0.0;
  for (int b = 0; b < nb; ++b) {
    if (top_q[b] <= 0) continue;
    if (policy == AEP_POLICY_FLFS) {
      bb = b;
      break;
    }
    const double sc = (double)top_q[b] + bonus[b];
    if (bb < 0 || sc > best) bb = b, best = sc;
  }
  if (bb < 0) return false;
  *pb = bb;
  *pe = top_e[bb];
  return true;
}

}  // namespace

namespace aep {

// Block-granularity pick over per-block totals R[nb] (a whole block drains,
// every expert of it).  The host knows only block totals without a device
// sync, so Algorithm 1's queue depth is replaced by the block's average queue
// R[b] / N_E and the score scaled by N_E: R[b] + sum_i R[(b + i) mod nb] *
// delta^i.
bool pick_block(const int64_t* R, int nb, int policy, double delta, int lookahead, int* pb) {
  std::vector<double> bonus((size_t)nb, 0.0);
  if (policy == AEP_POLICY_DEFRAG) bonus = lookahead_terms(std::vector<double>(R, R + nb), delta, lookahead);
  int bb = -1;
  double best = 0.0;
  for (int b = 0; b < nb; ++b) {
    if (R[b] <= 0) continue;
    if (policy == AEP_POLICY_FLFS) {
      bb = b;
      break;
    }
    const double sc = bonus[b] + (double)R[b];
    if (bb < 0 || sc > best) bb = b, best = sc;
  }
  if (bb < 0) return false;
  *pb = bb;
  return true;
}

}  // namespace aep

namespace {

bool bad_policy(int32_t policy, double delta, int32_t lookahead) {
  if (policy < AEP_POLICY_MTFS || policy > AEP_POLICY_DEFRAG) return true;
  if (policy == AEP_POLICY_DEFRAG && (lookahead < 0 || !(delta >= 0.0) || !std::isfinite(delta)))
    return true;
  return false;
}

struct Event {
  int64_t time;
  int64_t seq;
  int32_t block;                // target block (-1: a new request)
  std::vector<int64_t> tokens;  // token keys, in arrival order
};
struct EventLater {
  bool operator()(const Event* a, const Event* b) const {
    return a->time != b->time ? a->time > b->time : a->seq > b->seq;
  }
};

// token key = (request, iteration): request * 2^20 + iteration
constexpr int64_t kIterBits = 20;
inline int64_t tkey(int64_t r, int64_t it) { return (r << kIterBits) | it; }

}  // namespace

extern "C" {

aep_status aep_sched_pick(const int64_t* Q, int32_t n_blocks, int32_t n_experts, int32_t policy,
                          double delta, int32_t lookahead, int32_t* block, int32_t* expert) {
  if (!Q || !block || !expert || n_blocks <= 0 || n_experts <= 0) return AEP_ERR_INVALID_ARG;
  if (bad_policy(policy, delta, lookahead)) return AEP_ERR_INVALID_ARG;
  for (int64_t i = 0; i < (int64_t)n_blocks * n_experts; ++i)
    if (Q[i] < 0) return AEP_ERR_INVALID_ARG;
  int b, e;
  if (!pick_queue(Q, n_blocks, n_experts, policy, delta, lookahead, &b, &e)) return AEP_ERR_EMPTY;
  *block = b;
  *expert = e;
  return AEP_OK;
}

aep_status aep_sim_run(const aep_sim_config* cfg, aep_sim_trace* trace, aep_sim_summary* out) {
  if (!cfg || !out) return AEP_ERR_INVALID_ARG;
  const aep_sim_config& c = *cfg;
  const int NB = c.n_blocks, NE = c.n_experts, K = c.top_k;
  if (NB <= 0 || NB > 4096 || NE <= 0 || NE > 4096 || K <= 0 || K > NE || K > 64 || c.n_frag <= 0 ||
      c.n_frag > 4096 || c.attn_us < 1 || c.jitter_us < 0 || c.cost_fixed_us < 0 ||
      c.cost_row_ns < 0 || c.horizon_us < 0 || c.n_requests < 0 || c.n_requests > (1 << 20) ||
      (c.granularity != 0 && c.granularity != 1))
    return AEP_ERR_INVALID_ARG;
  if (bad_policy(c.policy, c.delta, c.lookahead)) return AEP_ERR_INVALID_ARG;
  if (c.n_requests > 0 && (!c.arrival_us || !c.out_len)) return AEP_ERR_INVALID_ARG;
  if (!c.expert_cdf) return AEP_ERR_INVALID_ARG;
  for (int e = 0; e < NE; ++e)
    if (c.expert_cdf[e] < (e ? c.expert_cdf[e - 1] : 0)) return AEP_ERR_INVALID_ARG;
  const int64_t cdf_total = c.expert_cdf[NE - 1];
  if (cdf_total <= 0) return AEP_ERR_INVALID_ARG;
  for (int32_t r = 0; r < c.n_requests; ++r)
    if (c.out_len[r] < 1 || c.out_len[r] >= (1 << kIterBits) || c.arrival_us[r] < 0 ||
        (r && c.arrival_us[r] < c.arrival_us[r - 1]))
      return AEP_ERR_INVALID_ARG;
  if (trace && trace->capacity > 0 &&
      (!trace->t_start || !trace->block || !trace->expert || !trace->rows || !trace->queued_after ||
       !trace->blocks_busy_after))
    return AEP_ERR_INVALID_ARG;

  // queues: FIFO of token keys per (block, expert)
  std::vector<std::vector<int64_t>> Q((size_t)NB * NE);
  std::vector<size_t> head((size_t)NB * NE, 0);
  std::unordered_map<int64_t, int32_t> remaining;  // token key -> rows still queued at its block
  std::priority_queue<Event*, std::vector<Event*>, EventLater> events;
  std::vector<Event> pool;
  pool.reserve((size_t)c.n_requests);
  int64_t seq = 0;
  for (int32_t r = 0; r < c.n_requests; ++r) pool.push_back(Event{c.arrival_us[r], seq++, -1, {tkey(r, 0)}});
  for (auto& ev : pool) events.push(&ev);
  std::vector<Event*> owned;  // events created during the run

  auto queued = [&](int b, int e) { return (int64_t)(Q[(size_t)b * NE + e].size() - head[(size_t)b * NE + e]); };

  auto enqueue = [&](int64_t key, int b) {
    // top_k distinct experts, each drawn from the integer popularity CDF
    int chosen[64];
    int n = 0;
    for (uint64_t j = 0; n < K && j < 4096; ++j) {
      const uint64_t u = draw(c.seed, kStreamRoute, ((uint64_t)key << 12 | (uint64_t)b) * 4096 + j) %
                         (uint64_t)cdf_total;
      int e = 0;
      while ((uint64_t)c.expert_cdf[e] <= u) ++e;
      bool dup = false;
      for (int i = 0; i < n; ++i) dup = dup || chosen[i] == e;
      if (!dup) chosen[n++] = e;
    }
    for (int e = 0; n < K && e < NE; ++e) {  // (only if 4096 draws were not enough)
      bool dup = false;
      for (int i = 0; i < n; ++i) dup = dup || chosen[i] == e;
      if (!dup) chosen[n++] = e;
    }
    for (int i = 0; i < K; ++i) Q[(size_t)b * NE + chosen[i]].push_back(key);
    remaining[key] = K;
  };

  std::vector<int64_t> done_time((size_t)c.n_requests, -1);
  int64_t t = 0, steps = 0, rows_total = 0, busy = 0, tokens_passed = 0, requests_done = 0;
  int64_t recorded = 0;
  std::vector<int64_t> R(NB), tab((size_t)NB * NE);
  std::vector<int64_t> drained, left;
  while (true) {
    while (!events.empty() && events.top()->time <= t) {
      Event* ev = events.top();
      events.pop();
      const int b = ev->block < 0 ? 0 : ev->block;
      for (int64_t key : ev->tokens) enqueue(key, b);
    }
    bool any = false;
    for (int b = 0; b < NB; ++b) {
      R[b] = 0;
      for (int e = 0; e < NE; ++e) {
        tab[(size_t)b * NE + e] = queued(b, e);
        R[b] += tab[(size_t)b * NE + e];
      }
      any = any || R[b] > 0;
    }
    if (any && t < c.horizon_us) {
      int pb = 0, pe = -1;
      if (c.granularity == 0)
        pick_queue(tab.data(), NB, NE, c.policy, c.delta, c.lookahead, &pb, &pe);
      else
        aep::pick_block(R.data(), NB, c.policy, c.delta, c.lookahead, &pb);
      // drain
      drained.clear();
      int nonempty = 0;
      for (int e = (pe < 0 ? 0 : pe); e < (pe < 0 ? NE : pe + 1); ++e) {
        const size_t q = (size_t)pb * NE + e;
        if (queued(pb, e) == 0) continue;
        ++nonempty;
        drained.insert(drained.end(), Q[q].begin() + (std::ptrdiff_t)head[q], Q[q].end());
        Q[q].clear();
        head[q] = 0;
      }
      const int64_t rows = (int64_t)drained.size();
      const int64_t dur = (int64_t)nonempty * c.cost_fixed_us + (rows * c.cost_row_ns + 999) / 1000;
      const int64_t t_end = t + dur;
      // tokens whose last queued row of this block just ran, in drain order
      left.clear();
      for (int64_t key : drained) {
        auto it = remaining.find(key);
        if (--it->second == 0) {
          left.push_back(key);
          remaining.erase(it);
        }
      }
      tokens_passed += (int64_t)left.size();
      // attention stub: next block, or the next decode iteration at block 0
      const int nb_next = pb + 1 < NB ? pb + 1 : 0;
      std::vector<std::vector<int64_t>> frag((size_t)c.n_frag);
      for (int64_t key : left) {
        int64_t nkey = key;
        if (pb + 1 == NB) {
          const int64_t r = key >> kIterBits, it = key & ((1 << kIterBits) - 1);
          if (it + 1 == c.out_len[r]) {
            done_time[(size_t)r] = t_end;
            ++requests_done;
            continue;
          }
          nkey = tkey(r, it + 1);
        }
        const uint64_t f = draw(c.seed, kStreamFrag, (uint64_t)key << 12 | (uint64_t)pb) % (uint64_t)c.n_frag;
        frag[f].push_back(nkey);
      }
      for (int f = 0; f < c.n_frag; ++f) {
        if (frag[(size_t)f].empty()) continue;
        const int64_t jit =
            (int64_t)(draw(c.seed, kStreamJitter, (uint64_t)steps * 4096 + (uint64_t)f) % (uint64_t)(c.jitter_us + 1));
        Event* ev = new Event{t_end + c.attn_us + jit, seq++, nb_next, std::move(frag[(size_t)f])};
        owned.push_back(ev);
        events.push(ev);
      }
      if (trace && recorded < trace->capacity) {
        int64_t qa = 0;
        int busy_blocks = 0;
        for (int b = 0; b < NB; ++b) {
          int64_t rb = 0;
          for (int e = 0; e < NE; ++e) rb += queued(b, e);
          qa += rb;
          busy_blocks += rb > 0;
        }
        trace->t_start[recorded] = t;
        trace->block[recorded] = pb;
        trace->expert[recorded] = pe;
        trace->rows[recorded] = rows;
        trace->queued_after[recorded] = qa;
        trace->blocks_busy_after[recorded] = busy_blocks;
        if (trace->block_rows_after)
          for (int b = 0; b < NB; ++b) {
            int64_t rb = 0;
            for (int e = 0; e < NE; ++e) rb += queued(b, e);
            trace->block_rows_after[recorded * NB + b] = rb;
          }
        ++recorded;
      }
      ++steps;
      rows_total += rows;
      busy += dur;
      t = t_end;
    } else {
      if (events.empty() || t >= c.horizon_us) break;
      t = std::max(t, events.top()->time);
    }
  }
  int64_t still_queued = 0;
  for (int b = 0; b < NB; ++b)
    for (int e = 0; e < NE; ++e) still_queued += queued(b, e);
  for (Event* ev : owned) delete ev;
  out->steps = steps;
  out->rows = rows_total;
  out->busy_us = busy;
  out->end_us = t;
  out->token_passes = tokens_passed;
  out->requests_done = requests_done;
  out->rows_queued_at_end = still_queued;
  out->recorded = recorded;
  if (trace && trace->done_us)
    for (int32_t r = 0; r < c.n_requests; ++r) trace->done_us[r] = done_time[(size_t)r];
  return AEP_OK;
}

}  // extern "C"
