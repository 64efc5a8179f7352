"""Oracle of the expert-runtime model (TEST INFRASTRUCTURE ONLY).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may use
this module.

A plain event-by-event restatement of the model the library runs (Sec. 3.4
for the policies and the fragmentation they cause; Sec. 5 for requests
arriving over time), written with Python lists, dicts and heapq:

* request r puts its token (r, 0) into block 0 at arrival_us[r];
* a token entering block b is routed to top_k distinct experts: draw j of the
  routing stream gives u = draw mod (last CDF entry), and the expert is the
  first e with cdf[e] > u; repeated experts are skipped;
* when the runtime is free and rows are queued (and the time is before the
  horizon) the policy picks a (block, expert) queue (oracle/scheduler.py:
  pick_queue_mtfs, pick_queue_flfs, pick_defrag) or a whole block
  (pick_mtfs, pick_flfs, pick_layer_defrag over block totals), whose
  rows are drained in queue order (experts in id order for a block); the step
  lasts (non-empty experts) * cost_fixed_us + ceil(rows * cost_row_ns / 1000);
* at the end of the step every token whose last queued row of that block ran
  leaves it, in drain order; each goes to attention rank (fragment draw mod
  n_frag); each rank's list arrives at the next block attn_us + (jitter draw
  mod (jitter_us + 1)) later; after the last block the request either
  completes (its out_len-th token) or sends token (r, it + 1) to block 0 the
  same way;
* events due at the same time are delivered in creation order.

The generator is SplitMix64's output function (Steele, Lea, Flood 2014) on
seed + stream * 0xD1B54A32D192ED03 + counter * 0x9E3779B97F4A7C15 mod 2^64.

Parity: pinned by tests/test_oracle_sim.py (hand-traced runs at expert and
block granularity under every policy, with the scores at the decisions where
the policies part ways; conservation laws; the SplitMix64 reference
sequence) and compared step by step with the
library in tests/test_sched_host.py.
"""

from __future__ import annotations

import heapq
from typing import Dict, List, Sequence

from .scheduler import (pick_defrag, pick_flfs, pick_layer_defrag, pick_mtfs, pick_queue_flfs,
                        pick_queue_mtfs)

MASK = (1 << 64) - 1
GOLDEN = 0x9E3779B97F4A7C15
STREAM_MUL = 0xD1B54A32D192ED03
ROUTE, FRAG, JITTER = 1, 2, 3


def splitmix64_out(z: int) -> int:
    z &= MASK
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK
    return z ^ (z >> 31)


def draw(seed: int, stream: int, counter: int) -> int:
    return splitmix64_out(seed + stream * STREAM_MUL + counter * GOLDEN)


def _pick_queue(Q: List[List[int]], policy: str, delta: float, lookahead: int):
    if policy == "mtfs":
        return pick_queue_mtfs(Q)
    if policy == "flfs":
        return pick_queue_flfs(Q)
    return pick_defrag(Q, delta, lookahead)


def _pick_block(R: List[int], policy: str, delta: float, lookahead: int):
    if policy == "mtfs":
        return pick_mtfs(R)
    if policy == "flfs":
        return pick_flfs(R)
    return pick_layer_defrag(R, delta, lookahead)


def simulate(*, n_blocks: int, n_experts: int, top_k: int, n_frag: int, granularity: str, policy: str,
             arrival_us: Sequence[int], out_len: Sequence[int], expert_cdf: Sequence[int], attn_us: int,
             jitter_us: int, cost_fixed_us: int, cost_row_ns: int, horizon_us: int, seed: int,
             delta: float = 0.5, lookahead: int = 2) -> Dict[str, object]:
    NB, NE, K = n_blocks, n_experts, top_k
    cdf = [int(c) for c in expert_cdf]
    total = cdf[-1]
    queues = [[[] for _ in range(NE)] for _ in range(NB)]
    pending: Dict[tuple, int] = {}       # (request, iteration) -> rows still queued
    heap: list = []
    seq = 0
    for r, t_arr in enumerate(arrival_us):
        heapq.heappush(heap, (int(t_arr), seq, 0, [(r, 0)]))
        seq += 1

    def enter(token, b):
        r, it = token
        chosen: List[int] = []
        j = 0
        while len(chosen) < K and j < 4096:
            counter = ((((r << 20) | it) << 12 | b) * 4096 + j) & MASK
            u = draw(seed, ROUTE, counter) % total
            e = next(x for x in range(NE) if cdf[x] > u)
            if e not in chosen:
                chosen.append(e)
            j += 1
        for e in range(NE):
            if len(chosen) == K:
                break
            if e not in chosen:
                chosen.append(e)
        for e in chosen:
            queues[b][e].append(token)
        pending[token] = K

    t = 0
    steps = rows_total = busy = passes = done = 0
    done_us = [-1] * len(arrival_us)
    trace = {k: [] for k in ("t_start", "block", "expert", "rows", "queued_after", "blocks_busy_after",
                             "block_rows_after")}
    while True:
        while heap and heap[0][0] <= t:
            _, _, b, tokens = heapq.heappop(heap)
            for tok in tokens:
                enter(tok, b)
        table = [[len(queues[b][e]) for e in range(NE)] for b in range(NB)]
        R = [sum(row) for row in table]
        if sum(R) > 0 and t < horizon_us:
            if granularity == "expert":
                pb, pe = _pick_queue(table, policy, delta, lookahead)
                experts = [pe]
            else:
                pb, pe = _pick_block(R, policy, delta, lookahead), -1
                experts = list(range(NE))
            drained = []
            nonempty = 0
            for e in experts:
                if queues[pb][e]:
                    nonempty += 1
                    drained.extend(queues[pb][e])
                    queues[pb][e] = []
            rows = len(drained)
            dur = nonempty * cost_fixed_us + -(-(rows * cost_row_ns) // 1000)
            t_end = t + dur
            leaving = []
            for tok in drained:
                pending[tok] -= 1
                if pending[tok] == 0:
                    del pending[tok]
                    leaving.append(tok)
            passes += len(leaving)
            nxt = pb + 1 if pb + 1 < NB else 0
            ranks: List[List[tuple]] = [[] for _ in range(n_frag)]
            for tok in leaving:
                r, it = tok
                new = tok
                if pb + 1 == NB:
                    if it + 1 == out_len[r]:
                        done_us[r] = t_end
                        done += 1
                        continue
                    new = (r, it + 1)
                f = draw(seed, FRAG, ((((r << 20) | it) << 12) | pb) & MASK) % n_frag
                ranks[f].append(new)
            for f in range(n_frag):
                if ranks[f]:
                    jit = draw(seed, JITTER, (steps * 4096 + f) & MASK) % (jitter_us + 1)
                    heapq.heappush(heap, (t_end + attn_us + jit, seq, nxt, ranks[f]))
                    seq += 1
            after = [sum(len(q) for q in queues[b]) for b in range(NB)]
            trace["t_start"].append(t)
            trace["block"].append(pb)
            trace["expert"].append(pe)
            trace["rows"].append(rows)
            trace["queued_after"].append(sum(after))
            trace["blocks_busy_after"].append(sum(1 for a in after if a > 0))
            trace["block_rows_after"].append(after)
            steps += 1
            rows_total += rows
            busy += dur
            t = t_end
        else:
            if not heap or t >= horizon_us:
                break
            t = max(t, heap[0][0])
    return {"steps": steps, "rows": rows_total, "busy_us": busy, "end_us": t, "token_passes": passes,
            "requests_done": done, "rows_queued_at_end": sum(len(q) for row in queues for q in row),
            "trace": trace, "done_us": done_us}
