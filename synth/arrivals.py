"""Seeded request streams for the expert-runtime model (draws only).

A scenario fixes the model's shape (blocks, experts per block, top-k,
attention ranks), its cost model and a request stream: Poisson arrivals at
block 0 (exponential gaps at `rate` requests per second, as the paper's
serving experiments inject requests at a fixed rate, Sec. 5) with output
lengths drawn uniformly from [len_lo, len_hi], and an integer popularity
CDF over the experts, Zipf(s) in rank order.  Nothing here schedules or
queues anything.

Cost model (one GPU hosting every expert of every block): a step pays
cost_fixed_us per non-empty expert, the time to stream one Mixtral-8x7B
expert's bf16 weights (3 x 4096 x 14336 x 2 B = 352 MB) at the ~3.7 TB/s the
grouped FFN reaches on cold experts, and cost_row_ns per routed row, 6 d f
flops at the ~1.0 PFLOP/s it reaches on hot ones.
"""

from __future__ import annotations

import dataclasses
from typing import Dict

import numpy as np

from .workloads import rng

__all__ = ["Scenario", "SCENARIOS", "scenario", "request_stream"]


@dataclasses.dataclass(frozen=True)
class Scenario:
    name: str
    cfg_id: int
    n_blocks: int
    n_experts: int
    top_k: int
    n_frag: int
    rate: float          # requests per second
    len_lo: int
    len_hi: int
    zipf_s: float
    horizon_us: int
    attn_us: int = 1000
    jitter_us: int = 1000
    cost_fixed_us: int = 95
    cost_row_ns: int = 350
    description: str = ""


SCENARIOS: Dict[str, Scenario] = {
    # Mixtral-8x7B-sized model (32 blocks x 8 experts, top-2) near the load a
    # single GPU sustains: long requests, 4 attention ranks returning
    # fragments with up to 1 ms of jitter.
    "frag": Scenario("frag", 201, 32, 8, 2, 4, 20.0, 32, 256, 1.2, 20_000_000,
                     description="32 blocks x 8 experts, top-2, 20 req/s, 32-256 tokens, 4 attention ranks"),
    # many short requests above the rate the runtime serves with FLFS
    "livelock": Scenario("livelock", 202, 32, 8, 1, 4, 800.0, 1, 8, 1.2, 20_000_000,
                         description="32 blocks x 8 experts, top-1, 800 req/s, 1-8 tokens, 4 attention ranks"),
}


def scenario(name: str) -> Scenario:
    return SCENARIOS[name]


def request_stream(sc: Scenario) -> Dict[str, np.ndarray]:
    """arrival_us (int64, non-decreasing), out_len (int32), expert_cdf (int64)."""
    g = rng(sc.cfg_id, 0, 0, 0)
    n_max = int(sc.rate * sc.horizon_us / 1e6 * 1.5) + 16
    gaps = g.exponential(1e6 / sc.rate, n_max)
    t = np.floor(np.cumsum(gaps)).astype(np.int64)
    t = t[t < sc.horizon_us]
    out_len = g.integers(sc.len_lo, sc.len_hi + 1, t.size).astype(np.int32)
    p = 1.0 / np.arange(1, sc.n_experts + 1, dtype=np.float64) ** sc.zipf_s
    w = np.maximum(1, np.round(p / p.sum() * 1_000_000)).astype(np.int64)
    return {"arrival_us": t, "out_len": out_len, "expert_cdf": np.cumsum(w)}
