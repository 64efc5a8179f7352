"""Host-side scheduler and expert-runtime model (numpy arrays -> libaep).

`sched_pick` and `sim_run` marshal host arrays into aep_sched_pick and
aep_sim_run (include/aep.h); the policies and the model run in the library.
"""

from __future__ import annotations

import ctypes
from typing import Dict, Optional, Tuple

import numpy as np

from . import _lib as L

POLICIES = {"mtfs": L.AEP_POLICY_MTFS, "flfs": L.AEP_POLICY_FLFS, "defrag": L.AEP_POLICY_DEFRAG}


def sched_pick(Q: np.ndarray, policy: str, delta: float = 0.5, lookahead: int = 2) -> Optional[Tuple[int, int]]:
    """(block, expert) to run next from a table Q[n_blocks][n_experts] of
    queued rows, or None when every queue is empty."""
    Qc = np.ascontiguousarray(Q, dtype=np.int64)
    if Qc.ndim != 2:
        raise ValueError("Q must be [n_blocks][n_experts]")
    b, e = L._I32(-1), L._I32(-1)
    st = L.lib().aep_sched_pick(Qc.ctypes.data, Qc.shape[0], Qc.shape[1], POLICIES[policy], float(delta),
                                int(lookahead), ctypes.byref(b), ctypes.byref(e))
    if st == L.AEP_ERR_EMPTY:
        return None
    L.check(st, "aep_sched_pick")
    return int(b.value), int(e.value)


def sim_run(*, n_blocks: int, n_experts: int, top_k: int, n_frag: int, granularity: str, policy: str,
            arrival_us: np.ndarray, out_len: np.ndarray, expert_cdf: np.ndarray, attn_us: int,
            jitter_us: int, cost_fixed_us: int, cost_row_ns: int, horizon_us: int, seed: int,
            delta: float = 0.5, lookahead: int = 2, trace_capacity: int = 0) -> Dict[str, object]:
    """Run the expert-runtime model; returns the summary fields, the per-step
    trace (first trace_capacity steps) and per-request completion times."""
    arr = np.ascontiguousarray(arrival_us, dtype=np.int64)
    ol = np.ascontiguousarray(out_len, dtype=np.int32)
    cdf = np.ascontiguousarray(expert_cdf, dtype=np.int64)
    if arr.shape != ol.shape or cdf.shape != (n_experts,):
        raise ValueError("arrival_us/out_len/expert_cdf shapes")
    cfg = L.SimConfig(n_blocks, n_experts, top_k, n_frag, {"expert": 0, "block": 1}[granularity],
                      POLICIES[policy], float(delta), int(lookahead), int(arr.size), int(attn_us),
                      int(jitter_us), int(cost_fixed_us), int(cost_row_ns), int(horizon_us),
                      int(seed) & 0xFFFFFFFFFFFFFFFF, arr.ctypes.data, ol.ctypes.data, cdf.ctypes.data)
    cap = int(trace_capacity)
    tr = {"t_start": np.zeros(cap, np.int64), "block": np.zeros(cap, np.int32), "expert": np.zeros(cap, np.int32),
          "rows": np.zeros(cap, np.int64), "queued_after": np.zeros(cap, np.int64),
          "blocks_busy_after": np.zeros(cap, np.int32), "block_rows_after": np.zeros((cap, n_blocks), np.int64)}
    done = np.zeros(arr.size, np.int64)
    trace = L.SimTrace(cap, *(tr[k].ctypes.data for k in ("t_start", "block", "expert", "rows", "queued_after",
                                                          "blocks_busy_after", "block_rows_after")),
                       done.ctypes.data)
    summ = L.SimSummary()
    L.check(L.lib().aep_sim_run(ctypes.byref(cfg), ctypes.byref(trace), ctypes.byref(summ)), "aep_sim_run")
    out: Dict[str, object] = {n: int(getattr(summ, n)) for n, _ in L.SimSummary._fields_}
    n = out["recorded"]
    out["trace"] = {k: v[:n].copy() for k, v in tr.items()}
    out["done_us"] = done
    return out
