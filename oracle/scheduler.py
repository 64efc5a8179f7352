"""Oracle of the layer-pick policies (TEST INFRASTRUCTURE ONLY).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may use
this module.

* most-tokens-first-serve (MTFS, Sec. 3.4): run the queue holding the most
  tokens.
* first-layer-first-serve (FLFS, Sec. 3.4): run the lowest-numbered block that
  holds any token.
* defragging scheduler (Sec. 3.4, Algorithm 1): for block b the lookahead score
  is sum_{i=1..L} (tokens queued in block (b+i) mod N_B / N_E) * delta^i; a
  non-empty queue (b, e) scores lookahead(b) + Q[b][e]; the arg-max is run.

Readings where the algorithm is silent or inconsistent: the lookahead depth L
is a parameter (the listing's bound clashes with the top-K symbol); the
average uses N_E; ties go to the lowest (b, e) in row-major order; when every
queue is empty there is nothing to run (None).  With delta = 0 the score is
the queue depth alone, i.e. MTFS over (block, expert) queues.

Parity: pinned by tests/test_oracle_scheduler.py (hand-computed queue tables).
"""

from __future__ import annotations

from typing import Optional, Sequence, Tuple

import numpy as np

__all__ = ["pick_mtfs", "pick_flfs", "defrag_scores", "pick_defrag"]


def pick_mtfs(rows: Sequence[int]) -> Optional[int]:
    best, best_rows = None, 0
    for b, r in enumerate(rows):
        if r > best_rows:
            best, best_rows = b, r
    return best


def pick_flfs(rows: Sequence[int]) -> Optional[int]:
    for b, r in enumerate(rows):
        if r > 0:
            return b
    return None


def defrag_scores(Q: np.ndarray, delta: float, lookahead: int) -> np.ndarray:
    Q = np.asarray(Q, dtype=np.float64)
    NB, NE = Q.shape
    scores = np.zeros((NB, NE), dtype=np.float64)
    for b in range(NB):
        lscore = 0.0
        for i in range(1, lookahead + 1):
            lscore += (Q[(b + i) % NB].sum() / NE) * delta ** i
        for e in range(NE):
            if Q[b, e] > 0:
                scores[b, e] = lscore + Q[b, e]
    return scores


def pick_defrag(Q: np.ndarray, delta: float, lookahead: int) -> Optional[Tuple[int, int]]:
    Q = np.asarray(Q)
    if not np.any(Q > 0):
        return None
    s = defrag_scores(Q, delta, lookahead)
    best = None
    for b in range(s.shape[0]):
        for e in range(s.shape[1]):
            if Q[b, e] > 0 and (best is None or s[b, e] > s[best]):
                best = (b, e)
    return best
