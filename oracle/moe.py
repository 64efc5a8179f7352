"""Oracle of one MoE layer computed through mu-queues (TEST INFRASTRUCTURE ONLY).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may use
this module.  It shares no code with the HIP path.

What is computed, and where the paper states it:

* route      -- gating and top-K selection are the last operators of the
               attention layer (Sec. 3.1 Overview; Sec. 3.2 "Top-K support");
               the selected experts' gate weights travel with the token as
               ``Topk_weights`` (Sec. 3.2, Table 1).  The paper does not define
               the router; this follows the usual softmax top-K gate (reading
               R1/R2 in the design notes): select on the logits (value desc,
               expert id asc), weights = softmax probabilities of the selected
               experts, renormalised over the K selected when ``renorm``.
* LayerQueues.enqueue_* -- the receptor files each arriving token under its
               LayerID = (block, expert) queue (Sec. 3.2, four-stage engine;
               a routed token is duplicated K times, one copy per expert).
* rebatch    -- the executor drains one layer's queues and merges every
               individually arrived fragment into one contiguous batch
               (Sec. 3.2; Sec. 5.4 "Schedule" stage).  Row order inside the
               batch: experts ascending, each expert's queue in arrival order.
* expert_ffn -- each expert is a bias-free SwiGLU FFN (Mixtral experts, the
               paper's evaluation model, Sec. 5): y = W_down (silu(W_gate x) *
               (W_up x)), silu(g) = g / (1 + e^-g).
* combine    -- the top-K merge (Sec. 3.2 "Top-K support"): a token's K
               expert outputs are summed with their gate weights (shared
               experts, when present, with weight 1), slot order ascending.
* brute_dense -- the same layer evaluated densely (every expert on every
               token, masked), with no queues, used to pin the queued path.

Parity: every function is pinned by tests/test_oracle_*.py (library
routines, closed forms, invariants and brute force); none is unpinned.
"""

from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "bf16_to_f64", "e4m3_to_f64", "act_to_f64", "weights_to_f64", "route",
    "Entry", "LayerQueues", "Batch", "rebatch", "gather", "silu", "swiglu",
    "expert_ffn", "combine", "moe_layer", "brute_dense", "topk_sorted",
]


# ----------------------------------------------------------------------------
# element formats (inputs are widened exactly before any arithmetic)
# ----------------------------------------------------------------------------

def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float64; bf16 is the top half of an f32."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def e4m3_to_f64(codes: np.ndarray) -> np.ndarray:
    """OCP FP8 e4m3fn codes (uint8) -> float64.

    Sign bit, 4-bit exponent with bias 7, 3-bit mantissa.  Exponent field 0
    encodes subnormals m * 2^-9; otherwise (1 + m/8) * 2^(e-7).  The single
    pattern S.1111.111 is NaN; there are no infinities.
    """
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    s = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = (c & 0x7).astype(np.float64)
    mag = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.exp2((e - 7).astype(np.float64)))
    mag = np.where((e == 0xF) & ((c & 0x7) == 0x7), np.nan, mag)
    return s * mag


def act_to_f64(a: np.ndarray, fmt: str) -> np.ndarray:
    if fmt == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    if fmt == "bf16":
        return bf16_to_f64(a)
    raise ValueError(fmt)


def weights_to_f64(ws: Dict[str, np.ndarray], wdt: str) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """(W_gate [f,d], W_up [f,d], W_down [d,f]) as float64.

    fp8 weights dequantise exactly as code * per-output-channel scale.
    """
    if wdt == "fp8":
        f = ws["gate"].shape[0]
        sgu = bf16_to_f64(ws["gate_up_scale"])
        sd = bf16_to_f64(ws["down_scale"])
        return (e4m3_to_f64(ws["gate"]) * sgu[:f, None],
                e4m3_to_f64(ws["up"]) * sgu[f:, None],
                e4m3_to_f64(ws["down"]) * sd[:, None])
    return (act_to_f64(ws["gate"], wdt), act_to_f64(ws["up"], wdt), act_to_f64(ws["down"], wdt))


# ----------------------------------------------------------------------------
# routing
# ----------------------------------------------------------------------------

def route(logits: np.ndarray, k: int, renorm: bool = True) -> Tuple[np.ndarray, np.ndarray]:
    """Top-k gate of a fragment: (idx int32 [T,k], w float32 [T,k]).

    Selection compares the f32 logits themselves (larger first, equal values
    -> lower expert id first), so exp() rounding can never create ties.
    Probabilities are softmax over all E logits in float64; with ``renorm``
    the k selected probabilities are divided by their sum.
    """
    l = np.asarray(logits, dtype=np.float32)
    assert l.ndim == 2 and 1 <= k <= l.shape[1]
    assert np.all(np.isfinite(l)), "gate logits must be finite"
    order = np.argsort(-l, axis=1, kind="stable")   # stable: ties keep ascending id
    idx = order[:, :k]
    l64 = l.astype(np.float64)
    z = np.exp(l64 - l64.max(axis=1, keepdims=True))
    p = z / z.sum(axis=1, keepdims=True)
    sel = np.take_along_axis(p, idx, axis=1)
    w = sel / sel.sum(axis=1, keepdims=True) if renorm else sel
    return idx.astype(np.int32), w.astype(np.float32)


def topk_sorted(logits_row: Sequence[float], k: int) -> List[int]:
    """Reference selection for one token by a full sort (used by brute_dense)."""
    return sorted(range(len(logits_row)), key=lambda e: (-float(logits_row[e]), e))[:k]


# ----------------------------------------------------------------------------
# mu-queues
# ----------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Entry:
    token: int        # layer-local token id (output row of the combine)
    slot: int         # top-k slot j of this duplicate
    w: float          # gate weight (f32 value)
    ref: Tuple[int, int]  # (fragment, row): where the input row lives


class LayerQueues:
    """One layer's mu-queues: a FIFO of entries per expert.

    The row data is not copied on enqueue: an entry refers to its row inside
    the fragment it arrived in, as the paper's token metadata refers to input
    tensors resident on the GPU (Table 1).
    """

    def __init__(self, E: int, k: int, S: int = 0, renorm: bool = True):
        self.E, self.k, self.S, self.renorm = E, k, S, renorm
        self.q: List[List[Entry]] = [[] for _ in range(E)]
        self.fragments: List[np.ndarray] = []
        self.token_ref: Dict[int, Tuple[int, int]] = {}
        self.n_tokens = 0

    @property
    def rows(self) -> int:
        return sum(len(q) for q in self.q)

    def enqueue_routed(self, x: np.ndarray, logits: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
        """Route a fragment and append its k duplicates per token.

        Appends in arrival order: tokens ascending, slots ascending; token ids
        continue the layer's running token count.
        """
        idx, w = route(logits, self.k, self.renorm)
        fi = len(self.fragments)
        self.fragments.append(x)
        base = self.n_tokens
        for t in range(idx.shape[0]):
            self.token_ref[base + t] = (fi, t)
            for j in range(self.k):
                self.q[int(idx[t, j])].append(Entry(base + t, j, float(w[t, j]), (fi, t)))
        self.n_tokens += idx.shape[0]
        return idx, w

    def enqueue_rows(self, expert: int, x: np.ndarray, token_ids: np.ndarray, gate_w: np.ndarray,
                     n_tokens: int, slots: Optional[np.ndarray] = None) -> None:
        """Append explicit rows (already routed elsewhere) to one expert's queue."""
        assert 0 <= expert < self.E
        fi = len(self.fragments)
        self.fragments.append(x)
        n = len(token_ids)
        for i in range(n):
            tok = int(token_ids[i])
            assert 0 <= tok < n_tokens
            s = 0 if slots is None else int(slots[i])
            self.q[expert].append(Entry(tok, s, float(np.float32(gate_w[i])), (fi, i)))
        self.n_tokens = max(self.n_tokens, n_tokens)


@dataclasses.dataclass
class Batch:
    """A drained layer, merged into one contiguous batch."""
    counts: np.ndarray      # int32 [E + S]: rows per group (shared groups: n_tokens)
    offsets: np.ndarray     # int64 [E + S + 1]: first row of each group
    row_token: np.ndarray   # int32 [N]: token of each routed row
    row_slot: np.ndarray    # int32 [N]
    row_w: np.ndarray       # float32 [N]
    row_ref: List[Tuple[int, int]]
    pos: np.ndarray         # int32 [n_tokens, k]: batch row of (token, slot), -1 if absent
    posw: np.ndarray        # float32 [n_tokens, k]: gate weight of (token, slot), 0 if absent
    n_tokens: int
    n_routed: int           # N
    S: int
    token_ref: List[Tuple[int, int]]  # input row of each token (shared experts' input)

    @property
    def n_rows_total(self) -> int:
        return self.n_routed + self.S * self.n_tokens


def rebatch(lq: LayerQueues) -> Batch:
    """Drain every expert queue of the layer into one batch (and empty them).

    Expert segments follow in ascending expert id, each in queue (arrival)
    order; shared-expert groups follow with every token in ascending order.
    """
    E, S, k, T = lq.E, lq.S, lq.k, lq.n_tokens
    counts = np.array([len(q) for q in lq.q] + [T] * S, dtype=np.int32)
    offsets = np.zeros(E + S + 1, dtype=np.int64)
    for g in range(E + S):
        offsets[g + 1] = offsets[g] + counts[g]
    entries = [en for q in lq.q for en in q]
    N = len(entries)
    pos = np.full((T, k), -1, dtype=np.int32)
    posw = np.zeros((T, k), dtype=np.float32)
    for r, en in enumerate(entries):
        assert pos[en.token, en.slot] == -1, "two rows claim one (token, slot)"
        pos[en.token, en.slot] = r
        posw[en.token, en.slot] = en.w
    token_ref = [lq.token_ref[t] for t in range(T)] if S else []
    b = Batch(counts=counts, offsets=offsets,
              row_token=np.array([en.token for en in entries], dtype=np.int32),
              row_slot=np.array([en.slot for en in entries], dtype=np.int32),
              row_w=np.array([en.w for en in entries], dtype=np.float32),
              row_ref=[en.ref for en in entries], pos=pos, posw=posw,
              n_tokens=T, n_routed=N, S=S, token_ref=token_ref)
    b.fragments = lq.fragments  # rows stay where they arrived
    lq.q = [[] for _ in range(E)]
    lq.fragments, lq.token_ref, lq.n_tokens = [], {}, 0
    return b


def gather(b: Batch) -> np.ndarray:
    """The contiguous input batch Xp (a bit copy, in the stored format).

    Rows [0, N): routed rows in batch order.  When shared experts exist, rows
    [N, N + n_tokens) hold every token in id order (read by all shared groups).
    """
    frags = b.fragments
    refs = list(b.row_ref) + list(b.token_ref)
    if not refs:
        return np.zeros((0, 0))
    return np.stack([frags[fi][ri] for fi, ri in refs])


# ----------------------------------------------------------------------------
# expert FFN and combine
# ----------------------------------------------------------------------------

def silu(g: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        return g / (1.0 + np.exp(-g))


def swiglu(x: np.ndarray, wg: np.ndarray, wu: np.ndarray, wd: np.ndarray) -> np.ndarray:
    """y = W_down (silu(W_gate x) * (W_up x)) for rows x [n, d]."""
    return (silu(x @ wg.T) * (x @ wu.T)) @ wd.T


def expert_ffn(b: Batch, xp: np.ndarray, weights: Sequence[Dict[str, np.ndarray]],
               act: str, wdt: str) -> np.ndarray:
    """Every group's FFN on its rows; float64 [N + S * n_tokens, d].

    An expert with no queued rows is skipped (its weights are not read).
    """
    E = len(b.counts) - b.S
    d = xp.shape[1]
    y = np.zeros((b.n_rows_total, d), dtype=np.float64)
    for g in range(E):
        n = int(b.counts[g])
        if n == 0:
            continue
        o = int(b.offsets[g])
        y[o:o + n] = swiglu(act_to_f64(xp[o:o + n], act), *weights_to_f64(weights[g], wdt))
    if b.S:
        xs = act_to_f64(xp[b.n_routed:b.n_routed + b.n_tokens], act)
        for s in range(b.S):
            o = b.n_routed + s * b.n_tokens
            y[o:o + b.n_tokens] = swiglu(xs, *weights_to_f64(weights[E + s], wdt))
    return y


def combine(b: Batch, y: np.ndarray) -> np.ndarray:
    """out[t] = sum_j posw[t,j] * y[pos[t,j]] (slot order) + sum_s y_shared_s[t]."""
    T, k = b.pos.shape
    d = y.shape[1]
    out = np.zeros((T, d), dtype=np.float64)
    for j in range(k):
        p = b.pos[:, j]
        m = p >= 0
        out[m] += b.posw[m, j].astype(np.float64)[:, None] * y[p[m]]
    for s in range(b.S):
        o = b.n_routed + s * T
        out += y[o:o + T]
    return out


def moe_layer(lq: LayerQueues, weights: Sequence[Dict[str, np.ndarray]], act: str, wdt: str) -> Dict[str, object]:
    """Drain lq and run the whole layer; returns every intermediate."""
    b = rebatch(lq)
    xp = gather(b)
    y = expert_ffn(b, xp, weights, act, wdt)
    return {"batch": b, "xp": xp, "y": y, "out": combine(b, y)}


# ----------------------------------------------------------------------------
# dense brute force (no queues)
# ----------------------------------------------------------------------------

def brute_dense(x: np.ndarray, logits: np.ndarray, weights: Sequence[Dict[str, np.ndarray]],
                k: int, renorm: bool, S: int, act: str, wdt: str) -> np.ndarray:
    """out[t] = sum_e [e in topk(t)] w_e(t) FFN_e(x_t) + sum_s FFN_s(x_t).

    Every expert runs on every token; the routing mask is applied afterwards.
    Selection uses a full sort per token; weights are float64 softmax values
    (renormalised over the selected experts when ``renorm``).
    """
    T, E = logits.shape
    x64 = act_to_f64(x, act)
    l64 = np.asarray(logits, dtype=np.float32).astype(np.float64)
    mask_w = np.zeros((T, E), dtype=np.float64)
    for t in range(T):
        sel = topk_sorted(logits[t], k)
        p = np.exp(l64[t] - l64[t].max())
        p /= p.sum()
        tot = sum(p[e] for e in sel) if renorm else 1.0
        for e in sel:
            mask_w[t, e] = p[e] / tot
    out = np.zeros((T, x.shape[1]), dtype=np.float64)
    for e in range(E):
        out += mask_w[:, e:e + 1] * swiglu(x64, *weights_to_f64(weights[e], wdt))
    for s in range(S):
        out += swiglu(x64, *weights_to_f64(weights[E + s], wdt))
    return out
