"""Seeded synthetic workloads shaped like the paper's expert-layer traffic.

The paper evaluates on Mixtral-8x7B-style layers whose router is replaced by
random expert selection from a skewed (exponential) popularity profile fitted
to a public instruction dataset (Sec. 5, evaluation setup).  Neither that
dataset nor trained weights are used here: every input below is drawn from a
seeded numpy PCG64 stream, with the shapes and the skewed expert popularity of
the five workloads this package knows about (``WORKLOADS``).

Recipe (identical for every workload):
  * stream: ``PCG64(SeedSequence(250508944, spawn_key=(cfg, layer, expert, tag)))``
  * activations x ~ N(0, 1); weights ~ 0.02 * N(0, 1); gate logits
    ~ N(0, 1) + beta_e with beta_e = -s * ln(rank_e), rank a seeded
    permutation of 1..E, so that softmax(beta) is exactly Zipf(s);
  * bf16 workloads store activations and weights as bf16 bit patterns
    (uint16, round-to-nearest-even from the f32 draw); logits stay f32;
  * fp8 weights: OCP e4m3fn codes with one bf16 scale per output channel,
    scale = bf16(max|W_row| / 448), code = e4m3(W / scale) rounded to nearest
    even and saturated at +-448.

Nothing here computes any part of the MoE layer.
"""

from __future__ import annotations

import dataclasses
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

SEED = 250508944
NO_EXPERT = 1000  # spawn-key stand-in for "not tied to one expert"

TAG_X, TAG_LOGITS, TAG_RANK, TAG_WG, TAG_WU, TAG_WD, TAG_DEPTH, TAG_PERM, TAG_GATEW, TAG_LAYERS = range(10)

__all__ = [
    "SEED", "Workload", "WORKLOADS", "workload", "rng", "round_to_bf16_bits",
    "bf16_bits_to_f32", "zipf_bias", "fragment_sizes", "layer_fragments",
    "expert_weights", "all_expert_weights", "rows_workload", "encode_e4m3",
    "quantize_rows_e4m3", "weight_source", "E4M3_MAX",
]


def rng(cfg_id: int, layer: int, expert: int, tag: int) -> np.random.Generator:
    """One independent seeded stream per (workload, layer, expert, tensor)."""
    ss = np.random.SeedSequence(SEED, spawn_key=(int(cfg_id), int(layer), int(expert), int(tag)))
    return np.random.Generator(np.random.PCG64(ss))


# ----------------------------------------------------------------------------
# element formats
# ----------------------------------------------------------------------------

def round_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """f32 -> bf16 bit pattern (uint16), round to nearest, ties to even.

    Inputs are finite draws; NaN handling is not needed here.
    """
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).copy()
    u += ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    u >>= np.uint32(16)
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


E4M3_MAX = 448.0


def encode_e4m3(a: np.ndarray) -> np.ndarray:
    """f32 -> OCP FP8 e4m3fn code (uint8): nearest, ties to even, saturating.

    e4m3fn: 1 sign, 4 exponent (bias 7), 3 mantissa bits; no infinities; only
    S.1111.111 is NaN, so the largest finite magnitude is 1.75 * 2^8 = 448.
    Magnitudes below 2^-6 are subnormal with quantum 2^-9.
    """
    a = np.asarray(a, dtype=np.float32)
    sign = np.signbit(a).astype(np.uint8) << np.uint8(7)
    mag = np.minimum(np.abs(a).astype(np.float64), E4M3_MAX)
    code = np.zeros(mag.shape, dtype=np.int64)
    sub = mag < 2.0 ** -6
    # subnormal range (and zero): code = rint(mag / 2^-9); 8 lands on 2^-6 = code 8
    code[sub] = np.rint(mag[sub] * 2.0 ** 9).astype(np.int64)
    nm = ~sub
    if np.any(nm):
        _, ex = np.frexp(mag[nm])          # mag = m * 2^ex, m in [0.5, 1)
        e = ex.astype(np.int64) - 1         # floor(log2 mag), in [-6, 8]
        q = np.rint(np.ldexp(mag[nm], (3 - e).astype(np.int32))).astype(np.int64)  # in [8, 16]
        code[nm] = ((e + 7) << 3) + (q - 8)
    code = np.minimum(code, 0x7E)           # 0x7F is NaN: saturate to 448
    return (code.astype(np.uint8) | sign).astype(np.uint8)


def quantize_rows_e4m3(w_bits: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Per-output-channel e4m3 quantisation of a bf16 [rows, K] weight matrix.

    Returns (codes uint8 [rows, K], scale bf16 bits uint16 [rows]).  A row that
    is entirely zero gets scale 1.
    """
    w = bf16_bits_to_f32(w_bits)
    amax = np.max(np.abs(w), axis=1)
    s_bits = round_to_bf16_bits((amax / np.float32(E4M3_MAX)).astype(np.float32))
    s = bf16_bits_to_f32(s_bits)
    zero = s == 0
    if np.any(zero):
        s_bits = s_bits.copy()
        s_bits[zero] = round_to_bf16_bits(np.array([1.0], np.float32))[0]
        s = bf16_bits_to_f32(s_bits)
    q = encode_e4m3((w / s[:, None]).astype(np.float32))
    return q, s_bits


# ----------------------------------------------------------------------------
# workload specs
# ----------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int
    d: int
    f: int
    E: int                     # routed experts resident on the GPU
    k: int                     # top-k (slots per token)
    zipf_s: float
    act: str = "bf16"          # "f32" | "bf16"
    wdt: str = "bf16"          # "f32" | "bf16" | "fp8"
    tokens: Tuple[int, ...] = (256,)   # tokens queued per layer
    n_frag: int = 1            # fragments each layer's tokens arrive in
    S: int = 0                 # shared experts (see every token, weight 1)
    renorm: bool = True
    mode: str = "routed"       # "routed": logits -> router; "rows": explicit per-expert rows
    weight_cfg: Optional[int] = None  # seed namespace for weights (default cfg_id)
    rotate_layers: bool = False       # layer l, expert e uses weights of layer 0, expert (e + l) % E
    depth_max: int = 4096      # "rows" mode: per-expert depth n_r = max(1, floor(depth_max * r^-s))
    description: str = ""

    @property
    def n_layers(self) -> int:
        return len(self.tokens)

    def flops_per_row(self) -> int:
        return 6 * self.d * self.f


WORKLOADS: Dict[str, Workload] = {
    "c1": Workload("c1", 1, d=256, f=512, E=8, k=2, zipf_s=1.0, act="f32", wdt="f32",
                   tokens=(256,), n_frag=1,
                   description="tiny MoE layer, fp32: 256 tokens, d=256, ffn=512, 8 experts, top-2, Zipf s=1.0"),
    "c1f4": Workload("c1f4", 1, d=256, f=512, E=8, k=2, zipf_s=1.0, act="f32", wdt="f32",
                     tokens=(256,), n_frag=4,
                     description="c1 arriving as 4 fragments"),
    "c2": Workload("c2", 2, d=4096, f=14336, E=8, k=2, zipf_s=1.2, tokens=(4096,), n_frag=4,
                   description="Mixtral-8x7B-style MoE layer, bf16: 4096 tokens, d=4096, ffn=14336, "
                               "8 experts, top-2, Zipf s=1.2, 4 fragments"),
    "c3": Workload("c3", 3, d=2048, f=1408, E=64, S=2, k=6, zipf_s=1.1, tokens=(8192,), n_frag=4,
                   description="fine-grained MoE layer, bf16: 8192 tokens, d=2048, ffn=1408, "
                               "64 routed + 2 shared experts, top-6, Zipf s=1.1"),
    "c4": Workload("c4", 4, d=4096, f=2048, E=16, k=1, zipf_s=1.3, mode="rows", depth_max=4096,
                   description="one GPU's expert-parallel share: 16 of 128 experts, d=4096, ffn=2048, "
                               "bf16, per-expert queue depths Zipf s=1.3 over 1..4096"),
    "c4fp8": Workload("c4fp8", 4, d=4096, f=2048, E=16, k=1, zipf_s=1.3, mode="rows", wdt="fp8",
                      depth_max=4096,
                      description="c4 with OCP e4m3fn weights and per-channel bf16 scales"),
    "c5": Workload("c5", 5, d=4096, f=14336, E=8, k=2, zipf_s=1.2,
                   tokens=(-1,) * 8, n_frag=4, weight_cfg=2, rotate_layers=True,
                   description="asynchronous 8-layer drain: 8 MoE layers at the c2 shape, "
                               "0..8192 tokens each, 32768 tokens total, most-tokens-first"),
}


def _c5_tokens() -> Tuple[int, ...]:
    sizes = np.array([8192, 7168, 6144, 5120, 3072, 2048, 1024, 0], dtype=np.int64)
    perm = rng(5, 0, NO_EXPERT, TAG_LAYERS).permutation(8)
    return tuple(int(v) for v in sizes[perm])


WORKLOADS["c5"] = dataclasses.replace(WORKLOADS["c5"], tokens=_c5_tokens())


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def weight_source(w: Workload, layer: int, expert: int) -> Tuple[int, int, int]:
    """Seed key (cfg, layer, expert) of the weights used by (layer, expert)."""
    cfg = w.cfg_id if w.weight_cfg is None else w.weight_cfg
    if w.rotate_layers and expert < w.E:
        return cfg, 0, (expert + layer) % w.E
    if w.rotate_layers:
        return cfg, 0, expert
    return cfg, layer, expert


# ----------------------------------------------------------------------------
# routed-mode inputs
# ----------------------------------------------------------------------------

def zipf_bias(w: Workload, layer: int) -> np.ndarray:
    """beta_e = -s ln(rank_e); softmax(beta) is the Zipf(s) pmf over the ranks."""
    ranks = rng(w.cfg_id, layer, NO_EXPERT, TAG_RANK).permutation(w.E) + 1
    return (-w.zipf_s * np.log(ranks.astype(np.float64))).astype(np.float32)


def fragment_sizes(T: int, F: int) -> List[int]:
    """Split T tokens into F arrival fragments, sizes as equal as possible."""
    F = max(1, F)
    base, rem = divmod(T, F)
    return [base + (1 if i < rem else 0) for i in range(F)]


def _act(w: Workload, a32: np.ndarray) -> np.ndarray:
    return a32 if w.act == "f32" else round_to_bf16_bits(a32)


def layer_fragments(w: Workload, layer: int) -> List[Dict[str, np.ndarray]]:
    """Per-fragment activations x [t, d] and gate logits [t, E] (f32).

    x is f32 for f32 workloads and bf16 bits (uint16) otherwise.  Fragments of
    size zero are skipped.
    """
    assert w.mode == "routed"
    T = w.tokens[layer]
    if T <= 0:
        return []
    x = rng(w.cfg_id, layer, NO_EXPERT, TAG_X).standard_normal((T, w.d), dtype=np.float32)
    z = rng(w.cfg_id, layer, NO_EXPERT, TAG_LOGITS).standard_normal((T, w.E), dtype=np.float32)
    logits = (z + zipf_bias(w, layer)[None, :]).astype(np.float32)
    xs = _act(w, x)
    out, t0 = [], 0
    for n in fragment_sizes(T, w.n_frag):
        if n:
            out.append({"x": np.ascontiguousarray(xs[t0:t0 + n]),
                        "logits": np.ascontiguousarray(logits[t0:t0 + n])})
        t0 += n
    return out


# ----------------------------------------------------------------------------
# weights
# ----------------------------------------------------------------------------

def _draw_matrix(key: Tuple[int, int, int], tag: int, shape: Tuple[int, int], fmt: str) -> np.ndarray:
    a = rng(key[0], key[1], key[2], tag).standard_normal(shape, dtype=np.float32)
    a *= np.float32(0.02)
    return a if fmt == "f32" else round_to_bf16_bits(a)


def expert_weights(w: Workload, layer: int, expert: int) -> Dict[str, np.ndarray]:
    """Weights of one expert (expert >= E: shared expert expert - E).

    Layout (out x in, K contiguous): gate [f, d], up [f, d], down [d, f].
    f32 workloads: float32 arrays.  bf16: uint16 bit patterns.  fp8: codes
    (uint8) for gate/up/down plus bf16 scale bits ``gate_up_scale`` [2f]
    (gate channels then up channels) and ``down_scale`` [d]; the bf16 weights
    they were quantised from are kept under ``*_bf16``.
    """
    key = weight_source(w, layer, expert)
    fmt = "f32" if w.wdt == "f32" else "bf16"
    ws = {
        "gate": _draw_matrix(key, TAG_WG, (w.f, w.d), fmt),
        "up": _draw_matrix(key, TAG_WU, (w.f, w.d), fmt),
        "down": _draw_matrix(key, TAG_WD, (w.d, w.f), fmt),
    }
    if w.wdt != "fp8":
        return ws
    qg, sg = quantize_rows_e4m3(ws["gate"])
    qu, su = quantize_rows_e4m3(ws["up"])
    qd, sd = quantize_rows_e4m3(ws["down"])
    return {"gate": qg, "up": qu, "down": qd,
            "gate_up_scale": np.concatenate([sg, su]), "down_scale": sd,
            "gate_bf16": ws["gate"], "up_bf16": ws["up"], "down_bf16": ws["down"]}


def all_expert_weights(w: Workload, layer: int, threads: int = 8,
                       experts: Optional[Sequence[int]] = None) -> List[Dict[str, np.ndarray]]:
    """Weights of every resident expert of a layer (routed, then shared)."""
    ids = list(range(w.E + w.S)) if experts is None else list(experts)
    if threads <= 1 or len(ids) == 1:
        return [expert_weights(w, layer, e) for e in ids]
    with ThreadPoolExecutor(max_workers=threads) as ex:
        return list(ex.map(lambda e: expert_weights(w, layer, e), ids))


# ----------------------------------------------------------------------------
# rows-mode inputs (explicit per-expert queues, one GPU's share of a larger layer)
# ----------------------------------------------------------------------------

def rows_workload(w: Workload, layer: int = 0) -> Dict[str, object]:
    """Explicit per-expert queue contents for "rows" workloads.

    Depths: n_r = max(1, floor(depth_max * r^-s)) for popularity ranks
    r = 1..E, assigned to experts by a seeded permutation.  Every row gets its
    own output slot (token id: a seeded permutation of 0..N-1) and a gate
    weight ~ U(0, 1) (f32); rows are x ~ N(0, 1) in the activation format.
    """
    assert w.mode == "rows"
    r = np.arange(1, w.E + 1, dtype=np.float64)
    depth_by_rank = np.maximum(1, np.floor(w.depth_max * r ** (-w.zipf_s))).astype(np.int64)
    perm = rng(w.cfg_id, layer, NO_EXPERT, TAG_DEPTH).permutation(w.E)
    depths = np.empty(w.E, dtype=np.int64)
    depths[perm] = depth_by_rank
    N = int(depths.sum())
    tok = rng(w.cfg_id, layer, NO_EXPERT, TAG_PERM).permutation(N).astype(np.int32)
    gw = rng(w.cfg_id, layer, NO_EXPERT, TAG_GATEW).random(N, dtype=np.float32)
    x = _act(w, rng(w.cfg_id, layer, NO_EXPERT, TAG_X).standard_normal((N, w.d), dtype=np.float32))
    per_expert, r0 = [], 0
    for e in range(w.E):
        n = int(depths[e])
        per_expert.append({"x": np.ascontiguousarray(x[r0:r0 + n]),
                           "token_ids": np.ascontiguousarray(tok[r0:r0 + n]),
                           "gate_w": np.ascontiguousarray(gw[r0:r0 + n])})
        r0 += n
    return {"depths": depths, "n_tokens": N, "experts": per_expert}
