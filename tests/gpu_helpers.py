"""Helpers of the GPU parity tests: move synth inputs to the device, run the
HIP path through the C ABI, run the oracle on the same inputs, compare."""

from __future__ import annotations

import sys
import time
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

import oracle
import synth

BF16_RTOL = 2e-2   # outputs of bf16 / fp8-weight workloads
F32_RTOL = 1e-5    # outputs of the fp32 workload
# gate weights: f32 exp / sum / divide against the float64 softmax rounded to
# f32: a few units of 2^-24 plus the argument rounding of (logit - max)
W_RTOL = 4e-6


def log(msg: str) -> None:
    sys.stdout.write(f"[{time.strftime('%H:%M:%S')}] {msg}\n")
    sys.stdout.flush()


def to_dev(a: np.ndarray, fmt: str) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if fmt == "bf16":
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    if fmt == "f32":
        return torch.from_numpy(a.astype(np.float32, copy=False)).cuda()
    if fmt == "fp8":
        return torch.from_numpy(a.astype(np.uint8, copy=False)).cuda()
    if fmt == "i32":
        return torch.from_numpy(a.astype(np.int32, copy=False)).cuda()
    raise ValueError(fmt)


def to_host(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def act_f64(a: np.ndarray, fmt: str) -> np.ndarray:
    return oracle.act_to_f64(a, fmt)


def assert_close(got: np.ndarray, ref: np.ndarray, rtol: float, what: str) -> Dict[str, float]:
    """|got - ref| <= atol + rtol |ref| elementwise, atol = rtol * rms(ref)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    atol = rtol * rms
    err = np.abs(got - ref)
    bad = err > atol + rtol * np.abs(ref)
    stats = {"max_abs": float(err.max()) if err.size else 0.0, "rms_ref": rms,
             "normwise": float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))}
    assert not bad.any(), (f"{what}: {int(bad.sum())} of {bad.size} elements out of tolerance; "
                           f"worst {err.max():.3e} (atol {atol:.3e}); {stats}")
    return stats


def upload_weights(ctx, w: synth.Workload, layer: int, ws: Sequence[Dict[str, np.ndarray]]):
    """Register host weights (synth format) with the context; returns device tensors."""
    fmt = "f32" if w.wdt == "f32" else ("fp8" if w.wdt == "fp8" else "bf16")
    dev = []
    for e, ex in enumerate(ws):
        g, u, d = to_dev(ex["gate"], fmt), to_dev(ex["up"], fmt), to_dev(ex["down"], fmt)
        sgu = sd = None
        if w.wdt == "fp8":
            sgu, sd = to_dev(ex["gate_up_scale"], "bf16"), to_dev(ex["down_scale"], "bf16")
        ctx.set_expert_weights(layer, e, g, u, d, sgu, sd)
        dev.append((g, u, d, sgu, sd))
    return dev


def make_context(w: synth.Workload, max_tokens: Optional[int] = None):
    import paper_2505_08944_amd as aep
    if max_tokens is None:
        if w.mode == "rows":
            max_tokens = synth.rows_workload(w)["n_tokens"]
        else:
            max_tokens = max(max(w.tokens), 1)
    return aep.Context(w.n_layers, w.E, w.d, w.f, w.k, n_shared=w.S, renorm=w.renorm, act=w.act,
                       wdt=("fp8" if w.wdt == "fp8" else w.wdt), max_tokens_per_layer=max_tokens)


def run_routed_layer(ctx, w: synth.Workload, layer: int, frags: List[Dict[str, np.ndarray]]):
    """Enqueue fragments, drain the layer; returns host copies of every stage."""
    dev_frags, routing = [], []
    for fr in frags:
        x = to_dev(fr["x"], w.act)
        lg = to_dev(fr["logits"], "f32")
        dev_frags.append((x, lg))
        routing.append(ctx.route_enqueue(layer, x, lg, routing_out=True))
    b = ctx.rebatch(layer)
    y = ctx.expert_ffn(b)
    out = ctx.combine(b, y)
    res = {
        "idx": [to_host(i) for i, _ in routing], "w": [to_host(v) for _, v in routing],
        "counts": to_host(b.counts()), "offsets": to_host(b.offsets()), "row_token": to_host(b.row_token()),
        "row_weight": to_host(b.row_weight()), "pos": to_host(b.token_pos()), "posw": to_host(b.token_weight()),
        "x_perm": to_host(b.x_perm()), "y": to_host(y), "out": to_host(out),
        "n_tokens": b.n_tokens, "n_routed": b.n_routed, "n_rows": b.n_rows,
    }
    ctx.release(b)
    ctx.sync()
    return res


def oracle_routed_layer(w: synth.Workload, frags, ws, full_ffn: bool = True):
    lq = oracle.LayerQueues(w.E, w.k, w.S, w.renorm)
    routing = [lq.enqueue_routed(fr["x"], fr["logits"]) for fr in frags]
    b = oracle.rebatch(lq)
    xp = oracle.gather(b)
    res = {"routing": routing, "batch": b, "xp": xp}
    if full_ffn:
        y = oracle.expert_ffn(b, xp, ws, w.act, "f32" if w.wdt == "f32" else w.wdt)
        res["y"] = y
        res["out"] = oracle.combine(b, y)
    return res


def check_routing_and_queues(w, got, ref):
    """Bit-exact: routing indices, counts, offsets, row order, pos, gathered rows."""
    for (ri, rw), gi, gw in zip(ref["routing"], got["idx"], got["w"]):
        assert np.array_equal(gi, ri), "routing indices differ"
        np.testing.assert_allclose(gw, rw, rtol=W_RTOL, atol=0)
    b = ref["batch"]
    assert got["n_routed"] == b.n_routed and got["n_tokens"] == b.n_tokens
    assert np.array_equal(got["counts"], b.counts), (got["counts"], b.counts)
    assert np.array_equal(got["offsets"], b.offsets.astype(np.int32))
    assert np.array_equal(got["row_token"], b.row_token)
    assert np.array_equal(got["pos"], b.pos)
    np.testing.assert_allclose(got["row_weight"], b.row_w, rtol=W_RTOL, atol=0)
    np.testing.assert_allclose(got["posw"], b.posw, rtol=W_RTOL, atol=0)
    assert got["x_perm"].shape == ref["xp"].shape
    assert np.array_equal(got["x_perm"], ref["xp"]), "gathered rows are not a bit copy"
