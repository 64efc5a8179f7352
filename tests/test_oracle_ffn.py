"""Pins of the oracle's SwiGLU experts, combine and whole-layer composition."""

import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_silu_textbook_values_and_torch():
    assert oracle.silu(np.array([0.0]))[0] == 0.0
    assert oracle.silu(np.array([1.0]))[0] == pytest.approx(1.0 / (1.0 + math.exp(-1.0)), rel=1e-15)
    assert oracle.silu(np.array([-800.0]))[0] == 0.0          # no overflow trouble
    assert oracle.silu(np.array([800.0]))[0] == 800.0
    g = np.linspace(-30, 30, 2001)
    ref = torch.nn.functional.silu(torch.from_numpy(g)).numpy()
    np.testing.assert_allclose(oracle.silu(g), ref, rtol=1e-14, atol=1e-300)


def test_swiglu_against_torch_modules():
    r = np.random.default_rng(0)
    x, wg, wu, wd = (r.standard_normal(s) for s in [(7, 24), (40, 24), (40, 24), (24, 40)])
    F = torch.nn.functional
    t = lambda a: torch.from_numpy(a)
    ref = F.linear(F.silu(F.linear(t(x), t(wg))) * F.linear(t(x), t(wu)), t(wd)).numpy()
    np.testing.assert_allclose(oracle.swiglu(x, wg, wu, wd), ref, rtol=1e-12, atol=1e-14)


def test_scalar_closed_form():
    # d = f = 1: y = wd * silu(wg x) * (wu x); x=2, wg=.5, wu=3, wd=-1 -> -6 silu(1)
    y = oracle.swiglu(np.array([[2.0]]), np.array([[0.5]]), np.array([[3.0]]), np.array([[-1.0]]))
    assert y[0, 0] == pytest.approx(-6.0 / (1.0 + math.exp(-1.0)), rel=1e-15)


def _small(seed, T=40, E=6, k=2, S=0, d=12, f=20, renorm=True, sizes=None, wdt="f32", act="f32"):
    w = synth.Workload("t", 90 + seed, d=d, f=f, E=E, k=k, S=S, zipf_s=1.0, act=act, wdt=wdt,
                       tokens=(T,), n_frag=1, renorm=renorm)
    r = np.random.default_rng(seed)
    x32 = r.standard_normal((T, d)).astype(np.float32)
    x = x32 if act == "f32" else synth.round_to_bf16_bits(x32)
    l = (r.standard_normal((T, E)) + synth.zipf_bias(w, 0)).astype(np.float32)
    ws = synth.all_expert_weights(w, 0, threads=1)
    return w, x, l, ws


def _queued(w, x, l, ws, sizes=None):
    lq = oracle.LayerQueues(w.E, w.k, w.S, w.renorm)
    t0 = 0
    for n in (sizes or [x.shape[0]]):
        lq.enqueue_routed(x[t0:t0 + n], l[t0:t0 + n])
        t0 += n
    return oracle.moe_layer(lq, ws, w.act, w.wdt)


@pytest.mark.parametrize("kw", [
    dict(seed=1), dict(seed=2, k=1), dict(seed=3, k=6, E=6), dict(seed=4, renorm=False, k=3),
    dict(seed=5, S=2, k=3, E=10), dict(seed=6, sizes=[5, 0, 30, 5]), dict(seed=7, act="bf16", wdt="bf16"),
    dict(seed=8, act="bf16", wdt="fp8", S=1), dict(seed=9, T=1, E=3, k=2),
])
def test_queued_equals_brute_dense(kw):
    sizes = kw.pop("sizes", None)
    w, x, l, ws = _small(**kw)
    res = _queued(w, x, l, ws, [s for s in sizes if s] if sizes else None)
    ref = oracle.brute_dense(x, l, ws, w.k, w.renorm, w.S, w.act, w.wdt)
    # the queued path carries f32 gate weights, the dense path float64 ones
    scale = np.abs(ref).max() + 1e-30
    np.testing.assert_allclose(res["out"], ref, rtol=0, atol=2e-7 * scale)


def test_identical_experts_reduce_to_dense_ffn():
    w, x, l, ws = _small(11, E=5, k=3)
    ws = [ws[0]] * w.E
    res = _queued(w, x, l, ws)
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    F = torch.nn.functional
    dense = F.linear(F.silu(F.linear(t(x), t(ws[0]["gate"]))) * F.linear(t(x), t(ws[0]["up"])), t(ws[0]["down"])).numpy()
    np.testing.assert_allclose(res["out"], dense, rtol=1e-6, atol=1e-9)


def test_zero_and_doubled_down_projection():
    w, x, l, ws = _small(12, S=1, k=2)
    base = _queued(w, x, l, ws)["out"]
    zero = [dict(e, down=np.zeros_like(e["down"])) for e in ws]
    assert np.all(_queued(w, x, l, zero)["out"] == 0.0)
    dbl = [dict(e, down=e["down"] * np.float32(2.0)) for e in ws]
    assert np.array_equal(_queued(w, x, l, dbl)["out"], 2.0 * base)


def test_expert_relabelling_is_invisible():
    w, x, l, ws = _small(13, E=7, k=3)
    base = _queued(w, x, l, ws)["out"]
    p = np.random.default_rng(1).permutation(w.E)     # new expert i is old expert p[i]
    out = _queued(w, x, np.ascontiguousarray(l[:, p]), [ws[i] for i in p])["out"]
    np.testing.assert_allclose(out, base, rtol=1e-12, atol=1e-14)


def test_top1_combine_copies_the_expert_row():
    w, x, l, ws = _small(14, k=1)
    res = _queued(w, x, l, ws)
    b = res["batch"]
    assert np.array_equal(res["out"], res["y"][b.pos[:, 0]])


def test_shared_experts_add_with_weight_one():
    w, x, l, ws = _small(15, S=2, k=2)
    ws = [dict(e, down=np.zeros_like(e["down"])) for e in ws[:w.E]] + ws[w.E:]
    out = _queued(w, x, l, ws)["out"]
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    F = torch.nn.functional
    ref = sum(F.linear(F.silu(F.linear(t(x), t(e["gate"]))) * F.linear(t(x), t(e["up"])), t(e["down"])).numpy()
              for e in ws[w.E:])
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-14)


def test_fp8_weights_are_code_times_scale():
    w, x, l, ws = _small(16, act="bf16", wdt="fp8")
    deq = []
    for e in ws:
        g, u, dn = oracle.weights_to_f64(e, "fp8")
        deq.append({"gate": g.astype(np.float32), "up": u.astype(np.float32), "down": dn.astype(np.float32)})
        # code * scale is exact in f32 (4 + 8 significant bits)
        assert np.array_equal(g, g.astype(np.float32).astype(np.float64))
        # quantisation error: at most half a code step of the scaled grid
        ref = synth.bf16_bits_to_f32(e["gate_bf16"]).astype(np.float64)
        s = oracle.bf16_to_f64(e["gate_up_scale"][:w.f])[:, None]
        assert np.all(np.abs(g - ref) <= s * 2.0 ** -4 * np.maximum(np.abs(ref / s), 2.0 ** -6) + 1e-30)
    a = _queued(w, x, l, ws)["out"]
    b = _queued(dict_w(w, wdt="f32"), x, l, deq)["out"]
    np.testing.assert_allclose(a, b, rtol=0, atol=0)


def dict_w(w, **kw):
    import dataclasses
    return dataclasses.replace(w, **kw)


def test_empty_expert_weights_are_not_read():
    w, x, l, ws = _small(17, E=6, k=1)
    l[:, 4] = -50.0   # expert 4 never chosen
    ws = list(ws)
    ws[4] = None
    res = _queued(w, x, l, ws)
    assert res["batch"].counts[4] == 0


def test_hand_worked_layer():
    fx = json.load(open(os.path.join(GOLDEN, "tiny_layer.json")))
    s = lambda g: g / (1.0 + math.exp(-g))
    e = math.e
    lq = oracle.LayerQueues(3, 2)
    lq.enqueue_routed(np.array(fx["x"], np.float32)[:, None], np.array(fx["logits"], np.float32))
    ws = [{k: np.array([[v]], np.float32) for k, v in ex.items()} for ex in fx["experts"]]
    res = oracle.moe_layer(lq, ws, "f32", "f32")
    y_ref = [2 * s(2.0), -s(-1.0), -0.5 * s(2.0), -s(4.0), 0.0, 0.0]
    np.testing.assert_allclose(res["y"][:, 0], y_ref, rtol=1e-15, atol=1e-300)
    np.testing.assert_allclose(res["y"][:, 0], fx["y_rows"], rtol=1e-15, atol=1e-300)
    out_ref = [0.4 * (-0.5 * s(2.0)), 0.5 * 2 * s(2.0) - 0.5 * s(4.0), (1 / (e + 1)) * (-s(-1.0))]
    np.testing.assert_allclose(res["out"][:, 0], out_ref, rtol=1e-6)
    np.testing.assert_allclose(res["out"][:, 0], fx["out"], rtol=1e-6)
