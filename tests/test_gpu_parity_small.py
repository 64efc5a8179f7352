"""GPU parity of the whole path against the oracle, element by element, at
sizes the oracle finishes in seconds (several tiles, ragged tails)."""

import dataclasses

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_helpers import (BF16_RTOL, F32_RTOL, assert_close, check_routing_and_queues, log, make_context,
                         oracle_routed_layer, run_routed_layer, to_dev, to_host, upload_weights)

pytestmark = pytest.mark.gpu

W = synth.Workload
SMALL = {
    "c1": synth.workload("c1"),
    "c1f4": synth.workload("c1f4"),
    # bf16, several 256-row tiles for the hot expert, f = 640 -> 5 gate/up
    # column tiles, d = 512 -> 2 down column tiles, ragged row tails
    "mid": W("mid", 101, d=512, f=640, E=8, k=2, zipf_s=1.2, tokens=(700,), n_frag=3),
    # shared experts, top-4 of 16, a 1-token fragment
    "mid_shared": W("mid_shared", 102, d=256, f=384, E=16, S=2, k=4, zipf_s=1.1, tokens=(301,), n_frag=2),
    # no renormalisation, top-3, f not a multiple of 128 (ragged gate/up columns)
    "mid_norenorm": W("mid_norenorm", 103, d=256, f=448, E=6, k=3, zipf_s=1.0, tokens=(260,), n_frag=1,
                      renorm=False),
    # 64 experts (the widest router), top-6, one fragment of 33 tokens
    "mid_e64": W("mid_e64", 104, d=128, f=192, E=64, k=6, zipf_s=1.1, tokens=(33,), n_frag=1),
    # fp8 weights through the router
    "mid_fp8": W("mid_fp8", 105, d=384, f=512, E=8, k=2, zipf_s=1.2, wdt="fp8", tokens=(530,), n_frag=2),
    # fp8 with K shorter than the prefetch distance of the small-tile ring
    # (d = 128: 2 K steps; f = 192: 3 K steps, ragged gate/up columns) and a
    # shared expert
    "short_fp8": W("short_fp8", 106, d=128, f=192, E=8, S=1, k=2, zipf_s=1.2, wdt="fp8", tokens=(300,),
                   n_frag=2),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_routed_layer_matches_oracle(name):
    w = SMALL[name]
    log(f"case {name}: T={w.tokens} d={w.d} f={w.f} E={w.E}+{w.S} k={w.k} {w.act}/{w.wdt}")
    frags = synth.layer_fragments(w, 0)
    ws = synth.all_expert_weights(w, 0, threads=4)
    ctx = make_context(w)
    upload_weights(ctx, w, 0, ws)
    got = run_routed_layer(ctx, w, 0, frags)
    ref = oracle_routed_layer(w, frags, ws)
    check_routing_and_queues(w, got, ref)
    rtol = F32_RTOL if w.act == "f32" else BF16_RTOL
    sy = assert_close(oracle.act_to_f64(got["y"], w.act), ref["y"], rtol, f"{name} y")
    so = assert_close(oracle.act_to_f64(got["out"], w.act), ref["out"], rtol, f"{name} out")
    log(f"case {name}: y {sy}  out {so}")


def test_rows_mode_fp8_and_bf16_match_oracle():
    base = W("rows_small", 106, d=256, f=320, E=5, k=1, zipf_s=1.3, mode="rows", depth_max=600)
    for wdt in ("bf16", "fp8"):
        w = dataclasses.replace(base, wdt=wdt)
        rw = synth.rows_workload(w)
        log(f"rows case {wdt}: depths {rw['depths'].tolist()}")
        ws = synth.all_expert_weights(w, 0, threads=4)
        ctx = make_context(w)
        upload_weights(ctx, w, 0, ws)
        lq = oracle.LayerQueues(w.E, w.k)
        keep = []
        for e, ex in enumerate(rw["experts"]):
            rows, tok, gw = to_dev(ex["x"], "bf16"), to_dev(ex["token_ids"], "i32"), to_dev(ex["gate_w"], "f32")
            keep.append((rows, tok, gw))
            ctx.enqueue_rows(0, e, rows, tok, gw, rw["n_tokens"])
            lq.enqueue_rows(e, ex["x"], ex["token_ids"], ex["gate_w"], rw["n_tokens"])
        b = ctx.rebatch(0)
        y = ctx.expert_ffn(b)
        out = ctx.combine(b, y)
        ref = oracle.moe_layer(lq, ws, "bf16", wdt)
        assert np.array_equal(to_host(b.counts()), ref["batch"].counts)
        assert np.array_equal(to_host(b.x_perm()), ref["xp"])
        assert np.array_equal(to_host(b.token_pos()), ref["batch"].pos)
        assert_close(oracle.bf16_to_f64(to_host(y)), ref["y"], BF16_RTOL, f"rows {wdt} y")
        assert_close(oracle.bf16_to_f64(to_host(out)), ref["out"], BF16_RTOL, f"rows {wdt} out")
        ctx.release(b)
        ctx.sync()


def test_fp8_decode_all_codes():
    import paper_2505_08944_amd as aep
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8).cuda()
    got = oracle.bf16_to_f64(to_host(aep.fp8_e4m3_to_bf16(codes)))
    ref = oracle.e4m3_to_f64(np.arange(256, dtype=np.uint8))
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    m = ~np.isnan(ref)
    assert np.array_equal(got[m], ref[m]) and np.array_equal(np.signbit(got[m]), np.signbit(ref[m]))


def test_top1_combine_is_the_expert_row_and_down_scaling_is_exact():
    w = W("top1", 107, d=256, f=256, E=4, k=1, zipf_s=1.0, tokens=(300,), n_frag=1)
    frags = synth.layer_fragments(w, 0)
    ws = synth.all_expert_weights(w, 0, threads=2)
    ctx = make_context(w)
    upload_weights(ctx, w, 0, ws)
    got = run_routed_layer(ctx, w, 0, frags)
    assert np.array_equal(got["out"], got["y"][got["pos"][:, 0]])  # w = 1 exactly
    # doubling W_down doubles y and out exactly
    ws2 = [dict(e, down=synth.round_to_bf16_bits(synth.bf16_bits_to_f32(e["down"]) * np.float32(2))) for e in ws]
    upload_weights(ctx, w, 0, ws2)
    got2 = run_routed_layer(ctx, w, 0, frags)
    y1, y2 = oracle.bf16_to_f64(got["y"]), oracle.bf16_to_f64(got2["y"])
    assert np.array_equal(y2, 2 * y1)
    assert np.array_equal(oracle.bf16_to_f64(got2["out"]), 2 * oracle.bf16_to_f64(got["out"]))


def test_run_twice_is_bit_identical():
    w = SMALL["mid_shared"]
    frags = synth.layer_fragments(w, 0)
    ws = synth.all_expert_weights(w, 0, threads=4)
    ctx = make_context(w)
    upload_weights(ctx, w, 0, ws)
    a = run_routed_layer(ctx, w, 0, frags)
    b = run_routed_layer(ctx, w, 0, frags)
    for key in ("x_perm", "y", "out", "pos", "posw"):
        assert np.array_equal(a[key], b[key]), key
