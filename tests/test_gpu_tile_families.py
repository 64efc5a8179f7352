"""GPU parity of every row-tile choice the plan makes, on explicit per-expert
queue depths (rows mode), against the oracle element by element.

Cold batch (its full 256-row tiles do not fill one round of the grid): a
remainder above 128 rows takes one tall 256-row tile, 65..128 rows one medium
tile, 1..64 rows one small tile.  Warm batch, per FFN stage: a remainder
above 128 rows takes one more big tile (rule B), unless those extra big
tiles would start another round of the grid in a stage with fewer than 4
rounds; then only a remainder above 192 rows does (rule A) and the others
take medium tiles and at most one small tile.  The depths below put at least
one expert on each branch (and exact multiples of 256, and empty experts),
for bf16 and fp8 weights; the mixed batch splits the same remainder
differently in its two stages."""

import dataclasses

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_helpers import BF16_RTOL, assert_close, log, make_context, to_dev, to_host, upload_weights

pytestmark = pytest.mark.gpu

COLD = [300, 200, 100, 40, 1, 256, 0, 129]          # big+small, tall, medium, small, small, big, -, tall
# rule B in both stages: 8 big + small, big, big, big + small, big + small, -,
# 2 big, big, medium
WARM = [2100, 230, 150, 300, 260, 0, 512, 193, 100]
# d = 512, f = 896: 128 big row tiles under rule A, 129 under rule B.  Gate/up
# (7 big column tiles) has 4 rounds either way: rule B, so the 150-row
# remainder takes a big tile.  Down (2 big column tiles) would go from 1 round
# to 2: rule A, so that remainder takes a medium and a small tile.
MIXED = [2048] * 13 + [2198, 2148, 2088]


def _rows(w, depths, seed):
    g = np.random.default_rng(seed)
    N = int(sum(depths))
    tok = g.permutation(N).astype(np.int32)
    gw = g.random(N, dtype=np.float32)
    x = synth.round_to_bf16_bits(g.standard_normal((N, w.d), dtype=np.float32))
    per, r0 = [], 0
    for n in depths:
        per.append({"x": x[r0:r0 + n], "token_ids": tok[r0:r0 + n], "gate_w": gw[r0:r0 + n]})
        r0 += n
    return N, per


@pytest.mark.parametrize("kind,wdt", [("cold", "bf16"), ("cold", "fp8"), ("warm", "bf16"), ("warm", "fp8"),
                                      ("mixed", "bf16"), ("short1", "bf16"), ("short1", "fp8"),
                                      ("short2", "bf16"), ("short2", "fp8")])
def test_tile_families_match_oracle(kind, wdt):
    # short1 / short2: the cold depths with K of 1, 2 or 3 steps of 64 in the
    # two stages, fewer than every ring's stages (the first pass of a refill
    # repeats loads of the prologue; past the last step loads repeat it)
    depths = {"cold": COLD, "warm": WARM, "mixed": MIXED, "short1": COLD, "short2": COLD}[kind]
    # warm: f = 8192 gives 64 big gate/up column tiles, so 8 + 2 + 1 + 1 + 1
    # full 256-row blocks fill more than one round of 256 CUs
    d, f = {"cold": (256, 320), "warm": (256, 8192), "mixed": (512, 896), "short1": (64, 192),
            "short2": (128, 64)}[kind]
    w = synth.Workload(f"fam_{kind}_{wdt}", 110, d=d, f=f, E=len(depths), k=1, zipf_s=1.0, mode="rows",
                       depth_max=max(depths), wdt=wdt)
    N, per = _rows(w, depths, {"cold": 11, "warm": 12, "mixed": 13, "short1": 14, "short2": 15}[kind])
    log(f"case {kind}/{wdt}: depths {depths}, d={w.d} f={w.f}")
    ws = synth.all_expert_weights(w, 0, threads=4)
    ctx = make_context(w, max_tokens=N)
    dev_w = upload_weights(ctx, w, 0, ws)
    lq = oracle.LayerQueues(w.E, 1)
    keep = []
    for e, ex in enumerate(per):
        if depths[e] == 0:
            continue
        t = (to_dev(ex["x"], "bf16"), to_dev(ex["token_ids"], "i32"), to_dev(ex["gate_w"], "f32"))
        keep.append(t)
        ctx.enqueue_rows(0, e, *t, N)
        lq.enqueue_rows(e, ex["x"], ex["token_ids"], ex["gate_w"], N)
    b = ctx.rebatch(0)
    y = ctx.expert_ffn(b)
    ref = oracle.moe_layer(lq, ws, "bf16", wdt)
    assert np.array_equal(to_host(b.counts()), ref["batch"].counts)
    st = assert_close(oracle.bf16_to_f64(to_host(y)), ref["y"], BF16_RTOL, f"{kind}/{wdt} y")
    log(f"case {kind}/{wdt}: y {st}")
    ctx.release(b)
    ctx.sync()
    del ctx, dev_w, keep


# Split-K: a launch of at most half a grid of tiles cuts every tile into
# n_split = min(4, grid / tiles, K / 512) pieces of consecutive K steps (the
# slot area permitting); the last piece to finish adds the pieces' f32
# partial sums in piece order.  Each case below puts at most 128 tiles into
# at least one launch with K >= 1024, on the families named.
SPLIT_CASES = {
    # 2 experts x 16 rows, small tiles: gate/up 32 tiles in 4 pieces, down 32 in 2
    "small": ([16, 16], 2048, 1024),
    # medium (100 rows) and tall (200 rows) tiles of a cold batch, 4 pieces
    "medium_tall": ([100, 200], 2048, 1024),
    # one 256-row expert: 16 big gate/up tiles in 2 pieces, 4 big down tiles in 4
    "big": ([256], 1024, 2048),
    # every family in one launch (big + medium, small, tall; an empty expert):
    # 56 gate/up and 28 down tiles, 2 pieces each
    "mixed": ([356, 30, 0, 200], 1024, 1024),
    # 100 big gate/up tiles (f = 12800): 2 pieces would need 50 MB of partial
    # sums, more than the 32 MB area, so that launch is not split; the down
    # launch (4 big tiles, K = 12800) is, in 4 pieces
    "area_cap": ([256], 1024, 12800),
}


@pytest.mark.parametrize("kind,wdt", [("small", "bf16"), ("small", "fp8"), ("medium_tall", "bf16"),
                                      ("medium_tall", "fp8"), ("big", "bf16"), ("big", "fp8"),
                                      ("mixed", "bf16"), ("mixed", "fp8"), ("area_cap", "bf16")])
def test_split_k_matches_oracle(kind, wdt):
    """Every element of y against the oracle, and a second run of the same
    batch bit-identical (the pieces are added in a fixed order, whichever
    finishes last)."""
    depths, d, f = SPLIT_CASES[kind]
    w = synth.Workload(f"split_{kind}_{wdt}", 111, d=d, f=f, E=len(depths), k=1, zipf_s=1.0, mode="rows",
                       depth_max=max(depths), wdt=wdt)
    N, per = _rows(w, depths, 21)
    log(f"case split {kind}/{wdt}: depths {depths}, d={d} f={f}")
    ws = synth.all_expert_weights(w, 0, threads=4)
    ctx = make_context(w, max_tokens=N)
    dev_w = upload_weights(ctx, w, 0, ws)
    lq = oracle.LayerQueues(w.E, 1)
    keep = []
    for e, ex in enumerate(per):
        if depths[e] == 0:
            continue
        t = (to_dev(ex["x"], "bf16"), to_dev(ex["token_ids"], "i32"), to_dev(ex["gate_w"], "f32"))
        keep.append((e, t))
        lq.enqueue_rows(e, ex["x"], ex["token_ids"], ex["gate_w"], N)
    ys = []
    for rep in range(2):
        for e, t in keep:
            ctx.enqueue_rows(0, e, *t, N)
        b = ctx.rebatch(0)
        ys.append(to_host(ctx.expert_ffn(b)))
        ctx.release(b)
    ctx.sync()
    ref = oracle.moe_layer(lq, ws, "bf16", wdt)
    st = assert_close(oracle.bf16_to_f64(ys[0]), ref["y"], BF16_RTOL, f"split {kind}/{wdt} y")
    assert np.array_equal(ys[0], ys[1]), "split-K results differ between runs"
    log(f"case split {kind}/{wdt}: y {st}, bit-identical rerun")
    del ctx, dev_w, keep


# Expert shapes of the weight-streaming sweep at their real sizes (the bench
# runs more experts of each): same-shape experts of n rows each.  Mixtral
# shape, 4 x 16 rows: 448 small gate/up tiles, and a down launch of 128 small
# tiles (K = 14336) split in 2; EP-share shape with fp8 weights, 12 x 64
# rows: 192 wide (64 x 256) small tiles per launch, not split; and, smaller
# than any sweep shape so that its fp8 weights quantise in seconds, a long-K
# fp8 down launch of 16 wide tiles (K = 4096) split in 4.
SWEEP_CASES = {
    "d4096_f14336_bf16_n16": (4, 16, 4096, 14336, "bf16"),
    "d4096_f2048_fp8_n64": (12, 64, 4096, 2048, "fp8"),
    "d2048_f4096_fp8_n64": (2, 64, 2048, 4096, "fp8"),
}


@pytest.mark.parametrize("case", sorted(SWEEP_CASES))
def test_sweep_shapes_match_oracle(case):
    """Every element of y against the oracle at the sweep's expert shapes."""
    G, n, d, f, wdt = SWEEP_CASES[case]
    depths = [n] * G
    w = synth.Workload(f"sweep_{case}", 113, d=d, f=f, E=G, k=1, zipf_s=1.0, mode="rows", depth_max=n,
                       wdt=wdt)
    N, per = _rows(w, depths, 23)
    log(f"case sweep {case}: {G} experts x {n} rows, d={d} f={f} {wdt}")
    ws = synth.all_expert_weights(w, 0, threads=8)
    ctx = make_context(w, max_tokens=N)
    dev_w = upload_weights(ctx, w, 0, ws)
    lq = oracle.LayerQueues(w.E, 1)
    keep = []
    for e, ex in enumerate(per):
        t = (to_dev(ex["x"], "bf16"), to_dev(ex["token_ids"], "i32"), to_dev(ex["gate_w"], "f32"))
        keep.append(t)
        ctx.enqueue_rows(0, e, *t, N)
        lq.enqueue_rows(e, ex["x"], ex["token_ids"], ex["gate_w"], N)
    b = ctx.rebatch(0)
    y = to_host(ctx.expert_ffn(b))
    ctx.release(b)
    ctx.sync()
    ref = oracle.moe_layer(lq, ws, "bf16", wdt)
    st = assert_close(oracle.bf16_to_f64(y), ref["y"], BF16_RTOL, f"sweep {case} y")
    log(f"case sweep {case}: y {st}")
    del ctx, dev_w, keep, ws
