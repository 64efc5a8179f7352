"""GPU parity at the full workload sizes, in the launch configuration bench.py
times (fragments routed into the mu-queues, re-batch, gate/up + down, combine).

Routing, counts, offsets, row order, (token, slot) positions and the gathered
rows are compared bit-exactly with the oracle over the whole layer.  Outputs
are compared on sampled tokens, which the oracle evaluates one by one with the
dense brute force (every expert on the token, masked by its routing), and by
properties that hold at any size (drain-order invariance, determinism).
"""

import gc

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_helpers import (BF16_RTOL, assert_close, check_routing_and_queues, log, make_context,
                         oracle_routed_layer, run_routed_layer, to_dev, to_host, upload_weights)

pytestmark = pytest.mark.gpu


def _free():
    gc.collect()
    torch.cuda.empty_cache()


def _sample_tokens(ref_batch, T, n=48):
    """Tokens to check one by one: spread over the layer, plus the first and
    last token and the first/last rows of every expert's segment."""
    pick = set(np.linspace(0, T - 1, n).astype(int).tolist())
    b = ref_batch
    E = len(b.counts) - b.S
    for e in range(E):
        if b.counts[e]:
            pick.add(int(b.row_token[b.offsets[e]]))
            pick.add(int(b.row_token[b.offsets[e] + b.counts[e] - 1]))
    return np.array(sorted(pick))


def _check_sampled(w, frags, ws, got_out, ref_batch, n=48):
    x = np.concatenate([f["x"] for f in frags])
    lg = np.concatenate([f["logits"] for f in frags])
    toks = _sample_tokens(ref_batch, x.shape[0], n)
    ref = oracle.brute_dense(x[toks], lg[toks], ws, w.k, w.renorm, w.S, w.act, w.wdt)
    return assert_close(oracle.act_to_f64(got_out[toks], w.act), ref, BF16_RTOL,
                        f"{w.name}: {len(toks)} sampled tokens")


@pytest.mark.parametrize("name", ["c2", "c3"])
def test_full_routed_layer(name):
    w = synth.workload(name)
    log(f"case {name}: {w.description}")
    frags = synth.layer_fragments(w, 0)
    ws = synth.all_expert_weights(w, 0, threads=16)
    ctx = make_context(w)
    dev = upload_weights(ctx, w, 0, ws)
    got = run_routed_layer(ctx, w, 0, frags)
    log(f"case {name}: GPU done, counts {got['counts'].tolist()}")
    ref = oracle_routed_layer(w, frags, ws, full_ffn=False)
    check_routing_and_queues(w, got, ref)
    log(f"case {name}: routing/queues/gather bit-exact")
    st = _check_sampled(w, frags, ws, got["out"], ref["batch"])
    log(f"case {name}: sampled outputs {st}")
    assert np.all(np.isfinite(oracle.act_to_f64(got["out"], w.act)))
    del ctx, dev
    _free()


@pytest.mark.parametrize("name", ["c4", "c4fp8"])
def test_full_rows_layer(name):
    """One GPU's expert-parallel share: explicit per-expert queues (Zipf depths
    4096..111), every row its own output slot."""
    w = synth.workload(name)
    log(f"case {name}: {w.description}")
    rw = synth.rows_workload(w)
    ws = synth.all_expert_weights(w, 0, threads=16)
    ctx = make_context(w)
    dev = upload_weights(ctx, w, 0, ws)
    keep = []
    lq = oracle.LayerQueues(w.E, w.k)
    for e, ex in enumerate(rw["experts"]):
        t = (to_dev(ex["x"], "bf16"), to_dev(ex["token_ids"], "i32"), to_dev(ex["gate_w"], "f32"))
        keep.append(t)
        ctx.enqueue_rows(0, e, *t, rw["n_tokens"])
        lq.enqueue_rows(e, ex["x"], ex["token_ids"], ex["gate_w"], rw["n_tokens"])
    b = ctx.rebatch(0)
    y = ctx.expert_ffn(b)
    out = ctx.combine(b, y)
    ref_b = oracle.rebatch(lq)
    ref_xp = oracle.gather(ref_b)
    assert np.array_equal(to_host(b.counts()), ref_b.counts)
    assert np.array_equal(to_host(b.offsets()), ref_b.offsets.astype(np.int32))
    assert np.array_equal(to_host(b.row_token()), ref_b.row_token)
    assert np.array_equal(to_host(b.token_pos()), ref_b.pos)
    assert np.array_equal(to_host(b.x_perm()), ref_xp)
    log(f"case {name}: queues/gather bit-exact, depths {rw['depths'].tolist()}")
    # sampled rows of every expert: first, last and a few in between
    yh, oh = to_host(y), to_host(out)
    rows = []
    for e in range(w.E):
        o, n = int(ref_b.offsets[e]), int(ref_b.counts[e])
        rows += sorted(set([o, o + n - 1] + [o + (n * q) // 5 for q in range(1, 5)]))
    rows = np.array(rows)
    ref_y = np.zeros((len(rows), w.d))
    for e in range(w.E):
        m = (rows >= ref_b.offsets[e]) & (rows < ref_b.offsets[e + 1])
        if m.any():
            ref_y[m] = oracle.swiglu(oracle.bf16_to_f64(ref_xp[rows[m]]), *oracle.weights_to_f64(ws[e], w.wdt))
    sy = assert_close(oracle.bf16_to_f64(yh[rows]), ref_y, BF16_RTOL, f"{name} sampled y rows")
    toks = ref_b.row_token[rows]
    ref_out = ref_b.row_w[rows].astype(np.float64)[:, None] * ref_y
    so = assert_close(oracle.bf16_to_f64(oh[toks]), ref_out, BF16_RTOL, f"{name} sampled out rows")
    log(f"case {name}: y {sy} out {so}")
    ctx.release(b)
    ctx.sync()
    del ctx, dev, keep
    _free()


def test_c5_multi_layer_drain():
    """Eight layers queued at once (0..8192 tokens each, 32768 in total); the
    most-tokens-first policy drains them one by one.  Checks: the pick order,
    per-layer queues bit-exact, sampled outputs on three layers against the
    dense brute force, and bit-identical layer outputs when the same queues
    are drained in the opposite order."""
    w = synth.workload("c5")
    log(f"case c5: layer tokens {w.tokens}")
    base = synth.all_expert_weights(synth.workload("c2"), 0, threads=16)  # rotated per layer
    ctx = make_context(w)
    base_dev = [[to_dev(ex[k], "bf16") for k in ("gate", "up", "down")] for ex in base]
    wdev = []
    for l in range(w.n_layers):
        for e in range(w.E):
            src = synth.weight_source(w, l, e)[2]
            t = [m.clone() for m in base_dev[src]]          # every (layer, expert) its own copy
            ctx.set_expert_weights(l, e, *t)
            wdev.append(t)
    frags = [synth.layer_fragments(w, l) for l in range(w.n_layers)]
    dev_frags = [[(to_dev(f["x"], "bf16"), to_dev(f["logits"], "f32")) for f in fl] for fl in frags]

    def fill():
        for l in range(w.n_layers):
            for x, lg in dev_frags[l]:
                ctx.route_enqueue(l, x, lg)

    def drain(order_fn):
        outs, order = {}, []
        while True:
            l = order_fn()
            if l is None:
                break
            order.append(l)
            outs[l] = to_host(ctx.run_layer(l))
        ctx.sync()
        return outs, order

    fill()
    rows = [ctx.queue_depth(l)[1] for l in range(w.n_layers)]
    assert rows == [2 * t for t in w.tokens]
    gpu_counts = [ctx.expert_counts(l) for l in range(w.n_layers)]
    outs, order = drain(lambda: ctx.pick_layer("mtfs"))
    remaining, expect = [2 * t for t in w.tokens], []
    while (nxt := oracle.pick_mtfs(remaining)) is not None:
        expect.append(nxt)
        remaining[nxt] = 0
    assert order == expect
    log(f"case c5: MTFS drain order {order}")
    # reverse drain order: identical per-layer outputs, bit for bit
    fill()
    outs2, order2 = drain(lambda: max([l for l in range(w.n_layers) if ctx.queue_depth(l)[1] > 0], default=None))
    assert order2 == sorted(order, reverse=True)
    for l in order:
        assert np.array_equal(outs[l], outs2[l]), f"layer {l} differs between drain orders"
    log("case c5: drain-order invariance bit-exact")
    # oracle: per-expert queue depths of every layer bit-exact; sampled
    # outputs on 3 layers
    for l in range(w.n_layers):
        lq = oracle.LayerQueues(w.E, w.k)
        for fr in frags[l]:
            lq.enqueue_routed(fr["x"], fr["logits"])
        b = oracle.rebatch(lq) if w.tokens[l] else None
        ref_counts = b.counts if b is not None else np.zeros(w.E, np.int32)
        assert np.array_equal(gpu_counts[l], ref_counts), (l, gpu_counts[l], ref_counts)
    lws = lambda l: [base[synth.weight_source(w, l, e)[2]] for e in range(w.E)]
    for l in order[:1] + order[len(order) // 2:len(order) // 2 + 1] + order[-1:]:
        x = np.concatenate([f["x"] for f in frags[l]])
        lg = np.concatenate([f["logits"] for f in frags[l]])
        toks = np.unique(np.linspace(0, x.shape[0] - 1, 16).astype(int))
        ref = oracle.brute_dense(x[toks], lg[toks], lws(l), w.k, w.renorm, 0, "bf16", "bf16")
        st = assert_close(oracle.bf16_to_f64(outs[l][toks]), ref, BF16_RTOL, f"c5 layer {l} sampled")
        log(f"case c5: layer {l} sampled {st}")
    del ctx, wdev, base_dev
    _free()
