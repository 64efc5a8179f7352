"""aep_bind_static_workspace: a context on the library's static workspace
(nothing allocated by the binding) computes what a context on a caller-
allocated workspace computes.

Bindings in a row on the same GPU, the second with a smaller layer, the
third one whose FFN launches are split along K: each
static-workspace layer (route, re-batch, FFN, combine) is compared bit for bit
with the same layer on a torch-allocated workspace (same kernels, same
inputs) and within tolerance with the oracle.  The second binding takes the
array over: the first context's calls are then refused.  A configuration
whose workspace exceeds the array is refused with AEP_ERR_CAPACITY.
"""

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_helpers import BF16_RTOL, assert_close, log, make_context, to_dev, to_host, upload_weights
from paper_2505_08944_amd import AEPError, Context
from paper_2505_08944_amd import _lib as L

pytestmark = pytest.mark.gpu


def _static_context(w, max_tokens):
    return Context(w.n_layers, w.E, w.d, w.f, w.k, n_shared=w.S, renorm=w.renorm, act=w.act,
                   wdt=("fp8" if w.wdt == "fp8" else w.wdt), max_tokens_per_layer=max_tokens,
                   static_workspace=True)


def _layer(ctx, w, frags):
    xs = [(to_dev(f["x"], w.act), to_dev(f["logits"], "f32")) for f in frags]
    for x, lg in xs:
        ctx.route_enqueue(0, x, lg)
    b = ctx.rebatch(0)
    y = ctx.expert_ffn(b)
    out = ctx.combine(b, y)
    ctx.release(b)
    ctx.sync()
    return to_host(y), to_host(out)


def _oracle_out(w, frags, ws):
    lq = oracle.LayerQueues(w.E, w.k, w.S, w.renorm)
    for f in frags:
        lq.enqueue_routed(f["x"], f["logits"])
    return oracle.moe_layer(lq, ws, w.act, w.wdt)["out"]


def test_static_workspace_matches_allocated_workspace():
    cases = [
        synth.Workload("static_a", 501, d=512, f=1024, E=8, k=2, S=1, zipf_s=1.2, tokens=(700,), n_frag=3),
        synth.Workload("static_b", 502, d=256, f=384, E=16, k=4, zipf_s=1.1, wdt="fp8", tokens=(90,), n_frag=2),
        # 2 experts, 32 tokens, top-1: 32 small tiles per FFN launch with K of
        # 2048 and 1024, so both launches are split along K and their piece
        # counters live in the static array
        synth.Workload("static_c", 504, d=2048, f=1024, E=2, k=1, zipf_s=1.0, tokens=(32,), n_frag=1),
    ]
    first = None
    for w in cases:
        log(f"case {w.name}: T={w.tokens[0]} d={w.d} f={w.f} E={w.E}+{w.S} k={w.k} {w.act}/{w.wdt}")
        frags = synth.layer_fragments(w, 0)
        ws = synth.all_expert_weights(w, 0, threads=4)
        ref_ctx = make_context(w)
        dref = upload_weights(ref_ctx, w, 0, ws)
        y_ref, out_ref = _layer(ref_ctx, w, frags)
        sctx = _static_context(w, w.tokens[0])
        assert sctx.workspace_bytes <= L.AEP_STATIC_WORKSPACE_BYTES
        dst = upload_weights(sctx, w, 0, ws)
        y, out = _layer(sctx, w, frags)
        assert np.array_equal(y, y_ref) and np.array_equal(out, out_ref), "static and allocated workspaces differ"
        st = assert_close(oracle.act_to_f64(out, w.act), _oracle_out(w, frags, ws), BF16_RTOL, f"{w.name} out")
        log(f"case {w.name}: bit-identical to the allocated workspace; against the oracle {st}")
        if first is not None:
            # the second binding took the array over
            with pytest.raises(AEPError) as e:
                first.expert_counts(0)
            assert e.value.status == L.AEP_ERR_STATE
        first = sctx
        del ref_ctx, dref, dst
    # a workspace larger than the array is refused
    big = synth.Workload("static_big", 503, d=4096, f=14336, E=8, k=2, zipf_s=1.2, tokens=(4096,))
    with pytest.raises(AEPError) as e:
        _static_context(big, 4096)
    assert e.value.status == L.AEP_ERR_CAPACITY
    torch.cuda.synchronize()
