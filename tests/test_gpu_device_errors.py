"""GPU: bad input that only the device sees (a non-finite logit, a token id
or slot out of range) sets the context's error flag.  The next aep_sync
reports it once as AEP_ERR_DEVICE and clears it; the offending value was
clamped, so every access stayed in bounds and the rest of the fragment is
routed exactly as the oracle routes it."""

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_helpers import log, make_context, to_dev, to_host, upload_weights
from paper_2505_08944_amd._lib import AEPError

pytestmark = pytest.mark.gpu

AEP_ERR_DEVICE = 5


def _expect_device_error(ctx):
    with pytest.raises(AEPError) as ei:
        ctx.sync()
    assert ei.value.status == AEP_ERR_DEVICE
    ctx.sync()  # reported once: the flag is clear again


def test_non_finite_logits_are_reported_and_clamped():
    w = synth.Workload("err_route", 120, d=128, f=128, E=8, k=2, zipf_s=1.0, tokens=(64,), n_frag=1)
    fr = synth.layer_fragments(w, 0)[0]
    lg = fr["logits"].copy()
    lg[5, 3] = np.nan          # one expert of token 5 unusable
    lg[9, :] = np.inf          # every expert of token 9 non-finite
    lg[17, 6] = -np.inf
    log("case err_route: NaN / +inf / -inf logits in tokens 5, 9, 17")
    ws = synth.all_expert_weights(w, 0, threads=4)
    ctx = make_context(w)
    dev_w = upload_weights(ctx, w, 0, ws)
    x = to_dev(fr["x"], "bf16")
    idx, wt = ctx.route_enqueue(0, x, to_dev(lg, "f32"), routing_out=True)
    _expect_device_error(ctx)
    gi, gw = to_host(idx), to_host(wt)
    # a non-finite logit ranks below every finite one; the device reads it
    # as the lowest finite float, so ties among such logits go to the lower id
    clean = np.where(np.isfinite(lg), lg, np.float32(-np.finfo(np.float32).max))
    ok = np.ones(w.tokens[0], bool)
    ok[[5, 9, 17]] = False
    ref_idx, ref_w = oracle.route(clean[ok], w.k, w.renorm)
    assert np.array_equal(gi[ok], ref_idx)
    np.testing.assert_allclose(gw[ok], ref_w, rtol=4e-6, atol=0)
    # token 5 / 17: the top 2 of the 7 finite logits, as if the bad one were absent
    for t, bad_e in ((5, 3), (17, 6)):
        keep = [e for e in range(w.E) if e != bad_e]
        ri, _ = oracle.route(lg[t:t + 1, keep], w.k, w.renorm)
        assert np.array_equal(gi[t], np.asarray(keep)[ri[0]]), (t, gi[t])
    # token 9: all equal, so experts 0 and 1 with weight 1/2 each
    assert np.array_equal(gi[9], [0, 1]) and np.allclose(gw[9], 0.5)
    # the layer still drains and combines; outputs are finite
    b = ctx.rebatch(0)
    out = ctx.combine(b, ctx.expert_ffn(b))
    ctx.release(b)
    ctx.sync()
    assert np.all(np.isfinite(oracle.act_to_f64(to_host(out), "bf16")))
    del ctx, dev_w


def test_rows_out_of_range_are_reported_and_clamped():
    w = synth.Workload("err_rows", 121, d=128, f=128, E=4, k=2, zipf_s=1.0, mode="rows", depth_max=64)
    ws = synth.all_expert_weights(w, 0, threads=4)
    n_tok = 40
    ctx = make_context(w, max_tokens=n_tok)
    dev_w = upload_weights(ctx, w, 0, ws)
    g = np.random.default_rng(7)
    rows = to_dev(synth.round_to_bf16_bits(g.standard_normal((3, w.d), dtype=np.float32)), "bf16")
    gw = to_dev(np.ones(3, np.float32), "f32")
    # token n_tok is one past the last id; slot 2 is one past top-2
    log("case err_rows: token id and slot one past their ranges")
    ctx.enqueue_rows(0, 1, rows, to_dev(np.array([3, n_tok, 4], np.int32), "i32"), gw, n_tok,
                     slots=to_dev(np.array([0, 0, 2], np.int32), "i32"))
    _expect_device_error(ctx)
    # the clamped rows are filed under token 0 / slot 0: the drain still runs
    b = ctx.rebatch(0)
    assert int(to_host(b.counts())[1]) == 3
    tok = to_host(b.row_token())
    assert sorted(tok[:3].tolist()) == [0, 3, 4]
    ctx.expert_ffn(b)
    ctx.release(b)
    ctx.sync()
    del ctx, dev_w
