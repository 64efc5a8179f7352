"""GPU parity of the token pool: a layer fed with caller token ids and drained
one expert at a time; each token's k expert rows are merged in its pool row
and the token is released when the last of its experts has run.

Checked against the oracle:
* readiness, bit-exact: after every drain the released ids are exactly the
  tokens whose last routed expert has just been drained (the routing comes
  from the oracle's top-k), and rows of tokens not released are untouched;
* values: a released token's output equals the dense definition of the layer
  (every expert on the token, masked by its routing, oracle.brute_dense)
  within the tolerance of its precision;
* ids are reusable after release; an id enqueued again before its release is
  reported by aep_sync; the whole-layer calls refuse a pool-mode layer.
"""

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_helpers import BF16_RTOL, F32_RTOL, assert_close, log, to_dev, to_host, upload_weights
from paper_2505_08944_amd import AEPError, Context

pytestmark = pytest.mark.gpu

W = synth.Workload
CASES = {
    "bf16": W("pool_bf16", 107, d=256, f=384, E=8, k=2, zipf_s=1.2, tokens=(300,), n_frag=3),
    "f32": W("pool_f32", 108, d=256, f=512, E=8, k=2, zipf_s=1.0, tokens=(200,), n_frag=3, act="f32",
             wdt="f32"),
    "top3_norenorm": W("pool_k3", 109, d=192, f=256, E=6, k=3, zipf_s=1.1, tokens=(150,), n_frag=3,
                       renorm=False),
}
TMAX = 512


def _ctx(w):
    return Context(1, w.E, w.d, w.f, w.k, renorm=w.renorm, act=w.act, wdt=w.wdt, max_tokens_per_layer=TMAX,
                   token_pool=True)


@pytest.mark.parametrize("name", list(CASES))
def test_pool_release_matches_oracle(name):
    w = CASES[name]
    log(f"case {name}: d={w.d} f={w.f} E={w.E} k={w.k} {w.act}/{w.wdt}")
    frags = synth.layer_fragments(w, 0)
    ws = synth.all_expert_weights(w, 0, threads=4)
    ctx = _ctx(w)
    dev_w = upload_weights(ctx, w, 0, ws)
    T = sum(f["x"].shape[0] for f in frags)
    ids = np.random.default_rng(w.cfg_id).permutation(TMAX)[:T].astype(np.int32)
    x_all = np.concatenate([f["x"] for f in frags])
    lg_all = np.concatenate([f["logits"] for f in frags])
    idx, _ = oracle.route(lg_all, w.k, w.renorm)
    ref = oracle.brute_dense(x_all, lg_all, ws, w.k, w.renorm, 0, w.act, w.wdt)
    rtol = F32_RTOL if w.act == "f32" else BF16_RTOL
    act = torch.float32 if w.act == "f32" else torch.bfloat16
    out = torch.full((TMAX, w.d), float("nan"), dtype=act, device="cuda")
    ready = torch.zeros(TMAX, dtype=torch.int32, device="cuda")
    remaining = {}                      # token -> experts still to run
    released = set()
    keep = []
    starts = np.cumsum([0] + [f["x"].shape[0] for f in frags])

    def enqueue(fi):
        f = frags[fi]
        t0, t1 = starts[fi], starts[fi + 1]
        tens = (to_dev(f["x"], w.act), to_dev(f["logits"], "f32"), to_dev(ids[t0:t1], "i32"))
        keep.append(tens)
        ctx.route_enqueue_ids(0, *tens)
        for t in range(t0, t1):
            remaining[t] = set(int(e) for e in idx[t])

    def drain(e):
        b = ctx.rebatch_expert(0, e)
        y = ctx.expert_ffn(b)
        ctx.pool_accumulate(b, y)
        ctx.release(b)
        ctx.pool_release(0, out, ready)
        done = set()
        for t, rem in remaining.items():
            if e in rem:
                rem.discard(e)
                if not rem:
                    done.add(t)
        for t in done:
            del remaining[t]
        got_ready = set(np.nonzero(to_host(ready))[0].tolist())
        assert got_ready == {int(ids[t]) for t in done}, (e, sorted(got_ready), sorted(ids[list(done)]))
        released.update(done)

    def drain_if_queued(e):
        if ctx.queue_depth(0)[1] == 0:
            return
        try:
            drain(e)
        except AEPError as err:
            assert err.status == 3          # AEP_ERR_EMPTY: nothing known to be queued for e

    # fragments arrive between drains; experts drained in a mixed order
    enqueue(0)
    for e in (3, 0, 5):
        drain_if_queued(e % w.E)
    enqueue(1)
    for e in (7, 1, 3):
        drain_if_queued(e % w.E)
    enqueue(2)
    for e in range(w.E):
        drain_if_queued(e)
    assert ctx.queue_depth(0)[1] == 0 and not remaining
    ctx.sync()
    o = oracle.act_to_f64(to_host(out), w.act)
    toks = np.array(sorted(released))
    st = assert_close(o[ids[toks]], ref[toks], rtol, f"{name} released tokens")
    log(f"case {name}: {len(toks)} tokens released; {st}")
    unused = np.setdiff1d(np.arange(TMAX), ids)
    assert np.all(np.isnan(o[unused])), "rows of ids never used must be untouched"
    del ctx, dev_w, keep


def test_pool_ids_reusable_collision_and_state_errors():
    w = CASES["bf16"]
    frags = synth.layer_fragments(w, 0)
    ws = synth.all_expert_weights(w, 0, threads=4)
    ctx = _ctx(w)
    dev_w = upload_weights(ctx, w, 0, ws)
    f = frags[0]
    n = f["x"].shape[0]
    x, lg = to_dev(f["x"], "bf16"), to_dev(f["logits"], "f32")
    ids = to_dev(np.arange(n, dtype=np.int32), "i32")
    ctx.route_enqueue_ids(0, x, lg, ids)
    # whole-layer calls refuse a pool-mode layer
    for call in (lambda: ctx.rebatch(0), lambda: ctx.route_enqueue(0, x, lg)):
        with pytest.raises(AEPError) as ei:
            call()
        assert ei.value.status == 4   # AEP_ERR_STATE
    out = torch.zeros((TMAX, w.d), dtype=torch.bfloat16, device="cuda")
    ready = torch.zeros(TMAX, dtype=torch.int32, device="cuda")
    for e in range(w.E):
        if ctx.queue_depth(0)[1] == 0:
            break
        b = ctx.rebatch_expert(0, e)
        y = ctx.expert_ffn(b)
        with pytest.raises(AEPError) as ei:
            ctx.combine(b, y)
        assert ei.value.status == 4
        ctx.pool_accumulate(b, y)
        ctx.release(b)
    ctx.pool_release(0, out, ready)
    ctx.sync()
    assert int(to_host(ready).sum()) == n
    first = to_host(out)[:n].copy()
    # the ids are free again: the same fragment runs again to the same outputs
    ctx.route_enqueue_ids(0, x, lg, ids)
    for e in range(w.E):
        if ctx.queue_depth(0)[1] == 0:
            break
        b = ctx.rebatch_expert(0, e)
        ctx.pool_accumulate(b, ctx.expert_ffn(b))
        ctx.release(b)
    ctx.pool_release(0, out, ready)
    ctx.sync()
    assert np.array_equal(to_host(out)[:n], first)
    # an id enqueued twice before its release is a device-reported error
    ctx.route_enqueue_ids(0, x[:4], lg[:4], ids[:4])
    ctx.route_enqueue_ids(0, x[:1], lg[:1], ids[:1])
    with pytest.raises(AEPError) as ei:
        ctx.sync()
    assert ei.value.status == 5       # AEP_ERR_DEVICE
    del ctx, dev_w
