"""GPU tests of the C ABI's contract (Sec. 3.2: the executor drains a layer's
queues and releases the batch; Sec. 3.4: the scheduler picks the layer) and of
the router on inputs the workload generators do not produce.

* every host-detected error (capacity overflow on both enqueue calls, a drain
  of an empty layer, a drain while a batch is outstanding, a stale batch
  handle, a double release, FFN or combine on a released batch) returns its
  status and leaves the queues as they were: host totals, device per-expert
  depths, and the result of the next valid drain against the oracle;
* aep_pick_layer under all three policies equals the oracle's picks over the
  layer totals after every drain of a random multi-layer state;
* routing of tie-heavy finite logits (a 0.25 grid) is bit-exact against the
  oracle for E = 8, 16, 64 and k up to 8;
* the largest fragment aep_create accepts (2^24 - 1 tokens) routes, queues
  and re-batches bit-exactly (routing against the oracle's route; counts,
  offsets and row order against histogram, cumulative sum and stable sort of
  the flattened expert ids, the textbook routines that pin the oracle's
  queues), and its outputs agree on sampled tokens;
* rows of several experts enqueued in one call leave the queues exactly as
  one call per expert does.
"""

import ctypes
import time

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_helpers import (BF16_RTOL, W_RTOL, assert_close, log, make_context, to_dev, to_host,
                         upload_weights)
from paper_2505_08944_amd import AEPError
from paper_2505_08944_amd import _lib as L

pytestmark = pytest.mark.gpu


def _status(fn, *a, **kw):
    try:
        fn(*a, **kw)
    except AEPError as e:
        return e.status
    return L.AEP_OK


def _small_workload(T=96, E=4, k=2, n_frag=3, layers=1):
    return synth.Workload("contract", 401, d=64, f=128, E=E, k=k, zipf_s=1.1, tokens=(T,) * layers,
                          n_frag=n_frag)


def _state(ctx, layers):
    return [(ctx.queue_depth(l), ctx.expert_counts(l).tolist()) for l in range(layers)]


def _check_layer_against_oracle(ctx, w, frags, ws, layer=0):
    b = ctx.rebatch(layer)
    y = ctx.expert_ffn(b)
    out = ctx.combine(b, y)
    lq = oracle.LayerQueues(w.E, w.k)
    for fr in frags:
        lq.enqueue_routed(fr["x"], fr["logits"])
    ref = oracle.moe_layer(lq, ws, w.act, w.wdt)
    assert np.array_equal(to_host(b.counts()), ref["batch"].counts)
    assert np.array_equal(to_host(b.row_token()), ref["batch"].row_token)
    assert_close(oracle.bf16_to_f64(to_host(out)), ref["out"], BF16_RTOL, "layer after error paths")
    ctx.release(b)
    ctx.sync()


def test_error_paths_leave_state_unchanged():
    w = _small_workload(T=96, layers=2)
    frags = synth.layer_fragments(w, 0)
    ws = synth.all_expert_weights(w, 0, threads=4)
    ctx = make_context(w, max_tokens=128)
    dev = upload_weights(ctx, w, 0, ws)
    upload_weights(ctx, w, 1, ws)
    for fr in frags:
        ctx.route_enqueue(0, to_dev(fr["x"], "bf16"), to_dev(fr["logits"], "f32"))
    before = _state(ctx, 2)
    assert before[0][0] == (96, 192) and before[1][0] == (0, 0)

    # capacity: 96 + 33 tokens > 128
    big = synth.layer_fragments(_small_workload(T=33, n_frag=1), 0)[0]
    st = _status(ctx.route_enqueue, 0, to_dev(big["x"], "bf16"), to_dev(big["logits"], "f32"))
    assert st == L.AEP_ERR_CAPACITY
    assert _state(ctx, 2) == before
    # capacity on explicit rows: expert 0 could already hold 96 rows, 40 more exceed 128
    rows = to_dev(np.zeros((40, w.d), np.uint16), "bf16")
    ids = to_dev(np.arange(40, dtype=np.int32), "i32")
    gw = to_dev(np.ones(40, np.float32), "f32")
    assert _status(ctx.enqueue_rows, 0, 0, rows, ids, gw, 128) == L.AEP_ERR_CAPACITY
    assert _status(ctx.enqueue_rows, 0, 0, rows, ids, gw, 129) == L.AEP_ERR_CAPACITY   # n_tokens > capacity
    assert _state(ctx, 2) == before
    # drain of an empty layer
    assert _status(ctx.rebatch, 1) == L.AEP_ERR_EMPTY
    assert _state(ctx, 2) == before
    log("capacity and empty-drain errors: state unchanged")

    # a drain while a batch is outstanding; stale handle; double release;
    # FFN / combine on a released batch
    b = ctx.rebatch(0)
    assert ctx.queue_depth(0) == (0, 0)
    y = ctx.expert_ffn(b)
    assert _status(ctx.rebatch, 0) == L.AEP_ERR_STATE
    stale = L.Batch.from_buffer_copy(b.c)
    ctx.release(b)
    lib = L.lib()
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    assert lib.aep_release_batch(ctx.h, ctypes.byref(stale)) == L.AEP_ERR_STATE          # double release
    assert lib.aep_expert_ffn(ctx.h, ctypes.byref(stale), y.data_ptr(), s) == L.AEP_ERR_STATE
    out = torch.empty((stale.n_tokens, w.d), dtype=torch.bfloat16, device="cuda")
    assert lib.aep_combine(ctx.h, ctypes.byref(stale), y.data_ptr(), out.data_ptr(), s) == L.AEP_ERR_STATE
    # refill, drain again: the earlier handle now has a stale epoch
    for fr in frags:
        ctx.route_enqueue(0, to_dev(fr["x"], "bf16"), to_dev(fr["logits"], "f32"))
    refill = _state(ctx, 2)
    assert refill == before
    b2 = ctx.rebatch(0)
    assert stale.epoch != b2.c.epoch
    assert lib.aep_expert_ffn(ctx.h, ctypes.byref(stale), y.data_ptr(), s) == L.AEP_ERR_STATE
    assert lib.aep_combine(ctx.h, ctypes.byref(stale), y.data_ptr(), out.data_ptr(), s) == L.AEP_ERR_STATE
    assert lib.aep_release_batch(ctx.h, ctypes.byref(stale)) == L.AEP_ERR_STATE
    ctx.release(b2)
    ctx.sync()
    log("outstanding / stale / double-release errors refused")
    # the queues are intact: a valid drain still matches the oracle
    for fr in frags:
        ctx.route_enqueue(0, to_dev(fr["x"], "bf16"), to_dev(fr["logits"], "f32"))
    assert _state(ctx, 2) == before
    _check_layer_against_oracle(ctx, w, frags, ws)
    del ctx, dev


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_pick_layer_matches_oracle_after_every_drain(seed):
    """Random per-layer row counts (some layers empty); after each drain of
    the MTFS pick, every policy's pick (several delta / lookahead) equals the
    oracle's pick over the same layer totals."""
    g = np.random.default_rng(seed)
    NL, E = 7, 4
    w = synth.Workload("pick", 402, d=64, f=64, E=E, k=1, zipf_s=1.0, tokens=(1,) * NL)
    ctx = make_context(w, max_tokens=64)
    ws = synth.all_expert_weights(w, 0, threads=2)
    keep = [upload_weights(ctx, w, l, ws) for l in range(NL)]
    rows_of = np.zeros(NL, np.int64)
    bufs = []
    for l in range(NL):
        for e in range(E):
            n = int(g.integers(0, 16)) * int(g.random() < 0.7)
            if n:
                # distinct token ids per expert: (token, slot 0) is unique in the layer
                t = (to_dev(np.zeros((n, w.d), np.uint16), "bf16"),
                     to_dev(16 * e + np.arange(n, dtype=np.int32), "i32"), to_dev(np.ones(n, np.float32), "f32"))
                bufs.append(t)
                ctx.enqueue_rows(l, e, *t, 64)
                rows_of[l] += n
    params = [(0.5, 2), (1.0, 1), (0.9, 3), (0.0, 2), (0.75, 6)]
    drains = 0
    while True:
        R = rows_of.tolist()
        assert [ctx.queue_depth(l)[1] for l in range(NL)] == R
        assert ctx.pick_layer("mtfs") == oracle.pick_mtfs(R)
        assert ctx.pick_layer("flfs") == oracle.pick_flfs(R)
        for delta, la in params:
            assert ctx.pick_layer("defrag", delta, la) == oracle.pick_layer_defrag(R, delta, la), (R, delta, la)
        nxt = oracle.pick_mtfs(R)
        if nxt is None:
            break
        ctx.run_layer(nxt)
        rows_of[nxt] = 0
        drains += 1
    ctx.sync()
    log(f"seed {seed}: picks equal after each of {drains} drains")
    del ctx, keep, bufs


@pytest.mark.parametrize("E,k", [(8, 2), (8, 8), (16, 3), (16, 8), (64, 6), (64, 8), (64, 1)])
def test_router_tie_heavy_logits(E, k):
    """Logits on a coarse 0.25 grid (many exact ties): selection bit-exact
    against the oracle (ties -> lower expert id), weights within W_RTOL."""
    g = np.random.default_rng(1000 * E + k)
    T = 777
    logits = (np.round(g.normal(0, 0.6, (T, E)) * 4) / 4).astype(np.float32)
    logits[5] = 0.0                       # one token with every logit equal
    logits[6, :] = -1.0
    logits[6, E - 1] = 2.0
    w = synth.Workload("ties", 403, d=64, f=64, E=E, k=k, zipf_s=1.0, tokens=(T,))
    ctx = make_context(w, max_tokens=T)
    x = to_dev(np.zeros((T, 64), np.uint16), "bf16")
    idx, wt = ctx.route_enqueue(0, x, to_dev(logits, "f32"), routing_out=True)
    ridx, rw = oracle.route(logits, k, True)
    assert np.array_equal(to_host(idx), ridx)
    np.testing.assert_allclose(to_host(wt), rw, rtol=W_RTOL, atol=0)
    assert np.array_equal(ctx.expert_counts(0), np.bincount(ridx.ravel(), minlength=E))
    assert to_host(idx)[5].tolist() == list(range(k))
    ctx.sync()
    n_ties = int(sum(len(set(r.tolist())) < E for r in logits))
    log(f"E={E} k={k}: {n_ties} of {T} tokens hold tied logits; routing bit-exact")
    del ctx


def test_largest_fragment():
    """One fragment of 2^24 - 1 tokens (the largest aep_create accepts), E = 8,
    top-2, d = ffn = 64: routing, counts, offsets, row order, (token, slot)
    positions bit-exact; sampled gathered rows bit-exact; sampled outputs
    against the dense brute force."""
    T = (1 << 24) - 1
    w = synth.Workload("maxfrag", 404, d=64, f=64, E=8, k=2, zipf_s=1.2, tokens=(T,), n_frag=1)
    log(f"largest fragment: T={T}, generating inputs")
    fr = synth.layer_fragments(w, 0)[0]
    ws = synth.all_expert_weights(w, 0, threads=8)
    ctx = make_context(w, max_tokens=T)
    dev = upload_weights(ctx, w, 0, ws)
    x, lg = to_dev(fr["x"], "bf16"), to_dev(fr["logits"], "f32")
    # append time at two sizes on a scratch context (linear in T)
    small = make_context(w, max_tokens=T)
    sdev = upload_weights(small, w, 0, ws)
    times = {}
    for n in (T // 16, T):
        best = None
        for rep in range(2):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            small.route_enqueue(0, x[:n], lg[:n])
            torch.cuda.synchronize()
            dt = time.perf_counter() - t0
            best = dt if best is None else min(best, dt)
            small.run_layer(0)
        times[n] = best
    log(f"route + append: {T // 16} tokens {times[T // 16] * 1e3:.2f} ms, {T} tokens {times[T] * 1e3:.2f} ms")
    del small, sdev
    torch.cuda.empty_cache()
    idx, wt = ctx.route_enqueue(0, x, lg, routing_out=True)
    b = ctx.rebatch(0)
    y = ctx.expert_ffn(b)
    out = ctx.combine(b, y)
    torch.cuda.synchronize()
    log("largest fragment: GPU done")
    ridx, rw = oracle.route(fr["logits"], w.k, True)
    assert np.array_equal(to_host(idx), ridx)
    np.testing.assert_allclose(to_host(wt), rw, rtol=W_RTOL, atol=0)
    flat = ridx.ravel()
    counts = np.bincount(flat, minlength=w.E).astype(np.int32)
    assert np.array_equal(to_host(b.counts()), counts)
    assert np.array_equal(to_host(b.offsets()), np.concatenate([[0], np.cumsum(counts)]).astype(np.int32))
    order = np.argsort(flat, kind="stable")           # row r holds (token, slot) = divmod(order[r], k)
    assert np.array_equal(to_host(b.row_token()), (order // w.k).astype(np.int32))
    pos = np.empty(T * w.k, np.int32)
    pos[order] = np.arange(T * w.k, dtype=np.int32)
    assert np.array_equal(to_host(b.token_pos()).ravel(), pos)
    log("largest fragment: routing, counts, offsets, row order, positions bit-exact")
    g = np.random.default_rng(7)
    rows = np.unique(np.concatenate([g.integers(0, T * w.k, 2000), [0, T * w.k - 1],
                                     np.concatenate([[0], np.cumsum(counts)])[1:-1]]))
    xp = b.x_perm()
    assert np.array_equal(to_host(xp[torch.from_numpy(rows).cuda()]), fr["x"][order[rows] // w.k])
    toks = np.unique(np.concatenate([g.integers(0, T, 300), [0, T - 1]]))
    ref = oracle.brute_dense(fr["x"][toks], fr["logits"][toks], ws, w.k, w.renorm, 0, "bf16", "bf16")
    st = assert_close(oracle.bf16_to_f64(to_host(out[torch.from_numpy(toks).cuda()])), ref, BF16_RTOL,
                      "largest fragment sampled tokens")
    log(f"largest fragment: gathered rows bit-exact, sampled outputs {st}")
    ctx.release(b)
    ctx.sync()
    del ctx, dev, x, lg, y, out
    torch.cuda.empty_cache()


@pytest.mark.parametrize("wdt", ["bf16", "fp8"])
def test_grouped_enqueue_equals_per_expert_enqueues(wdt):
    """aep_enqueue_rows_grouped leaves the queues exactly as aep_enqueue_rows
    once per expert in ascending order: the same counts, the same gathered
    rows and the same FFN output bit for bit (empty experts included), and
    both against the oracle.  A grouped call one row past an expert's
    capacity returns AEP_ERR_CAPACITY and changes nothing."""
    depths = [300, 0, 17, 129, 64, 1, 0, 250]
    w = synth.Workload(f"grouped_{wdt}", 402, d=256, f=512, E=len(depths), k=1, zipf_s=1.0, mode="rows",
                       depth_max=max(depths), wdt=wdt)
    g = np.random.default_rng(7)
    N = int(sum(depths))
    x = synth.round_to_bf16_bits(g.standard_normal((N, w.d), dtype=np.float32))
    tok = g.permutation(N).astype(np.int32)
    gw = g.random(N, dtype=np.float32)
    ws = synth.all_expert_weights(w, 0, threads=4)
    xd, td, gd = to_dev(x, "bf16"), to_dev(tok, "i32"), to_dev(gw, "f32")
    log(f"case grouped {wdt}: depths {depths}")
    results = []
    for grouped in (False, True):
        ctx = make_context(w, max_tokens=N)
        dev_w = upload_weights(ctx, w, 0, ws)
        if grouped:
            # one row past expert 3's capacity: refused, nothing changes
            over = list(depths)
            over[3] = ctx.max_tokens + 1  # an expert's queue holds at most max_tokens rows
            before = (ctx.queue_depth(0), ctx.expert_counts(0).tolist())
            xo = torch.zeros((sum(over), w.d), dtype=torch.bfloat16, device="cuda")
            to_ = torch.zeros(sum(over), dtype=torch.int32, device="cuda")
            go = torch.zeros(sum(over), dtype=torch.float32, device="cuda")
            assert _status(ctx.enqueue_rows_grouped, 0, over, xo, to_, go, N) == L.AEP_ERR_CAPACITY
            assert (ctx.queue_depth(0), ctx.expert_counts(0).tolist()) == before
            ctx.enqueue_rows_grouped(0, depths, xd, td, gd, N)
        else:
            o = 0
            for e, n in enumerate(depths):
                ctx.enqueue_rows(0, e, xd[o:o + n], td[o:o + n], gd[o:o + n], N)
                o += n
        assert ctx.expert_counts(0).tolist() == depths
        b = ctx.rebatch(0)
        xp = to_host(b.x_perm())
        y = to_host(ctx.expert_ffn(b))
        ctx.release(b)
        ctx.sync()
        results.append((xp, y))
        del ctx, dev_w
    assert np.array_equal(results[0][0], results[1][0]), "gathered rows differ"
    assert np.array_equal(results[0][1], results[1][1]), "FFN outputs differ"
    lq = oracle.LayerQueues(w.E, 1)
    o = 0
    for e, n in enumerate(depths):
        if n:
            lq.enqueue_rows(e, x[o:o + n], tok[o:o + n], gw[o:o + n], N)
        o += n
    ref = oracle.moe_layer(lq, ws, "bf16", wdt)
    st = assert_close(oracle.bf16_to_f64(results[1][1]), ref["y"], BF16_RTOL, f"grouped {wdt} y")
    log(f"case grouped {wdt}: bit-identical to per-expert enqueues; y {st}")
