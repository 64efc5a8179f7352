"""A whole drain step (route + append of a fragment, re-batch, gate/up, down,
combine, release) captured in a HIP graph replays bit-identically: none of
these calls synchronises or records a memset node, and the host-side queue
state returns to where it started after one step.  Replays alternate with
eager steps and host synchronisations, and every replay is checked against
the eager result and against the oracle's layer (per-element tolerance)."""

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_helpers import BF16_RTOL, assert_close, log, make_context, to_dev, to_host, upload_weights

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["mid", "mid_shared", "mid_fp8"])
def test_layer_step_graph_replays_match_eager(name):
    import test_gpu_parity_small as small
    w = small.SMALL[name]
    frags = synth.layer_fragments(w, 0)
    ws = synth.all_expert_weights(w, 0, threads=4)
    ctx = make_context(w)
    dev = upload_weights(ctx, w, 0, ws)
    xs = [(to_dev(f["x"], w.act), to_dev(f["logits"], "f32")) for f in frags]
    T = sum(x.shape[0] for x, _ in xs)
    act = torch.bfloat16
    y = torch.empty((T * w.k + w.S * T, w.d), dtype=act, device="cuda")
    out = torch.empty((T, w.d), dtype=act, device="cuda")

    def step():
        for x, lg in xs:
            ctx.route_enqueue(0, x, lg)
        b = ctx.rebatch(0)
        ctx.expert_gate_up(b)
        ctx.expert_down(b, y)
        ctx.combine(b, y, out)
        ctx.release(b)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    ref = out.clone()
    lq = oracle.LayerQueues(w.E, w.k, w.S, w.renorm)
    for f in frags:
        lq.enqueue_routed(f["x"], f["logits"])
    want = oracle.moe_layer(lq, ws, w.act, w.wdt)["out"]
    assert_close(oracle.act_to_f64(to_host(ref), w.act), want, BF16_RTOL, f"{name} eager step")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for i in range(4):
        out.fill_(0)
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), f"replay {i}"
        assert_close(oracle.act_to_f64(to_host(out), w.act), want, BF16_RTOL, f"{name} replay {i}")
        out.fill_(0)
        step()                      # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(out, ref), f"eager step after replay {i}"
    ctx.sync()
    log(f"case {name}: 4 graph replays and 4 eager steps bit-identical, and within tolerance of the oracle")
    del graph, ctx, dev
