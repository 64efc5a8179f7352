"""Clock probe of the FFN launches (aep_set_clock_probe): while on, every
bf16-path launch writes each workgroup's elapsed shader-clock cycles and
100 MHz ticks; off again, launches leave the buffer alone; the outputs are
the same with the probe on and off."""

import numpy as np
import pytest
import torch

from paper_2505_08944_amd import Context

pytestmark = pytest.mark.gpu


def _batch(d=256, f=512, E=4, n=(300, 64, 0, 17)):
    dev = torch.device("cuda", 0)
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    ctx = Context(1, E, d, f, 1, max_tokens_per_layer=sum(n))
    W = []
    for e in range(E):
        m = [(torch.randn(s, generator=g, device=dev) * 0.02).to(torch.bfloat16) for s in [(f, d), (f, d), (d, f)]]
        ctx.set_expert_weights(0, e, *m)
        W.append(m)
    x = torch.randn((sum(n), d), generator=g, device=dev).to(torch.bfloat16)
    tok = torch.arange(sum(n), dtype=torch.int32, device=dev)
    gw = torch.ones(sum(n), dtype=torch.float32, device=dev)
    o = 0
    for e, c in enumerate(n):
        if c:
            ctx.enqueue_rows(0, e, x[o:o + c], tok[o:o + c], gw[o:o + c], sum(n))
        o += c
    return ctx, W, x, ctx.rebatch(0)


def test_clock_probe_records_and_turns_off():
    ctx, W, x, b = _batch()
    ncu = torch.cuda.get_device_properties(0).multi_processor_count
    y0 = torch.empty((b.n_rows, 256), dtype=torch.bfloat16, device="cuda")
    ctx.expert_ffn(b, y0)
    clk = torch.zeros((ncu, 2), dtype=torch.int64, device="cuda")
    ctx.set_clock_probe(clk)
    y1 = torch.empty_like(y0)
    ctx.expert_ffn(b, y1)
    ctx.set_clock_probe(None)
    torch.cuda.synchronize()
    c = clk.cpu().numpy()
    ran = c[:, 0] > 0
    assert ran.sum() >= 8, "every workgroup of the launch records its cycles"
    assert np.all(c[ran, 1] > 0)
    ghz = c[ran, 0].sum() / (c[ran, 1].sum() / 100e6) / 1e9
    assert 0.3 < ghz < 3.5, ghz
    assert torch.equal(y0, y1), "the probe does not change the outputs"
    clk.zero_()
    ctx.expert_ffn(b, y1)
    torch.cuda.synchronize()
    assert int(clk.abs().sum()) == 0, "off: launches leave the buffer alone"
    ctx.release(b)
    ctx.sync()


def test_clock_probe_rejects_bad_buffers():
    ctx, W, x, b = _batch()
    for bad in (torch.zeros((4, 2), dtype=torch.int32, device="cuda"),
                torch.zeros((4, 3), dtype=torch.int64, device="cuda"),
                torch.zeros((4, 2), dtype=torch.int64)):
        with pytest.raises(ValueError):
            ctx.set_clock_probe(bad)
    ctx.release(b)
