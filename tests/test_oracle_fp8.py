"""Pins of the e4m3fn decode (oracle) and encode (input generator)."""

import json
import os

import numpy as np
import torch

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
ALL = np.arange(256, dtype=np.uint8)


def test_decode_matches_torch_float8_e4m3fn():
    ref = torch.from_numpy(ALL.copy()).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = oracle.e4m3_to_f64(ALL)
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    m = ~np.isnan(ref)
    assert np.array_equal(got[m], ref[m])
    assert np.array_equal(np.signbit(got[m]), np.signbit(ref[m]))


def test_decode_spec_anchors():
    fx = json.load(open(os.path.join(GOLDEN, "e4m3_anchors.json")))
    for a in fx["anchors"]:
        v = oracle.e4m3_to_f64(np.array([a["code"]], np.uint8))[0]
        if a["value"] == "nan":
            assert np.isnan(v)
        else:
            assert v == a["value"] and np.signbit(v) == np.signbit(a["value"])
    pos = oracle.e4m3_to_f64(ALL[:127])
    assert np.all(np.diff(pos) > 0)  # codes 0..126 strictly increasing


def _brute_nearest(v):
    """Nearest finite code by exhaustive search; ties -> even code; saturate."""
    vals = oracle.e4m3_to_f64(ALL)
    out = np.empty(v.shape, np.uint8)
    for i, x in enumerate(v.astype(np.float64)):
        best = None
        for c in range(256):
            if np.isnan(vals[c]) or (c == 0x80):
                continue
            dist = abs(vals[c] - x)
            if best is None or dist < best[0] or (dist == best[0] and c % 2 == 0 and best[1] % 2 == 1):
                best = (dist, c)
        c = best[1]
        if vals[c] == 0.0 and np.signbit(x):
            c = 0x80
        out[i] = c
    return out


def test_encoder_is_nearest_even_saturating():
    r = np.random.default_rng(0)
    vals = oracle.e4m3_to_f64(ALL[:127])
    mids = ((vals[:-1] + vals[1:]) / 2).astype(np.float32)       # exact ties
    v = np.concatenate([
        r.standard_normal(400).astype(np.float32) * np.float32(30),
        r.standard_normal(200).astype(np.float32) * np.float32(0.01),
        mids, -mids, vals.astype(np.float32),
        np.array([448, 460, 464, 500, 1e6, -449, -1e9, 2.0 ** -10, 2.0 ** -11, -2.0 ** -10, 0.0], np.float32),
    ]).astype(np.float32)
    got = synth.encode_e4m3(v)
    ref = _brute_nearest(v)
    bad = np.nonzero(got != ref)[0]
    assert bad.size == 0, (v[bad[:5]], got[bad[:5]], ref[bad[:5]])


def test_encoder_matches_torch_in_range():
    r = np.random.default_rng(1)
    v = (r.standard_normal(20000) * 40).astype(np.float32)
    v = v[np.abs(v) < 440]
    ref = torch.from_numpy(v).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(synth.encode_e4m3(v), ref)


def test_row_quantiser_scale_rule():
    r = np.random.default_rng(2)
    w = synth.round_to_bf16_bits((r.standard_normal((16, 64)) * 0.02).astype(np.float32))
    w[3] = 0
    q, s_bits = synth.quantize_rows_e4m3(w)
    s = oracle.bf16_to_f64(s_bits)
    wf = synth.bf16_bits_to_f32(w).astype(np.float64)
    assert s[3] == 1.0 and np.all(q[3] & 0x7F == 0)
    amax = np.abs(wf).max(axis=1)
    nz = amax > 0
    np.testing.assert_allclose(s[nz], amax[nz] / 448.0, rtol=2 ** -8)
    deq = oracle.e4m3_to_f64(q) * s[:, None]
    assert np.all(np.abs(deq) <= 448.0 * s[:, None])
    rel = np.abs(deq - wf) / np.maximum(np.abs(wf), 1e-30)
    assert np.all((rel <= 2.0 ** -4 + 1e-12) | (np.abs(wf) < 2.0 ** -6 * s[:, None]))
