"""Checks of the seeded input generator (formats, skew, determinism)."""

import numpy as np
import torch

import synth


def test_bf16_rounding_matches_torch():
    r = np.random.default_rng(0)
    a = np.concatenate([r.standard_normal(100000).astype(np.float32) * np.float32(3),
                        np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 0.0, -0.0], np.float32)])
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(synth.round_to_bf16_bits(a), ref)
    np.testing.assert_array_equal(synth.bf16_bits_to_f32(ref), torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).float().numpy())


def test_zipf_bias_is_zipf_pmf():
    w = synth.workload("c3")
    b = synth.zipf_bias(w, 0).astype(np.float64)
    p = np.sort(np.exp(b) / np.exp(b).sum())[::-1]
    r = np.arange(1, w.E + 1, dtype=np.float64)
    z = r ** -w.zipf_s
    np.testing.assert_allclose(p, z / z.sum(), rtol=1e-6)


def test_determinism_and_fragments():
    w = synth.workload("c1f4")
    a = synth.layer_fragments(w, 0)
    b = synth.layer_fragments(w, 0)
    assert len(a) == 4 and [f["x"].shape[0] for f in a] == [64] * 4
    for fa, fb in zip(a, b):
        assert fa["x"].tobytes() == fb["x"].tobytes() and fa["logits"].tobytes() == fb["logits"].tobytes()
    one = synth.layer_fragments(synth.workload("c1"), 0)[0]
    assert np.array_equal(np.concatenate([f["x"] for f in a]), one["x"])
    assert synth.fragment_sizes(10, 4) == [3, 3, 2, 2] and synth.fragment_sizes(0, 3) == [0, 0, 0]


def test_rows_workload_depths():
    w = synth.workload("c4")
    rw = synth.rows_workload(w)
    assert sorted(rw["depths"].tolist(), reverse=True) == [4096, 1663, 981, 675, 505, 398, 326, 274, 235, 205,
                                                            181, 161, 145, 132, 121, 111]
    assert rw["n_tokens"] == 10209
    toks = np.concatenate([e["token_ids"] for e in rw["experts"]])
    assert sorted(toks.tolist()) == list(range(10209))


def test_c5_layer_sizes():
    w = synth.workload("c5")
    assert sorted(w.tokens) == [0, 1024, 2048, 3072, 5120, 6144, 7168, 8192] and sum(w.tokens) == 32768
    assert synth.weight_source(w, 3, 6) == (2, 0, 1)
