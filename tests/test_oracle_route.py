"""Pins of the oracle's router (softmax top-k gate) against independent facts."""

import json
import math
import os

import numpy as np
import pytest
import scipy.special

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _logits(T, E, seed, grid=None):
    r = np.random.default_rng(seed)
    l = r.standard_normal((T, E)).astype(np.float32)
    if grid:
        l = (np.round(l / grid) * grid).astype(np.float32)  # many exact ties
    return l


@pytest.mark.parametrize("T,E,k,grid", [(300, 16, 4, 0.25), (200, 8, 2, None), (64, 64, 6, 0.5), (50, 5, 5, 1.0)])
def test_selection_defining_property(T, E, k, grid):
    """Each selected expert beats every later slot and every unselected expert
    under (logit desc, id asc); slots hold distinct ids in [0, E)."""
    l = _logits(T, E, 1 + T + E, grid)
    idx, _ = oracle.route(l, k)
    assert idx.shape == (T, k) and idx.dtype == np.int32

    def before(a, b, t):
        return l[t, a] > l[t, b] or (l[t, a] == l[t, b] and a < b)

    for t in range(T):
        sel = [int(e) for e in idx[t]]
        assert len(set(sel)) == k and all(0 <= e < E for e in sel)
        for j in range(k - 1):
            assert before(sel[j], sel[j + 1], t)
        for e in range(E):
            if e not in sel:
                assert before(sel[-1], e, t)


def test_full_k_renorm_equals_softmax():
    l = _logits(128, 12, 7)
    idx, w = oracle.route(l, 12, renorm=True)
    back = np.zeros_like(w)
    np.put_along_axis(back, idx, w, axis=1)
    ref = scipy.special.softmax(l.astype(np.float64), axis=1)
    np.testing.assert_allclose(back, ref, rtol=1e-6, atol=0)


def test_non_renorm_is_softmax_probability():
    l = _logits(128, 8, 9)
    idx, w = oracle.route(l, 2, renorm=False)
    ref = np.take_along_axis(scipy.special.softmax(l.astype(np.float64), axis=1), idx, axis=1)
    np.testing.assert_allclose(w, ref, rtol=1e-6, atol=0)


def test_top1_renorm_is_exactly_one_and_sums():
    l = _logits(256, 8, 11)
    _, w1 = oracle.route(l, 1)
    assert np.all(w1 == np.float32(1.0))
    _, w3 = oracle.route(l, 3)
    np.testing.assert_allclose(w3.astype(np.float64).sum(axis=1), 1.0, rtol=0, atol=1e-6)
    assert np.all(np.diff(w3, axis=1) <= 0)  # descending logits -> descending weights


def test_all_equal_logits_pick_lowest_ids():
    l = np.full((5, 9), 0.125, dtype=np.float32)
    idx, w = oracle.route(l, 4)
    assert (idx == np.arange(4)).all()
    np.testing.assert_allclose(w, 0.25, rtol=1e-7)


def test_rejects_non_finite():
    l = _logits(4, 4, 3)
    l[2, 1] = np.nan
    with pytest.raises(AssertionError):
        oracle.route(l, 2)
    l[2, 1] = np.inf
    with pytest.raises(AssertionError):
        oracle.route(l, 2)


def test_hand_worked_router():
    fx = json.load(open(os.path.join(GOLDEN, "tiny_layer.json")))
    l = np.array(fx["logits"], dtype=np.float32)
    idx, w = oracle.route(l, fx["k"], fx["renorm"])
    assert idx.tolist() == fx["idx"]
    e = math.e
    np.testing.assert_allclose(w, [[3 / 5, 2 / 5], [0.5, 0.5], [e / (e + 1), 1 / (e + 1)]], rtol=1e-6)
    np.testing.assert_allclose(w, fx["w"], rtol=1e-6)
