"""Pins of the layer-pick policies against hand-worked queue tables."""

import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
CASES = json.load(open(os.path.join(GOLDEN, "defrag_alg1.json")))["cases"]


@pytest.mark.parametrize("case", CASES, ids=[str(i) for i in range(len(CASES))])
def test_defrag_hand_worked(case):
    Q = np.array(case["Q"])
    s = oracle.defrag_scores(Q, case["delta"], case["L"])
    np.testing.assert_allclose(s, case["scores"], rtol=0, atol=1e-12)
    pick = oracle.pick_defrag(Q, case["delta"], case["L"])
    assert (None if pick is None else list(pick)) == case["pick"]
    rows = Q.sum(axis=1).tolist()
    if "mtfs" in case:
        assert oracle.pick_mtfs(rows) == case["mtfs"]
    if "flfs" in case:
        assert oracle.pick_flfs(rows) == case["flfs"]


def test_delta_zero_is_mtfs_over_queues():
    r = np.random.default_rng(3)
    for _ in range(50):
        Q = r.integers(0, 5, size=(6, 4))
        pick = oracle.pick_defrag(Q, 0.0, 3)
        if Q.max() == 0:
            assert pick is None
            continue
        flat = int(np.argmax(Q))  # first maximum in row-major order
        assert pick == divmod(flat, Q.shape[1])


def test_mtfs_and_flfs_ties_and_empty():
    assert oracle.pick_mtfs([0, 3, 3, 1]) == 1
    assert oracle.pick_mtfs([0, 0]) is None
    assert oracle.pick_flfs([0, 0, 2, 9]) == 2
    assert oracle.pick_flfs([]) is None


LAYER_CASES = json.load(open(os.path.join(GOLDEN, "defrag_alg1.json")))["layer_cases"]


@pytest.mark.parametrize("case", LAYER_CASES, ids=[str(i) for i in range(len(LAYER_CASES))])
def test_layer_defrag_hand_worked(case):
    R = case["R"]
    np.testing.assert_allclose(oracle.layer_scores(R, case["delta"], case["L"]), case["scores"], rtol=0, atol=1e-12)
    assert oracle.pick_layer_defrag(R, case["delta"], case["L"]) == case["pick"]
    assert oracle.pick_mtfs(R) == case["mtfs"]
    assert oracle.pick_flfs(R) == case["flfs"]


def test_queue_policies_hand_worked():
    # FLFS takes the lowest block holding rows and its largest queue (ties:
    # lowest expert); MTFS the largest queue anywhere (ties: row-major first)
    Q = np.array([[0, 0, 0], [1, 4, 4], [9, 0, 0]])
    assert oracle.pick_queue_flfs(Q) == (1, 1)
    assert oracle.pick_queue_mtfs(Q) == (2, 0)
    assert oracle.pick_queue_mtfs([[3, 5], [5, 1]]) == (0, 1)
    assert oracle.pick_queue_flfs(np.zeros((2, 2), int)) is None
    assert oracle.pick_queue_mtfs(np.zeros((2, 2), int)) is None


def test_layer_form_is_algorithm1_on_block_averages():
    """With every queue of a block equal to the block's average, Algorithm 1's
    best queue score times N_E is the layer-granularity score."""
    r = np.random.default_rng(5)
    for _ in range(40):
        NB, NE = int(r.integers(1, 7)), int(r.choice([1, 2, 4, 8]))
        R = r.integers(0, 6, NB) * NE
        Q = np.repeat((R // NE)[:, None], NE, axis=1)
        delta, L = float(r.choice([0.0, 0.25, 0.5, 1.0])), int(r.integers(0, 4))
        s = oracle.defrag_scores(Q, delta, L)
        np.testing.assert_allclose(s.max(axis=1) * NE, oracle.layer_scores(R, delta, L), rtol=0, atol=1e-9)
        p = oracle.pick_defrag(Q, delta, L)
        assert (None if p is None else p[0]) == oracle.pick_layer_defrag(R, delta, L)
