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
