"""Pins of the oracle's mu-queues, re-batch and gather.

Library routines (histogram, cumulative sum, stable sort) and invariants
(bijection, fragment invariance, bit copies) fix what a correct drain must
produce.
"""

import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _frag_inputs(T, E, d, seed):
    r = np.random.default_rng(seed)
    x = r.standard_normal((T, d)).astype(np.float32)
    l = r.standard_normal((T, E)).astype(np.float32)
    l[:, 1] += 1.5  # skew
    return x, l


def _fill(lq, x, l, sizes):
    t0 = 0
    for n in sizes:
        lq.enqueue_routed(x[t0:t0 + n], l[t0:t0 + n])
        t0 += n


@pytest.mark.parametrize("T,E,k,sizes", [(97, 8, 2, [97]), (200, 16, 4, [13, 100, 0, 87]), (64, 6, 6, [1] * 64)])
def test_drain_matches_counting_sort(T, E, k, sizes):
    x, l = _frag_inputs(T, E, 8, T * 7 + E)
    lq = oracle.LayerQueues(E, k)
    _fill(lq, x, l, [s for s in sizes if s])
    assert lq.rows == T * k
    idx, w = oracle.route(l, k)
    b = oracle.rebatch(lq)
    flat = idx.ravel()
    # counts: histogram; offsets: exclusive scan
    np.testing.assert_array_equal(b.counts, np.bincount(flat, minlength=E))
    assert int(b.counts.sum()) == T * k
    np.testing.assert_array_equal(b.offsets, np.concatenate([[0], np.cumsum(np.bincount(flat, minlength=E))]))
    # row order: stable sort of the flattened (token, slot) sequence by expert id
    perm = np.argsort(flat, kind="stable")
    np.testing.assert_array_equal(b.row_token, perm // k)
    np.testing.assert_array_equal(b.row_slot, perm % k)
    np.testing.assert_array_equal(b.row_w, w.ravel()[perm])
    # pos is a bijection (token, slot) -> [0, T*k) and inverts the row order
    assert sorted(b.pos.ravel().tolist()) == list(range(T * k))
    np.testing.assert_array_equal(b.pos.ravel()[perm], np.arange(T * k))
    np.testing.assert_array_equal(b.posw, w)
    # drained
    assert lq.rows == 0 and lq.n_tokens == 0


def test_fragmenting_does_not_change_the_batch():
    T, E, k = 150, 8, 2
    x, l = _frag_inputs(T, E, 4, 5)
    ref = None
    for sizes in ([150], [50, 50, 50], [1, 148, 1], [7] * 21 + [3]):
        lq = oracle.LayerQueues(E, k)
        _fill(lq, x, l, sizes)
        b = oracle.rebatch(lq)
        xp = oracle.gather(b)
        cur = (b.counts.tolist(), b.offsets.tolist(), b.row_token.tolist(), b.row_slot.tolist(),
               b.row_w.tolist(), xp.tobytes())
        if ref is None:
            ref = cur
        assert cur == ref


def test_gather_is_a_bit_copy_of_token_rows():
    T, E, k, d = 120, 8, 3, 16
    x, l = _frag_inputs(T, E, d, 17)
    bits = x.view(np.uint32)  # arbitrary payloads
    lq = oracle.LayerQueues(E, k, S=2)
    _fill(lq, bits, l, [30, 90])
    b = oracle.rebatch(lq)
    xp = oracle.gather(b)
    assert xp.shape == (T * k + T, d) and xp.dtype == np.uint32
    np.testing.assert_array_equal(xp[:T * k], bits[b.row_token])
    np.testing.assert_array_equal(xp[T * k:], bits)  # shared experts see every token in id order
    assert b.counts[-2:].tolist() == [T, T]
    assert b.offsets[-1] == T * k + 2 * T and b.n_rows_total == T * k + 2 * T


def test_explicit_rows_append_verbatim_and_mix():
    E, k, d = 4, 2, 3
    lq = oracle.LayerQueues(E, k)
    xa = np.arange(5 * d, dtype=np.float32).reshape(5, d)
    xb = -np.arange(2 * d, dtype=np.float32).reshape(2, d)
    lq.enqueue_rows(2, xa, np.array([4, 0, 3, 1, 2], np.int32), np.linspace(0, 1, 5, dtype=np.float32), n_tokens=5)
    lq.enqueue_rows(0, xb, np.array([1, 4], np.int32), np.array([0.5, 0.25], np.float32), n_tokens=5,
                    slots=np.array([1, 1], np.int32))
    lq.enqueue_rows(2, xb[:1], np.array([0], np.int32), np.array([2.0], np.float32), n_tokens=5,
                    slots=np.array([1], np.int32))
    b = oracle.rebatch(lq)
    assert b.counts.tolist() == [2, 0, 6, 0]
    assert b.row_token.tolist() == [1, 4, 4, 0, 3, 1, 2, 0]
    assert b.row_slot.tolist() == [1, 1, 0, 0, 0, 0, 0, 1]
    xp = oracle.gather(b)
    np.testing.assert_array_equal(xp, np.concatenate([xb, xa, xb[:1]]))
    assert b.pos.tolist() == [[3, 7], [5, 0], [6, -1], [4, -1], [2, 1]]


def test_slot_collision_is_rejected():
    lq = oracle.LayerQueues(2, 1)
    x = np.zeros((1, 2), np.float32)
    lq.enqueue_rows(0, x, np.array([0], np.int32), np.array([1.0], np.float32), n_tokens=1)
    lq.enqueue_rows(1, x, np.array([0], np.int32), np.array([1.0], np.float32), n_tokens=1)
    with pytest.raises(AssertionError):
        oracle.rebatch(lq)


def test_hand_worked_queue_contents():
    fx = json.load(open(os.path.join(GOLDEN, "tiny_layer.json")))
    lq = oracle.LayerQueues(3, 2)
    lq.enqueue_routed(np.array(fx["x"], np.float32)[:, None], np.array(fx["logits"], np.float32))
    b = oracle.rebatch(lq)
    assert b.counts.tolist() == fx["counts"]
    assert b.offsets.tolist() == fx["offsets"]
    assert b.row_token.tolist() == fx["row_token"]
    assert b.row_slot.tolist() == fx["row_slot"]
    assert b.pos.tolist() == fx["pos"]
