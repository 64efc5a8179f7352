"""The scheduler pins catch plausible mistakes in the oracle.

Each test plants one mistake in oracle/scheduler.py (on the CPU, by patching
the module for the duration of the test) and checks that at least one pin --
the hand-worked score tables of Algorithm 1 (queue and layer granularity) or
the hand-traced runtime-model runs -- no longer holds.  A mistake no pin sees
would leave that rule of the oracle unchecked.
"""

import json
import os

import numpy as np
import pytest

from oracle import scheduler as osched
from oracle import sim

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TABLES = json.load(open(os.path.join(GOLDEN, "defrag_alg1.json")))
TRACES = json.load(open(os.path.join(GOLDEN, "sim_hand_traces.json")))


def _tables_hold() -> bool:
    for c in TABLES["cases"]:
        Q = np.array(c["Q"])
        if not np.allclose(osched.defrag_scores(Q, c["delta"], c["L"]), c["scores"], rtol=0, atol=1e-12):
            return False
        p = osched.pick_defrag(Q, c["delta"], c["L"])
        if (None if p is None else list(p)) != c["pick"]:
            return False
        rows = Q.sum(axis=1).tolist()
        if "mtfs" in c and osched.pick_mtfs(rows) != c["mtfs"]:
            return False
        if "flfs" in c and osched.pick_flfs(rows) != c["flfs"]:
            return False
    for c in TABLES["layer_cases"]:
        if not np.allclose(osched.layer_scores(c["R"], c["delta"], c["L"]), c["scores"], rtol=0, atol=1e-12):
            return False
        if osched.pick_layer_defrag(c["R"], c["delta"], c["L"]) != c["pick"]:
            return False
        if osched.pick_mtfs(c["R"]) != c["mtfs"] or osched.pick_flfs(c["R"]) != c["flfs"]:
            return False
    return True


def _traces_hold() -> bool:
    for spec in TRACES["runs"]:
        r = sim.simulate(**TRACES["base"], granularity=spec["granularity"], policy=spec["policy"],
                         delta=spec["delta"], lookahead=spec["lookahead"], arrival_us=spec["arrival_us"],
                         out_len=spec["out_len"])
        tr = r["trace"]
        if tr["t_start"] != spec["t_start"] or tr["block"] != spec["block"] or tr["rows"] != spec["rows"]:
            return False
        if "expert" in spec and tr["expert"] != spec["expert"]:
            return False
        if r["done_us"] != spec["done_us"]:
            return False
    return True


def test_pins_hold_on_the_oracle_as_written():
    assert _tables_hold() and _traces_hold()


def _patch(monkeypatch, name, fn):
    monkeypatch.setattr(osched, name, fn)
    if hasattr(sim, name):
        monkeypatch.setattr(sim, name, fn)


PLANTED = {
    # every lookahead block weighted delta (the decay exponent dropped)
    "no decay": ("_decay_weights", lambda delta, L: np.full(int(L), float(delta))),
    # weights delta^0 .. delta^(L-1) (the exponent off by one)
    "decay off by one": ("_decay_weights", lambda delta, L: np.cumprod(np.r_[1.0, np.full(max(int(L) - 1, 0),
                                                                                          float(delta))])[:int(L)]),
    # ties to the highest index instead of the lowest
    "last maximum on ties": ("_first_max", lambda s: int(len(np.asarray(s)) - 1 - np.argmax(np.asarray(s)[::-1]))),
    # FLFS runs the block's first non-empty queue instead of its largest
    "FLFS first queue": ("_largest_queue", lambda row: int(np.flatnonzero(np.asarray(row) > 0)[0])),
    # FLFS picks the most loaded block instead of the lowest non-empty one
    "FLFS largest block": ("pick_flfs", lambda rows: osched.pick_mtfs(rows)),
    # lookahead over the blocks before b instead of after it
    "lookahead backwards": ("lookahead_terms", lambda load, delta, L: sum(
        (np.roll(np.asarray(load, float), i) * delta ** i for i in range(1, int(L) + 1)),
        np.zeros(len(load)))),
    # lookahead stops at the last block (no wrap round to block 0)
    "no wrap": ("lookahead_terms", lambda load, delta, L: np.array(
        [sum(load[b + i] * delta ** i for i in range(1, int(L) + 1) if b + i < len(load))
         for b in range(len(load))], dtype=float)),
    # the lookahead term sums the next blocks' queues instead of averaging them
    "no average": ("defrag_scores", lambda Q, delta, L: np.where(
        np.asarray(Q) > 0, np.asarray(Q, float) + osched.lookahead_terms(np.asarray(Q, float).sum(axis=1), delta, L)[:, None],
        0.0)),
}


@pytest.mark.parametrize("mistake", list(PLANTED))
def test_planted_mistake_fails_a_pin(monkeypatch, mistake):
    name, fn = PLANTED[mistake]
    _patch(monkeypatch, name, fn)
    assert not (_tables_hold() and _traces_hold()), f"no pin catches: {mistake}"
