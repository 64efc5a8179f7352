"""Pins of the expert-runtime model oracle (oracle/sim.py).

* the generator against the published SplitMix64 sequence;
* two runs traced by hand from the model's rules (event order, step cost,
  attention hops, iteration hand-off, completion);
* conservation laws on random runs (every queued row runs once, token passes
  = requests x tokens x blocks, rows = passes x top_k, latency lower bound);
* routing: a CDF with one non-empty expert sends every row there.
"""

import json
import os

import numpy as np
import pytest

from oracle import scheduler as osched
from oracle import sim

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_splitmix64_reference_sequence():
    ref = json.load(open(os.path.join(GOLDEN, "splitmix64.json")))
    x, got = ref["seed"], []
    for _ in ref["outputs"]:
        x = (x + sim.GOLDEN) & sim.MASK
        got.append(sim.splitmix64_out(x))
    assert got == [int(h, 16) for h in ref["outputs"]]
    # draw(seed, stream 0, counter) is the counter-th output of that sequence
    assert sim.draw(0, 0, 2) == int(ref["outputs"][1], 16)


BASE = dict(n_blocks=2, n_experts=2, top_k=1, n_frag=1, attn_us=100, jitter_us=0, cost_fixed_us=5,
            cost_row_ns=1000, horizon_us=10**9, seed=1, delta=0.5, lookahead=1)


def test_hand_traced_two_requests():
    # expert 0 only (cdf [1, 1]); r0 at t=0, r1 at t=10, one token each.
    # t=0 run (0,0): 1 row, 5 + 1 us -> 6; r0 reaches block 1 at 106.
    # t=10 run (0,0) -> 16; r1 reaches block 1 at 116.
    # t=106 run (1,0) -> 112: r0 completes.  t=116 run (1,0) -> 122: r1 completes.
    for pol in ("mtfs", "flfs", "defrag"):
        r = sim.simulate(**BASE, granularity="expert", policy=pol, arrival_us=[0, 10], out_len=[1, 1],
                         expert_cdf=[1, 1])
        assert r["trace"]["t_start"] == [0, 10, 106, 116]
        assert r["trace"]["block"] == [0, 0, 1, 1]
        assert r["trace"]["expert"] == [0, 0, 0, 0]
        assert r["trace"]["rows"] == [1, 1, 1, 1]
        assert r["done_us"] == [112, 122]
        assert (r["steps"], r["rows"], r["busy_us"], r["end_us"], r["token_passes"], r["requests_done"]) == \
            (4, 4, 24, 122, 4, 2)


def test_hand_traced_batching_and_iterations():
    # three requests at t=0, two tokens each for r0, one for r1 and r2; one
    # expert; whole-block steps.  t=0: block 0 holds 3 rows -> 5 + 3 = 8 us;
    # all leave, arrive at block 1 at 108 (one rank, no jitter).  t=108: block
    # 1, 3 rows -> 116; r1, r2 complete; r0's second token reaches block 0 at
    # 216 -> 222, block 1 at 322 -> 328, complete.
    r = sim.simulate(**BASE, granularity="block", policy="mtfs", arrival_us=[0, 0, 0], out_len=[2, 1, 1],
                     expert_cdf=[1, 1])
    assert r["trace"]["t_start"] == [0, 108, 216, 322]
    assert r["trace"]["rows"] == [3, 3, 1, 1]
    assert r["trace"]["expert"] == [-1, -1, -1, -1]
    assert r["done_us"] == [328, 116, 116]
    assert r["token_passes"] == 8 and r["requests_done"] == 3


def test_horizon_stops_new_steps():
    r = sim.simulate(**{**BASE, "horizon_us": 50}, granularity="expert", policy="mtfs", arrival_us=[0, 10],
                     out_len=[1, 1], expert_cdf=[1, 1])
    # both block-0 steps start before 50; at 106 r0 reaches block 1, but no
    # step may start any more: the run stops there with that row queued
    assert r["trace"]["t_start"] == [0, 10]
    assert (r["requests_done"], r["end_us"], r["rows_queued_at_end"]) == (0, 106, 1)


def test_single_expert_cdf_routes_every_row_there():
    r = sim.simulate(**{**BASE, "n_experts": 4}, granularity="expert", policy="mtfs",
                     arrival_us=[0, 3, 7, 9], out_len=[3, 1, 2, 2], expert_cdf=[0, 0, 5, 5])
    assert set(r["trace"]["expert"]) == {2}


@pytest.mark.parametrize("seed", [3, 4, 5])
@pytest.mark.parametrize("granularity", ["expert", "block"])
@pytest.mark.parametrize("policy", ["mtfs", "flfs", "defrag"])
def test_conservation_laws(seed, granularity, policy):
    rng = np.random.default_rng(seed)
    n = 30
    arr = np.cumsum(rng.integers(0, 300, n)).tolist()
    ol = rng.integers(1, 5, n).tolist()
    NB, NE, K = 3, 4, 2
    r = sim.simulate(n_blocks=NB, n_experts=NE, top_k=K, n_frag=3, granularity=granularity, policy=policy,
                     arrival_us=arr, out_len=ol, expert_cdf=[5, 9, 12, 13], attn_us=150, jitter_us=80,
                     cost_fixed_us=20, cost_row_ns=700, horizon_us=10**9, seed=seed, delta=0.5, lookahead=2)
    assert r["requests_done"] == n and r["rows_queued_at_end"] == 0
    assert r["token_passes"] == NB * sum(ol)
    assert r["rows"] == K * r["token_passes"] == sum(r["trace"]["rows"])
    assert r["busy_us"] <= r["end_us"]
    for i in range(n):
        assert r["done_us"][i] - arr[i] >= (ol[i] * NB - 1) * 150
    t = r["trace"]["t_start"]
    assert all(b >= a for a, b in zip(t, t[1:]))


TRACES = json.load(open(os.path.join(GOLDEN, "sim_hand_traces.json")))


def _run_traced(spec, base=TRACES["base"]):
    kw = {k: v for k, v in base.items()}
    return sim.simulate(**kw, granularity=spec["granularity"], policy=spec["policy"], delta=spec["delta"],
                        lookahead=spec["lookahead"], arrival_us=spec["arrival_us"], out_len=spec["out_len"])


@pytest.mark.parametrize("spec", TRACES["runs"], ids=[r["name"] for r in TRACES["runs"]])
def test_hand_traced_policy_runs(spec):
    """Block and expert granularity, three blocks, two experts: every step of
    the hand trace (time, block, expert, rows, queue state), completion times,
    and the scores at the decisions where the policies part ways."""
    r = _run_traced(spec)
    tr = r["trace"]
    assert tr["t_start"] == spec["t_start"]
    assert tr["block"] == spec["block"]
    assert tr["rows"] == spec["rows"]
    if "expert" in spec:
        assert tr["expert"] == spec["expert"]
    else:
        assert set(tr["expert"]) == {-1}
    if "block_rows_after" in spec:
        assert tr["block_rows_after"] == spec["block_rows_after"]
    assert r["done_us"] == spec["done_us"]
    for dcs in spec["decisions"]:
        i = spec["t_start"].index(dcs["t"])
        if "R" in dcs:
            assert spec["block"][i] == dcs["pick"]
            if "scores" in dcs:
                np.testing.assert_allclose(osched.layer_scores(dcs["R"], spec["delta"], spec["lookahead"]),
                                           dcs["scores"], rtol=0, atol=1e-12)
        else:
            assert [spec["block"][i], spec["expert"][i]] == dcs["pick"]
            if "scores" in dcs:
                np.testing.assert_allclose(osched.defrag_scores(np.array(dcs["Q"]), spec["delta"], spec["lookahead"]),
                                           dcs["scores"], rtol=0, atol=1e-12)
