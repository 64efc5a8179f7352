"""The two failure modes of Sec. 3.4 reproduced on the expert-runtime model
(libaep's aep_sim_run, host only), on the seeded request streams of
synth.arrivals:

* most-tokens-first-serve fragments batches: with (block, expert) queues and a
  long-request stream near capacity, its steps drain a few rows each while
  rows sit in most blocks at once, and hardly any request finishes;
  first-layer-first-serve keeps the tokens in a few blocks and big batches;
* first-layer-first-serve live-locks: with many short requests arriving
  faster than it drains them, new arrivals keep block 0 busy and no request
  ever completes, while MTFS and the defragging scheduler finish every
  (or nearly every) request of the first half of the run.
"""

import dataclasses

import numpy as np

import synth
from paper_2505_08944_amd import sched


def _run(name, policy, granularity, horizon_us, delta=0.5, lookahead=2):
    sc = dataclasses.replace(synth.scenario(name), horizon_us=horizon_us)
    st = synth.request_stream(sc)
    r = sched.sim_run(n_blocks=sc.n_blocks, n_experts=sc.n_experts, top_k=sc.top_k, n_frag=sc.n_frag,
                      granularity=granularity, policy=policy, arrival_us=st["arrival_us"], out_len=st["out_len"],
                      expert_cdf=st["expert_cdf"], attn_us=sc.attn_us, jitter_us=sc.jitter_us,
                      cost_fixed_us=sc.cost_fixed_us, cost_row_ns=sc.cost_row_ns, horizon_us=sc.horizon_us,
                      seed=sc.cfg_id, delta=delta, lookahead=lookahead, trace_capacity=10**6)
    done = r["done_us"] >= 0
    first = st["arrival_us"] < horizon_us // 2
    return {"rows_per_step": r["rows"] / r["steps"], "blocks": float(r["trace"]["blocks_busy_after"].mean()),
            "done_first_half": float(done[first].mean()), "tokens_done": int(st["out_len"][done].sum())}


def test_mtfs_fragments_expert_queues():
    m = _run("frag", "mtfs", "expert", 10_000_000)
    f = _run("frag", "flfs", "expert", 10_000_000)
    assert m["rows_per_step"] < 0.5 * f["rows_per_step"]
    assert m["blocks"] > 5 * f["blocks"]
    assert m["tokens_done"] < 0.2 * f["tokens_done"]


def test_flfs_livelocks_on_short_requests():
    for gran in ("block", "expert"):
        f = _run("livelock", "flfs", gran, 4_000_000)
        m = _run("livelock", "mtfs", gran, 4_000_000)
        d = _run("livelock", "defrag", gran, 4_000_000, 0.9, 4)
        assert f["done_first_half"] < 0.02 and f["tokens_done"] < 0.02 * m["tokens_done"]
        assert m["done_first_half"] > 0.9 and d["done_first_half"] > 0.9
