#!/usr/bin/env python3
"""Benchmark of the AEP expert-layer hot path on one MI355X.

One step = one pass of the whole path over one batch of synthetic input:
four arriving fragments are routed and appended to the layer's mu-queues,
the layer is drained (re-batch + gather), the grouped SwiGLU experts run
(gate/up launch, down launch) and the top-k combine writes the output.
Inputs and weights are resident in HBM before the timed region starts.

Default workload: a Mixtral-8x7B-style MoE layer in bf16 -- 4096 queued
tokens, d = 4096, ffn = 14336, 8 experts, top-2, Zipf(1.2) expert skew,
arriving as 4 fragments.

Prints ONE JSON line (rank 0, N = 1).  Besides the throughput it reports the
roofline position of the dominant kernel (the gate/up launch, timed with HIP
events on the stream it runs on) and the CPU oracle timed on a bounded
sample of the same workload on this host.
"""

from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

METRIC = "expert-layer tokens/sec + % MFMA peak (hot) / % HBM BW (cold), Zipf-skewed"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_SCLK_GHZ = 2.4     # clock the published MFMA peaks assume
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c2", help="synth workload name (routed mode)")
    ap.add_argument("--cpu-budget-s", type=float, default=15.0,
                    help="CPU seconds the oracle baseline may use (it runs whole-layer passes until the budget "
                         "is spent, at least one)")
    ap.add_argument("--cpu-sample-tokens", type=int, default=0,
                    help="tokens of the workload the CPU oracle is timed on")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--ep-layer", choices=["bf16", "fp8"], default=None,
                    help="only the EP share as a whole layer (16 experts, rows mode), with these weights")
    ap.add_argument("--threads", type=int, default=min(16, os.cpu_count() or 1),
                    help="host threads for input generation")
    ap.add_argument("--no-cold", action="store_true",
                    help="skip the cold-expert (weight-streaming) measurements")
    ap.add_argument("--step-only", action="store_true",
                    help="time the step alone: skip the cold, hot-expert and 8-layer drain measurements")
    ap.add_argument("--cold-only", action="store_true",
                    help="only the weight-streaming measurements (cold experts and the sweep)")
    ap.add_argument("--cold-case", default=None,
                    choices=["finegrained_bf16", "ep_share_bf16", "ep_share_fp8", "sweep_d4096_f2048_bf16_n64"],
                    help="one cold measurement alone (for profiling its launches)")
    ap.add_argument("--sched-sim", action="store_true",
                    help="only run the host expert-runtime model (scheduling policies under a synthetic "
                         "request stream) and print its JSON summary")
    ap.add_argument("--pool", action="store_true",
                    help="only time the workload drained one expert at a time through the token pool "
                         "(route with caller ids, per-expert re-batch + FFN + pool merge, release) and print "
                         "its JSON summary")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES three times (reference "
                         "kernel for scaling HBM byte counters) and exit")
    return ap.parse_args()


HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "paper_2505_08944_amd", "csrc")


def kernel_source_sha256() -> str:
    """Hash of every HIP source and header the library is built from: HBM
    counter readings are only valid for the kernels they were taken on."""
    import hashlib
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".h")):
            with open(os.path.join(CSRC, name), "rb") as f:
                h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


def traffic_record(workload: str):
    """Per-launch HBM bytes of the gate/up kernel from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE summary of this workload, or None when
    there is none or the kernels changed since it was taken."""
    import re
    path = os.path.join(HERE, "profiles", f"ffn_gate_up_{workload}_hbm_traffic.md")
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    rec = dict(re.findall(r"^(\w+): (\S+)$", txt, re.M))
    try:
        if rec["source_sha256"] != kernel_source_sha256():
            return None
        return {"bytes": float(rec["hbm_bytes_per_launch"]), "fetch_bytes": float(rec["fetch_bytes_per_launch"]),
                "write_bytes": float(rec["write_bytes_per_launch"]), "source": os.path.relpath(path, HERE)}
    except (KeyError, ValueError):
        return None


SCHED_POLICIES = [("mtfs", 0.0, 0), ("flfs", 0.0, 0), ("defrag", 0.5, 2), ("defrag", 0.9, 4)]


def sched_sim(scenarios=("frag", "livelock"), granularities=("block", "expert"), horizon_us=None):
    """Scheduling policies on the host expert-runtime model (libaep's
    aep_sim_run): batch size per step, fragmentation (blocks holding queued
    rows after a step), decode throughput and request latency."""
    import synth
    from paper_2505_08944_amd import sched
    out = {}
    for name in scenarios:
        sc = synth.scenario(name)
        if horizon_us:
            sc = __import__("dataclasses").replace(sc, horizon_us=horizon_us)
        st = synth.request_stream(sc)
        arr, ol = st["arrival_us"], st["out_len"]
        res = {"description": sc.description, "requests": int(arr.size), "horizon_s": sc.horizon_us / 1e6}
        for gran in granularities:
            for pol, delta, la in SCHED_POLICIES:
                t0 = time.perf_counter()
                r = sched.sim_run(n_blocks=sc.n_blocks, n_experts=sc.n_experts, top_k=sc.top_k, n_frag=sc.n_frag,
                                  granularity=gran, policy=pol, arrival_us=arr, out_len=ol,
                                  expert_cdf=st["expert_cdf"], attn_us=sc.attn_us, jitter_us=sc.jitter_us,
                                  cost_fixed_us=sc.cost_fixed_us, cost_row_ns=sc.cost_row_ns,
                                  horizon_us=sc.horizon_us, seed=sc.cfg_id, delta=delta, lookahead=la,
                                  trace_capacity=2_000_000)
                wall = time.perf_counter() - t0
                done = r["done_us"] >= 0
                lat = (r["done_us"][done] - arr[done]) / 1e3
                first_half = arr < sc.horizon_us // 2
                tr = r["trace"]
                key = f"{gran}/{pol}" + (f"(d={delta},L={la})" if pol == "defrag" else "")
                res[key] = {
                    "steps": r["steps"], "rows_per_step": round(r["rows"] / max(r["steps"], 1), 2),
                    "blocks_holding_rows": round(float(tr["blocks_busy_after"].mean()), 2) if r["recorded"] else 0.0,
                    "busy_frac": round(r["busy_us"] / sc.horizon_us, 3),
                    "decode_tokens_per_s": round(float(ol[done].sum()) / (sc.horizon_us / 1e6), 1),
                    "requests_done_first_half": round(float(done[first_half].mean()), 4) if first_half.any() else None,
                    "latency_ms_p50": round(float(np.median(lat)), 1) if lat.size else None,
                    "latency_ms_p99": round(float(np.percentile(lat, 99)), 1) if lat.size else None,
                    "rows_queued_at_end": r["rows_queued_at_end"], "model_wall_s": round(wall, 2)}
        out[name] = res
    return out


def pool_measurement(name: str, steps: int, warmup: int, threads: int):
    """The workload's layer drained expert by expert through the token pool:
    route with caller ids, then for every expert re-batch, gate/up, down and
    pool merge, then one release.  Inputs resident in HBM; HIP events on the
    launch stream around whole steps."""
    import torch
    import synth
    import paper_2505_08944_amd as aep
    w = synth.workload(name)
    if w.S or w.mode != "routed" or w.n_layers != 1:
        raise SystemExit(f"--pool needs a one-layer routed workload without shared experts ({name} is not)")
    dev = torch.device("cuda", 0)
    frags = synth.layer_fragments(w, 0)
    ws = synth.all_expert_weights(w, 0, threads=threads)
    act = torch.bfloat16 if w.act == "bf16" else torch.float32

    def dev_t(a, fmt):
        a = np.ascontiguousarray(a)
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev) if fmt == "bf16" else \
            torch.from_numpy(a).to(dev)

    xs = [dev_t(f["x"], w.act) for f in frags]
    lgs = [dev_t(f["logits"], "f32") for f in frags]
    T = sum(x.shape[0] for x in xs)
    ids, o = [], 0
    for x in xs:
        ids.append(torch.arange(o, o + x.shape[0], dtype=torch.int32, device=dev))
        o += x.shape[0]
    ctx = aep.Context(1, w.E, w.d, w.f, w.k, act=w.act, wdt=w.wdt, max_tokens_per_layer=T, token_pool=True)
    wdev = []
    for e, ex in enumerate(ws):
        t = [dev_t(ex[k], w.wdt) for k in ("gate", "up", "down")]
        ctx.set_expert_weights(0, e, *t)
        wdev.append(t)
    del ws
    y = torch.empty((T, w.d), dtype=act, device=dev)
    out = torch.empty((T, w.d), dtype=act, device=dev)
    ready = torch.empty(T, dtype=torch.int32, device=dev)

    def step():
        for x, lg, i in zip(xs, lgs, ids):
            ctx.route_enqueue_ids(0, x, lg, i)
        for e in range(w.E):
            b = ctx.rebatch_expert(0, e)
            ctx.expert_gate_up(b)
            ctx.expert_down(b, y)
            ctx.pool_accumulate(b, y)
            ctx.release(b)
        ctx.pool_release(0, out, ready)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ctx.sync()
    ms = e0.elapsed_time(e1) / steps
    released = int(ready.sum().item())
    return {"workload": w.description or w.name, "mode": "expert-by-expert drains through the token pool",
            "tokens": T, "ms_per_step": round(ms, 4), "tokens_per_s": round(T / ms * 1e3, 1),
            "released_last_step": released, "steps": steps, "warmup": warmup}


def copy_calibration(nbytes: int) -> None:
    import torch
    src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": nbytes, "launches": 3}), flush=True)


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.sched_sim:
        print(json.dumps({"sched_sim": sched_sim()}), flush=True)
        return
    if args.pool:
        print(json.dumps({"pool": pool_measurement(args.workload, args.steps, args.warmup, args.threads)}),
              flush=True)
        return
    if args.cold_case:
        print(json.dumps({"cold_case": cold_case(args.cold_case)}), flush=True)
        return
    if args.ep_layer:
        print(json.dumps({"ep_share_layer": ep_share_layer(args.ep_layer)}), flush=True)
        return
    if args.cold_only:
        print(json.dumps({"cold": cold_measurements(args), "fig3_sweep": fig3_sweep()}), flush=True)
        return
    if args.gpus != 1:
        sys.stderr.write("bench.py measures one GPU: the library has no multi-GPU path (experts would "
                         "shard across GPUs by expert parallelism); run with --gpus 1.\n")
        sys.exit(2)

    import torch
    import synth
    import paper_2505_08944_amd as aep

    w = synth.workload(args.workload)
    assert w.mode == "routed" and w.n_layers == 1
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)

    # ---------------------------------------------------------------- inputs
    t_gen = time.perf_counter()
    frags = synth.layer_fragments(w, 0)
    ws = synth.all_expert_weights(w, 0, threads=args.threads)
    act = torch.bfloat16 if w.act == "bf16" else torch.float32

    def dev_t(a, fmt):
        a = np.ascontiguousarray(a)
        if fmt == "bf16":
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        if fmt == "fp8":
            return torch.from_numpy(a).to(dev)
        return torch.from_numpy(a).to(dev)

    xs = [dev_t(f["x"], w.act) for f in frags]
    lgs = [dev_t(f["logits"], "f32") for f in frags]
    T = sum(x.shape[0] for x in xs)
    ctx = aep.Context(1, w.E, w.d, w.f, w.k, n_shared=w.S, renorm=w.renorm, act=w.act, wdt=w.wdt,
                      max_tokens_per_layer=T)
    wfmt = "f32" if w.wdt == "f32" else ("fp8" if w.wdt == "fp8" else "bf16")
    wdev = []
    for e, ex in enumerate(ws):
        tens = [dev_t(ex[k], wfmt) for k in ("gate", "up", "down")]
        sc = [dev_t(ex["gate_up_scale"], "bf16"), dev_t(ex["down_scale"], "bf16")] if w.wdt == "fp8" else [None, None]
        ctx.set_expert_weights(0, e, *tens, *sc)
        wdev.append(tens + sc)
    del ws
    t_gen = time.perf_counter() - t_gen
    N_routed = T * w.k
    n_rows = N_routed + w.S * T
    y = torch.empty((n_rows, w.d), dtype=act, device=dev)
    out = torch.empty((T, w.d), dtype=act, device=dev)

    # ---------------------------------------------------------------- step
    def step(evs=None):
        if evs:
            evs[0].record()
        for x, lg in zip(xs, lgs):
            ctx.route_enqueue(0, x, lg)
        if evs:
            evs[1].record()
        b = ctx.rebatch(0)
        if evs:
            evs[2].record()
        ctx.expert_gate_up(b)
        if evs:
            evs[3].record()
        ctx.expert_down(b, y)
        if evs:
            evs[4].record()
        ctx.combine(b, y, out)
        if evs:
            evs[5].record()
        ctx.release(b)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ctx.sync()
    counts = None
    # expert counts of this workload (outside the timed region)
    for x, lg in zip(xs, lgs):
        ctx.route_enqueue(0, x, lg)
    counts = ctx.expert_counts(0).tolist()
    b = ctx.rebatch(0)
    ctx.release(b)
    torch.cuda.synchronize()

    K = args.steps
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        step(events[i])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ctx.sync()  # device error flag must be clear

    # shader clock the gate/up launch runs at (clock probe, outside the timed
    # steps): cycles over 100 MHz ticks, summed over the workgroups
    clk = torch.zeros((torch.cuda.get_device_properties(0).multi_processor_count, 2), dtype=torch.int64,
                      device=dev)
    for x, lg in zip(xs, lgs):
        ctx.route_enqueue(0, x, lg)
    b = ctx.rebatch(0)
    ctx.set_clock_probe(clk)
    ctx.expert_gate_up(b)
    ctx.set_clock_probe(None)
    ctx.release(b)
    torch.cuda.synchronize()
    ck = clk.cpu().numpy().astype(np.float64)
    ck = ck[ck[:, 1] > 0]
    sclk_ghz = float(ck[:, 0].sum() / (ck[:, 1].sum() / 100e6) / 1e9) if len(ck) else None

    stage_names = ["route_enqueue", "rebatch", "gate_up", "down", "combine"]
    stage_ms = {n: float(np.mean([events[i][j].elapsed_time(events[i][j + 1]) for i in range(K)]))
                for j, n in enumerate(stage_names)}
    ms_per_step = elapsed * 1e3 / K
    tokens_per_s = T * K / elapsed

    # dominant kernel: the gate/up launch (2/3 of the FFN flops)
    gu_flops = 4.0 * w.d * w.f * n_rows          # two GEMMs of 2*d*f flops per row
    # algorithmic HBM bytes of the launch: gathered rows in, weights of every
    # expert with rows (gate + up), h rows out
    wbytes = {"bf16": 2, "fp8": 1, "f32": 4}[w.wdt]
    abytes = 2 if w.act == "bf16" else 4
    live = sum(1 for c in counts if c > 0) + w.S
    gu_bytes = float(n_rows * w.d * abytes + live * 2 * w.f * w.d * wbytes + n_rows * w.f * abytes)
    ffn_flops = 6.0 * w.d * w.f * n_rows
    gu_s = stage_ms["gate_up"] / 1e3
    achieved = gu_flops / gu_s / 1e12
    ffn_s = (stage_ms["gate_up"] + stage_ms["down"]) / 1e3
    tr = traffic_record(args.workload)
    kname = {"bf16": "aep::ffn_dlds_kernel<true, false>", "fp8": "aep::ffn_dlds_kernel<true, true>"}.get(
        w.wdt, "aep::ffn_f32_kernel<true>")
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": None if tr is None else tr["bytes"],
                "kernel": kname + " (gate/up launch)",
                "traffic_detail": tr,
                "algorithmic_bytes": gu_bytes,
                "per_launch": {"flops": gu_flops, "rows": n_rows, "flops_per_row": 4 * w.d * w.f,
                               "avg_ms": round(stage_ms["gate_up"], 4)},
                "sclk_ghz": None if sclk_ghz is None else round(sclk_ghz, 3),
                "frac_at_sclk": None if sclk_ghz is None else
                round(achieved / (PEAK_BF16_TFLOPS * sclk_ghz / PEAK_SCLK_GHZ), 4)}

    res = {
        "metric": METRIC, "value": round(tokens_per_s, 1), "unit": "tokens/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16" if w.act == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": w.description or w.name, "tokens": T, "d_model": w.d, "d_ffn": w.f,
                   "experts": w.E, "shared_experts": w.S, "top_k": w.k, "zipf_s": w.zipf_s,
                   "fragments": len(xs), "weights": w.wdt, "expert_counts": counts},
        "roofline": roofline,
        "paper_context": {
            "note": "the paper's end-to-end serving gains and one expert-step time, on other hardware; "
                    "not comparable to this per-layer metric (hence vs_baseline null)",
            "throughput_vs_sglang_top1": {"short": 2.7, "medium": 2.3, "reasonable": 2.0},
            "setting": "Mixtral 8x7B (MQA attention), 8x A100-SXM4 80GB: 4 attention-DP + 4 expert-EP GPUs",
            "throughput_vs_sglang_16_gpus": 3.0,
            "expert_step_ms_one_a100": 0.8},
        "stage_ms": {k: round(v, 4) for k, v in stage_ms.items()},
        "ffn": {"tflops": round(ffn_flops / ffn_s / 1e12, 2),
                "mfma_frac": round(ffn_flops / ffn_s / 1e12 / PEAK_BF16_TFLOPS, 4)},
        "setup_s": round(t_gen, 1),
    }

    del ctx, xs, lgs, y, out
    torch.cuda.empty_cache()

    # ------------------------------------------- hot experts, 8-layer drain, cold
    if not args.step_only:
        mixtral = args.workload == "c2"
        if mixtral:
            res["drain_c5"] = drain_measurement(wdev, args.threads)
        res["hot"] = hot_measurements(max(counts[:w.E]) if mixtral else 0,
                                      res["drain_c5"]["hottest_queue_rows"] if mixtral else 0)
    del wdev
    torch.cuda.empty_cache()
    if not args.no_cold and not args.step_only:
        res["cold"] = cold_measurements(args)
        res["fig3_sweep"] = fig3_sweep()
        res["ep_share_layer"] = {wdt: ep_share_layer(wdt) for wdt in ("bf16", "fp8")}

    # ---------------------------------------------------------------- CPU oracle
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, args.cpu_sample_tokens, args.cpu_budget_s)
        if args.workload == "c2":
            # the same oracle on two more of the workloads, bounded samples
            # (context for the main value; about 12 s more of host time)
            others = {}
            for name, n_tok, budget in (("c1", 0, 2.0), ("c3", 512, 5.0)):
                ow = synth.workload(name)
                r = cpu_baseline(ow, n_tok, budget)
                others[name] = {"workload": ow.description or name, "value": r["value"], "unit": r["unit"],
                                "sample": r["sample"]}
            res["cpu_baseline"]["other_workloads"] = others

    print(json.dumps(res), flush=True)


def _flush(buf, mode="read"):
    """Evict L2 and the 256 MB Infinity Cache before a cold measurement by
    streaming a 1 GiB buffer.  "read" only reads it (the caches then hold
    clean lines); "write" also writes it, leaving dirty lines whose write-back
    the measured kernels would pay for."""
    if mode == "write":
        buf.add_(1)
    else:
        buf.max()


def time_rows_ffn(groups, d, f, wdt, reps=5, seed=0, flush="read"):
    """Grouped FFN over explicit per-expert rows (counts `groups`), weights of
    the given format drawn on the device; returns (seconds per gate/up + down,
    algorithmic bytes, flops).  Caches are flushed before every repetition."""
    import torch
    import paper_2505_08944_amd as aep
    dev = torch.device("cuda", 0)
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    E = len(groups)
    N = int(sum(groups))
    ctx = aep.Context(1, E, d, f, 1, wdt=wdt, max_tokens_per_layer=max(N, 1))
    W = []
    for e in range(E):
        if wdt == "fp8":
            mats = [torch.randint(0, 126, s, generator=g, device=dev, dtype=torch.uint8)
                    for s in [(f, d), (f, d), (d, f)]]
            sc = [torch.full((2 * f,), 1.0, dtype=torch.bfloat16, device=dev) * 0.001,
                  torch.full((d,), 1.0, dtype=torch.bfloat16, device=dev) * 0.001]
        else:
            mats = [(torch.randn(s, generator=g, device=dev) * 0.02).to(torch.bfloat16)
                    for s in [(f, d), (f, d), (d, f)]]
            sc = [None, None]
        ctx.set_expert_weights(0, e, *mats, *sc)
        W.append(mats + sc)
    rows = [torch.randn((n, d), generator=g, device=dev).to(torch.bfloat16) for n in groups]
    tok = torch.arange(N, dtype=torch.int32, device=dev)
    gw = torch.ones(N, dtype=torch.float32, device=dev)
    o = 0
    for e, n in enumerate(groups):
        if n:
            ctx.enqueue_rows(0, e, rows[e], tok[o:o + n], gw[o:o + n], N)
        o += n
    b = ctx.rebatch(0)
    y = torch.empty((b.n_rows, d), dtype=torch.bfloat16, device=dev)
    flush_mode = flush
    flush_buf = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    ctx.expert_gate_up(b)
    ctx.expert_down(b, y)
    times = []
    for _ in range(reps):
        if flush_mode != "none":
            _flush(flush_buf, flush_mode)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        ctx.expert_gate_up(b)
        ctx.expert_down(b, y)
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) / 1e3)
    ctx.release(b)
    ctx.sync()
    wbytes = 3 * d * f * (1 if wdt == "fp8" else 2) + (2 * (2 * f + d) if wdt == "fp8" else 0)
    nonempty = sum(1 for n in groups if n)
    byts = nonempty * wbytes + N * 2 * d * 2
    t = float(np.median(times))
    del ctx, W, rows, flush_buf
    torch.cuda.empty_cache()
    return t, byts, 6.0 * d * f * N


def ep_share_layer(wdt: str, steps: int = 20, warmup: int = 3):
    """One GPU's expert-parallel share as a whole layer: the 16 resident
    experts' queues (Zipf depths 4096 ... 111 rows) enqueued as explicit
    rows in one grouped call (one receive buffer, rows grouped by expert),
    re-batched and run through both FFN launches, steps back to back on one
    stream; rows/s = routed rows / time per step."""
    import synth
    import torch
    import paper_2505_08944_amd as aep
    dev = torch.device("cuda", 0)
    w4 = synth.workload("c4")
    groups = [int(n) for n in synth.rows_workload(w4)["depths"].tolist()]
    d, f, E, N = w4.d, w4.f, len(groups), int(sum(groups))
    g = torch.Generator(device=dev)
    g.manual_seed(4)
    ctx = aep.Context(1, E, d, f, 1, wdt=wdt, max_tokens_per_layer=N)
    W = []
    for e in range(E):
        if wdt == "fp8":
            mats = [torch.randint(0, 126, s, generator=g, device=dev, dtype=torch.uint8)
                    for s in [(f, d), (f, d), (d, f)]]
            sc = [torch.full((2 * f,), 1.0, dtype=torch.bfloat16, device=dev) * 0.001,
                  torch.full((d,), 1.0, dtype=torch.bfloat16, device=dev) * 0.001]
        else:
            mats = [(torch.randn(s, generator=g, device=dev) * 0.02).to(torch.bfloat16)
                    for s in [(f, d), (f, d), (d, f)]]
            sc = [None, None]
        ctx.set_expert_weights(0, e, *mats, *sc)
        W.append(mats + sc)
    rows = torch.randn((N, d), generator=g, device=dev).to(torch.bfloat16)
    tok = torch.arange(N, dtype=torch.int32, device=dev)
    gw = torch.ones(N, dtype=torch.float32, device=dev)
    y = torch.empty((N, d), dtype=torch.bfloat16, device=dev)

    def step():
        ctx.enqueue_rows_grouped(0, groups, rows, tok, gw, N)
        b = ctx.rebatch(0)
        ctx.expert_ffn(b, y[:b.n_rows])
        ctx.release(b)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ctx.sync()
    t = e0.elapsed_time(e1) / 1e3 / steps
    fl = 6.0 * d * f * N
    del ctx, W, rows, y
    torch.cuda.empty_cache()
    return {"experts": E, "rows": N, "weights": wdt, "ms_per_step": round(t * 1e3, 4),
            "rows_per_s": round(N / t, 1), "tflops": round(fl / t / 1e12, 1),
            "mfma_frac": round(fl / t / 1e12 / PEAK_BF16_TFLOPS, 4), "steps": steps}


def stream_reference():
    """The achievable-bandwidth reference beside the cold fractions: torch's
    own copy kernel over 1 GiB on this GPU (bytes read + written), caches
    flushed first (median of 5)."""
    import torch
    dev = torch.device("cuda", 0)
    n = 1 << 30
    src = torch.ones(n // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    flush_buf = torch.empty(n, dtype=torch.uint8, device=dev)
    res = {}
    for name, fn, moved in (("copy", lambda: dst.copy_(src), 2 * n),):
        fn()
        ts = []
        for _ in range(5):
            _flush(flush_buf, "read")
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) / 1e3)
        gbs = moved / float(np.median(ts)) / 1e9
        res[f"{name}_GBps"] = round(gbs, 1)
        res[f"{name}_frac"] = round(gbs / PEAK_HBM_GBS, 4)
    res["note"] = "torch copy_ of 1 GiB (bytes read + written), caches flushed"
    del src, dst, flush_buf
    torch.cuda.empty_cache()
    return res


def hot_measurements(c2_hot_rows: int, drain_hot_rows: int):
    """MFMA side of the metric: one expert's whole queue as a single group
    (gate/up + down), caches warm: the hottest queue of the Mixtral-style
    layer, the EP share's 4096-row expert (bf16 and fp8 weights) and the
    hottest queue of the 8-layer drain (row counts measured on the device)."""
    out = {}
    cases = []
    if c2_hot_rows:
        cases.append(("mixtral_hottest", c2_hot_rows, 4096, 14336, "bf16"))
    cases += [("ep_share_4096", 4096, 4096, 2048, "bf16"), ("ep_share_4096", 4096, 4096, 2048, "fp8")]
    if drain_hot_rows:
        cases.append(("drain_hottest", drain_hot_rows, 4096, 14336, "bf16"))
    for name, n, d, f, wdt in cases:
        t, byts, fl = time_rows_ffn([n], d, f, wdt, reps=5, flush="none")
        out[f"{name}_d{d}_f{f}_{wdt}"] = {"rows": n, "ms": round(t * 1e3, 4), "tflops": round(fl / t / 1e12, 1),
                                           "mfma_frac": round(fl / t / 1e12 / PEAK_BF16_TFLOPS, 4)}
    return out


def drain_measurement(c2_weights, threads: int, reps: int = 3):
    """The asynchronous 8-layer drain: 8 MoE layers at the Mixtral-style shape
    (layer weights: the layer's 8 experts drawn from the same 8 synthetic
    experts, rotated per layer, each (layer, expert) its own copy), 0..8192
    tokens per layer, 32768 in total.  One pass routes every layer's fragments
    into its mu-queues, then repeatedly picks the layer with the most queued
    rows (host, no sync), re-batches it, runs its experts and combines, until
    every queue is empty.  Wall time of the pass, host picks included."""
    import torch
    import synth
    import paper_2505_08944_amd as aep
    w = synth.workload("c5")
    dev = torch.device("cuda", 0)
    ctx = aep.Context(w.n_layers, w.E, w.d, w.f, w.k, max_tokens_per_layer=max(max(w.tokens), 1))
    wdev = []
    for l in range(w.n_layers):
        for e in range(w.E):
            src = synth.weight_source(w, l, e)[2]
            t = [m.clone() for m in c2_weights[src][:3]]
            ctx.set_expert_weights(l, e, *t)
            wdev.append(t)
    frags = []
    for l in range(w.n_layers):
        fl = []
        for f in synth.layer_fragments(w, l):
            x = torch.from_numpy(np.ascontiguousarray(f["x"]).view(np.int16)).view(torch.bfloat16).to(dev)
            fl.append((x, torch.from_numpy(np.ascontiguousarray(f["logits"])).to(dev)))
        frags.append(fl)
    ys = {l: torch.empty((2 * w.tokens[l], w.d), dtype=torch.bfloat16, device=dev) for l in range(w.n_layers)}
    outs = {l: torch.empty((w.tokens[l], w.d), dtype=torch.bfloat16, device=dev) for l in range(w.n_layers)}

    def one_pass():
        for l in range(w.n_layers):
            for x, lg in frags[l]:
                ctx.route_enqueue(l, x, lg)
        order = []
        while (l := ctx.pick_layer("mtfs")) is not None:
            order.append(l)
            b = ctx.rebatch(l)
            ctx.expert_gate_up(b)
            ctx.expert_down(b, ys[l])
            ctx.combine(b, ys[l], outs[l])
            ctx.release(b)
        return order

    one_pass()
    torch.cuda.synchronize()
    ctx.sync()
    hottest = 0
    for l in range(w.n_layers):
        for x, lg in frags[l]:
            ctx.route_enqueue(l, x, lg)
        hottest = max(hottest, int(ctx.expert_counts(l).max()))
    while (l := ctx.pick_layer("mtfs")) is not None:
        ctx.release(ctx.rebatch(l))
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        order = one_pass()
        torch.cuda.synchronize()
        times.append(time.perf_counter() - t0)
    ctx.sync()
    T = sum(w.tokens)
    t = float(np.median(times))
    flops = 6.0 * w.d * w.f * 2 * T
    res = {"workload": w.description, "layers": w.n_layers, "tokens": T, "layer_tokens": list(w.tokens),
           "order": order, "hottest_queue_rows": hottest, "ms": round(t * 1e3, 3),
           "tokens_per_s": round(T / t, 1), "ffn_tflops": round(flops / t / 1e12, 1), "reps": reps}
    del ctx, wdev, frags, ys, outs
    torch.cuda.empty_cache()
    return res


def cold_measurements(args):
    """Weight-streaming side of the metric: experts with <= 256 queued rows.

    * fine-grained layer (d=2048, ffn=1408): the cold experts of the routed
      64-expert layer (their counts from the same synthetic routing);
    * one GPU's EP share (d=4096, ffn=2048): the cold experts of the Zipf
      depths, bf16 and fp8 weights;
    """
    import synth
    import torch
    import paper_2505_08944_amd as aep
    out = {}
    # fine-grained layer: routed counts
    w3 = synth.workload("c3")
    frags = synth.layer_fragments(w3, 0)
    T = sum(f["x"].shape[0] for f in frags)
    ctx = aep.Context(1, w3.E, w3.d, w3.f, w3.k, n_shared=w3.S, max_tokens_per_layer=T)
    for f in frags:
        x = torch.from_numpy(f["x"].view(np.int16)).view(torch.bfloat16).cuda()
        lg = torch.from_numpy(f["logits"]).cuda()
        ctx.route_enqueue(0, x, lg)
    counts3 = ctx.expert_counts(0).tolist()
    del ctx
    cold3 = [n for n in counts3 if 0 < n <= 256]
    t, byts, fl = time_rows_ffn(cold3, w3.d, w3.f, "bf16")
    out["finegrained_d2048_f1408_bf16"] = {"experts": len(cold3), "rows": sum(cold3), "ms": round(t * 1e3, 4),
                                           "GBps": round(byts / t / 1e9, 1),
                                           "hbm_frac": round(byts / t / 1e9 / PEAK_HBM_GBS, 4),
                                           "bytes": byts}
    w4 = synth.workload("c4")
    depths = synth.rows_workload(w4)["depths"].tolist()
    cold4 = [n for n in depths if n <= 256]
    for wdt in ("bf16", "fp8"):
        t, byts, fl = time_rows_ffn(cold4, w4.d, w4.f, wdt)
        out[f"ep_share_d4096_f2048_{wdt}"] = {"experts": len(cold4), "rows": sum(cold4), "ms": round(t * 1e3, 4),
                                             "GBps": round(byts / t / 1e9, 1),
                                             "hbm_frac": round(byts / t / 1e9 / PEAK_HBM_GBS, 4), "bytes": byts}
    out["stream_reference"] = stream_reference()
    return out


def cold_case(name: str):
    """One cold measurement alone: its launches are the only FFN launches of
    the process (5 timed repetitions after one untimed pass, caches flushed
    before each), for rocprofv3 runs."""
    import synth
    if name == "finegrained_bf16":
        import torch
        import paper_2505_08944_amd as aep
        w3 = synth.workload("c3")
        frags = synth.layer_fragments(w3, 0)
        T = sum(f["x"].shape[0] for f in frags)
        ctx = aep.Context(1, w3.E, w3.d, w3.f, w3.k, n_shared=w3.S, max_tokens_per_layer=T)
        for f in frags:
            ctx.route_enqueue(0, torch.from_numpy(f["x"].view(np.int16)).view(torch.bfloat16).cuda(),
                              torch.from_numpy(f["logits"]).cuda())
        groups = [n for n in ctx.expert_counts(0).tolist() if 0 < n <= 256]
        del ctx
        d, f, wdt = w3.d, w3.f, "bf16"
    elif name.startswith("ep_share"):
        depths = synth.rows_workload(synth.workload("c4"))["depths"].tolist()
        groups = [n for n in depths if n <= 256]
        d, f, wdt = 4096, 2048, name.split("_")[-1]
    else:
        d, f, wdt = 4096, 2048, "bf16"
        groups = [64] * -(-(1 << 30) // (3 * d * f * 2))
    t, byts, fl = time_rows_ffn(groups, d, f, wdt)
    return {"case": name, "experts": len(groups), "rows": int(sum(groups)), "d": d, "f": f, "weights": wdt,
            "ms": round(t * 1e3, 4), "bytes": byts, "flops": fl,
            "hbm_frac": round(byts / t / 1e9 / PEAK_HBM_GBS, 4)}


def fig3_sweep(ns=(16, 32, 64, 128, 256), shapes=((2048, 1408), (4096, 2048), (4096, 14336)),
               wdts=("bf16", "fp8"), reps=3):
    """Weight-streaming sweep after the paper's single-layer throughput-vs-
    batch-size figure (Sec. 2, Fig. 3: small batches are bound by memory
    bandwidth).  For each expert shape (the fine-grained layer's, the EP
    share's, the Mixtral-style layer's) and weight format: G same-shape
    experts, G chosen so their weights total >= 1 GiB (4x the 256 MB Infinity
    Cache), each holding n queued rows; gate/up + down of the grouped launch
    timed with the caches flushed by a 1 GiB read before every repetition.
    Reported: algorithmic bytes (the weights of every expert, rows in, y out)
    over the time, as a fraction of 8 TB/s (median of reps)."""
    import torch
    import paper_2505_08944_amd as aep
    dev = torch.device("cuda", 0)
    flush_buf = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    points, groups = {}, {}
    for d, f in shapes:
        for wdt in wdts:
            wb = 3 * d * f * (1 if wdt == "fp8" else 2) + (2 * (2 * f + d) if wdt == "fp8" else 0)
            G = -(-(1 << 30) // wb)
            nmax = max(ns)
            g = torch.Generator(device=dev)
            g.manual_seed(d * 7 + f)
            ctx = aep.Context(1, G, d, f, 1, wdt=wdt, max_tokens_per_layer=G * nmax)
            W = []
            for e in range(G):
                if wdt == "fp8":
                    mats = [torch.randint(0, 126, sh, generator=g, device=dev, dtype=torch.uint8)
                            for sh in [(f, d), (f, d), (d, f)]]
                    sc = [torch.full((2 * f,), 0.001, dtype=torch.bfloat16, device=dev),
                          torch.full((d,), 0.001, dtype=torch.bfloat16, device=dev)]
                else:
                    mats = [(torch.randn(sh, generator=g, device=dev) * 0.02).to(torch.bfloat16)
                            for sh in [(f, d), (f, d), (d, f)]]
                    sc = [None, None]
                ctx.set_expert_weights(0, e, *mats, *sc)
                W.append(mats + sc)
            rows = torch.randn((G * nmax, d), generator=g, device=dev).to(torch.bfloat16)
            tok = torch.arange(G * nmax, dtype=torch.int32, device=dev)
            gw = torch.ones(G * nmax, dtype=torch.float32, device=dev)
            y = torch.empty((G * nmax, d), dtype=torch.bfloat16, device=dev)
            key = f"d{d}_f{f}_{wdt}"
            points[key], groups[key] = {}, G
            for n in ns:
                for e in range(G):
                    sl = slice(e * n, (e + 1) * n)
                    ctx.enqueue_rows(0, e, rows[sl], tok[sl], gw[sl], G * n)
                b = ctx.rebatch(0)
                yb = y[:b.n_rows]
                ctx.expert_gate_up(b)
                ctx.expert_down(b, yb)
                times = []
                for _ in range(reps):
                    _flush(flush_buf, "read")
                    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    e0.record()
                    ctx.expert_gate_up(b)
                    ctx.expert_down(b, yb)
                    e1.record()
                    torch.cuda.synchronize()
                    times.append(e0.elapsed_time(e1) / 1e3)
                ctx.release(b)
                t = float(np.median(times))
                points[key][f"n{n}"] = round((G * wb + G * n * 2 * d * 2) / t / 1e9 / PEAK_HBM_GBS, 4)
            ctx.sync()
            del ctx, W, rows, tok, gw, y
            torch.cuda.empty_cache()
    le64 = [v for k in points for n, v in points[k].items() if int(n[1:]) <= 64]
    return {"unit": "fraction of 8 TB/s (algorithmic bytes / time)", "experts": groups, "points": points,
            "le64_rows_min": min(le64), "le64_rows_mean": round(float(np.mean(le64)), 4)}


def cpu_baseline(w, n_tok: int, budget_s: float = 15.0):
    """The oracle, as it stands, on the first n_tok tokens of the workload (0:
    all of them), repeated while the time budget lasts; the median pass is
    reported."""
    import oracle
    import synth
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        blas_threads = None
    frags = synth.layer_fragments(w, 0)
    T = sum(f["x"].shape[0] for f in frags)
    n_tok = T if n_tok <= 0 else min(n_tok, T)
    x = np.concatenate([f["x"] for f in frags])[:n_tok]
    lg = np.concatenate([f["logits"] for f in frags])[:n_tok]
    ws = synth.all_expert_weights(w, 0, threads=min(16, os.cpu_count() or 1))
    times = []
    t_start = time.perf_counter()
    while not times or time.perf_counter() - t_start + times[-1] <= budget_s:
        t0 = time.perf_counter()
        lq = oracle.LayerQueues(w.E, w.k, w.S, w.renorm)
        lq.enqueue_routed(x, lg)
        oracle.moe_layer(lq, ws, w.act, "f32" if w.wdt == "f32" else w.wdt)
        times.append(time.perf_counter() - t0)
    dt = float(np.median(times))
    cpu = platform.processor() or platform.machine()
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": round(n_tok / dt, 2), "unit": "tokens/s", "cores": blas_threads, "kind": "oracle",
            "sample": f"{'all' if n_tok == T else f'first {n_tok} of'} {T} tokens, whole layer (route, queue, "
                      f"re-batch, float64 SwiGLU experts, combine); median of {len(times)} passes, "
                      f"{dt:.1f} s each",
            "host_cpu": cpu, "host_logical_cpus": os.cpu_count()}


if __name__ == "__main__":
    main()
