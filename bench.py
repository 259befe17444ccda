#!/usr/bin/env python3
"""Benchmark: generated tokens/s of a ragged mixture-of-agents batch on one MI355X.

One step = the whole batch: every routed expert call of the workload (and the
aggregator calls, if the workload has an aggregator) submitted, generated to
its max_new_tokens and collected through the C ABI. The default workload is
four Llama-1B-shape experts (bf16, random init) serving 256 queries routed
top-2 by Zipf(1.2) popularity, with bimodal instruct/reasoning generation
lengths (512 calls, 541,743 generated tokens at seed 0) -- the skewed,
straggler-heavy expert phase of the paper (Sections "Motivation" and
"Workload Characterisation"). Weights, prompts and routing are synthetic.

Prints one JSON line. The ``roofline`` object covers the kernel class with
the largest share of the timed region; ``run_roofline`` is the whole run's
roofline time (sum over every launch of max(bytes/8 TB/s, flops/2.5 PF/s))
over the measured wall time; ``cpu_baseline`` times the fp64 oracle on a
bounded sample of the same workload.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK = 8.0e12            # bytes/s, MI355X HBM3E
MFMA_BF16_PEAK = 2.5e15      # flop/s, dense bf16
METRIC = "generated tokens/s on 1 MI355X (ragged MoA batch); attn/GEMM % of HBM/MFMA roof"


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def measured_traffic(kernel):
    """HBM bytes per launch of ``kernel`` from the committed rocprofv3 counter
    summary, or None when none exists or the kernel source changed since."""
    import glob
    import hashlib
    src = os.path.join(ROOT, "paper_2606_03014_amd", "csrc", "kernels.hip")
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    for path in glob.glob(os.path.join(ROOT, "profiles", "*traffic*.md")):
        for line in open(path):
            line = line.strip()
            if line.startswith("{") and '"traffic_bytes_per_launch"' in line:
                rec = json.loads(line)
                if rec.get("kernel") == kernel and rec.get("kernels_source_sha256_16") == sha:
                    return rec["traffic_bytes_per_launch"]
    return None


def cpu_baseline(cfg, wl, weights0, budget_s):
    """The oracle, as it stands, on the first expert-0 call of the workload:
    prefill its prompt, then decode until the time budget runs out."""
    import numpy as np
    from oracle import transformer as T
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count()
    om = T.OracleModel(cfg.model, weights0)
    for name in weights0:                       # fp64 upcast of the weights: setup, not timed
        om.W(name)
    q, e, G = next(r for r in wl.expert_requests() if r[1] == 0)
    prompt = wl.prompts[q]
    kv = T.ContiguousKV(cfg.model.n_layers, cfg.model.n_kv_heads, cfg.model.head_dim)
    t0 = time.perf_counter()
    lg = T.forward_chunk(om, prompt, 0, kv, bf16_kv=True, want="last")[-1]
    toks = [T.argmax_lowest(lg)]
    while len(toks) < G and time.perf_counter() - t0 < budget_s:
        lg = T.forward_chunk(om, [toks[-1]], len(prompt) + len(toks) - 1, kv, bf16_kv=True)[-1]
        toks.append(T.argmax_lowest(lg))
    dt = time.perf_counter() - t0
    return {"value": len(toks) / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": (f"expert 0 call of query {q}: prefill of {len(prompt)} prompt tokens plus "
                       f"{len(toks) - 1} decode steps ({len(toks)} generated tokens, {dt:.1f} s, "
                       f"fp64 numpy oracle with a KV cache)")}


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="moa-4x1b-bf16")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--queries", type=int, default=None, help="fewer queries (quick runs only)")
    ap.add_argument("--time-every", type=int, default=8, help="time the kernels of 1 step in N")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only copy a MIB-sized device buffer 8 times (HBM counter calibration) and exit")
    args = ap.parse_args()
    if args.copy_probe:
        import torch
        n = args.copy_probe << 20
        a = torch.empty(n, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        for _ in range(8):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "copies": 8}))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); this build has no "
              "multi-GPU path: the engine runs every model of the batch on one MI355X.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from moa_inputs import CONFIGS, generate_weights, make_workload, pack_blob
    from paper_2606_03014_amd import Engine, run_feeder

    cfg = CONFIGS[args.workload]
    wl = make_workload(cfg.name, args.seed, n_queries=args.queries)
    n_models = cfg.n_experts + (1 if cfg.aggregator else 0)
    log(f"[bench] {cfg.name}: {wl.n_queries} queries, {len(wl.max_new)} expert calls, {n_models} models")
    t = time.perf_counter()
    weights = [generate_weights(cfg.model, cfg.dtype, args.seed, cfg.wid, m) for m in range(n_models)]
    log(f"[bench] weights generated in {time.perf_counter() - t:.1f} s")
    eng = Engine(cfg.model, cfg.dtype, cfg.engine, n_models)
    t = time.perf_counter()
    mids = [eng.load(pack_blob(w, cfg.model)) for w in weights]
    log(f"[bench] weights loaded in {time.perf_counter() - t:.1f} s; arena {eng.arena_bytes / 2**30:.1f} GiB")
    agg = mids[cfg.n_experts] if cfg.aggregator else -1

    t_start = [time.perf_counter()]

    def progress(info):
        if info.step % 1000 == 0:
            log(f"[bench]   engine step {info.step}: running {info.running}, pending {info.pending}, "
                f"{time.perf_counter() - t_start[0]:.1f} s")

    def one_step():
        t_start[0] = time.perf_counter()
        return run_feeder(eng, wl, mids[: cfg.n_experts], agg_model=agg, on_step=progress)

    for i in range(args.warmup):
        t = time.perf_counter()
        r = one_step()
        torch.cuda.synchronize()
        log(f"[bench] warmup {i}: {r.n_steps} engine steps, {r.tokens} tokens, {time.perf_counter() - t:.2f} s")

    eng.time_kernels(args.time_every, HBM_PEAK, MFMA_BF16_PEAK)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    tokens = 0
    n_engine_steps = 0
    for i in range(args.steps):
        r = one_step()
        tokens += r.tokens
        n_engine_steps += r.n_steps
        log(f"[bench] step {i}: {r.n_steps} engine steps, {r.tokens} tokens")
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    wall = t1 - t0
    stats = eng.kernel_stats()

    # kernel classes by timed share; per-class achieved rates
    total_timed = sum(s["ms"] for s in stats.values()) or 1.0
    for name, s in sorted(stats.items(), key=lambda kv: -kv[1]["ms"]):
        if s["launches"]:
            log(f"[bench] {name:12s} {100 * s['ms'] / total_timed:5.1f}% of timed  "
                f"{s['ms'] / s['launches'] * 1e3:8.1f} us/launch  "
                f"{s['bytes'] / (s['ms'] * 1e-3) / 1e9:8.1f} GB/s  {s['flops'] / (s['ms'] * 1e-3) / 1e12:7.1f} TF/s")
    dom_name, dom = max(stats.items(), key=lambda kv: kv[1]["ms"])
    intensity = dom["flops"] / max(dom["bytes"], 1.0)
    mfma_bound = intensity > MFMA_BF16_PEAK / HBM_PEAK
    if mfma_bound:
        achieved = dom["flops"] / (dom["ms"] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": MFMA_BF16_PEAK / 1e12, "unit": "TFLOP/s"}
    else:
        achieved = dom["bytes"] / (dom["ms"] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK / 1e9, "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = measured_traffic(dom_name)
    roof["kernel"] = dom_name
    roof["launches_timed"] = dom["launches"]
    roof["us_per_launch"] = dom["ms"] / max(dom["launches"], 1) * 1e3
    roof["algorithmic_bytes_per_launch"] = dom["bytes"] / max(dom["launches"], 1)
    run_roof_ms = sum(s["roof_ms_all"] for s in stats.values())

    out = {
        "metric": METRIC,
        "value": tokens / wall,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": cfg.name, "models": n_models, "queries": wl.n_queries,
                   "expert_calls": len(wl.max_new), "generated_tokens_per_step": tokens // args.steps,
                   "engine_steps_per_step": n_engine_steps // args.steps, "seed": args.seed,
                   "parallelism": "single GPU"},
        "roofline": roof,
        "run_roofline": {"roof_ms": run_roof_ms / args.steps, "measured_ms": wall * 1e3 / args.steps,
                         "frac": run_roof_ms / (wall * 1e3)},
    }
    eng.close()
    del eng
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, wl, weights[0], args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
