#!/usr/bin/env python3
"""Benchmark: generated tokens/s of a ragged mixture-of-agents batch on one MI355X.

The default workload is the paper's own setting (Section "Problem Setting";
Section "MOSAIC: Adaptive Aggregation"): three expert models and one
aggregator, all of Llama-8B shape (bf16, random init), co-resident on one GPU
with one shared paged KV pool. 1,024 queries are routed top-2 by Zipf(1.0)
popularity, and generation lengths are bimodal (60% instruct-style U[128,
1024], 40% reasoning-style lognormal with median 4,096 capped at 16,384).
The aggregator call of a query, on the query followed by its experts'
outputs, emits 512 tokens. Weights, prompts and routing are synthetic.

One bench step = a fixed block of ``--block-steps`` consecutive engine steps
(128 by default) of that workload's deterministic schedule, driven by the
host feeder from the first submit. The warm-up steps are the schedule's first
blocks (admission and the initial prefill burst). The timed steps are the
blocks that follow, a stated window of engine steps of the expert phase with
aggregator calls arriving. Every token those engine steps emit is counted
(their decode rows plus the prompts they complete). Nothing is skipped: each
engine step runs every layer of every row of every model it holds. The whole
workload takes about 42,000 engine steps, too long for one bench run.
``--block-steps 0`` makes a bench step the whole batch (other workloads).

Prints one JSON line. ``roofline`` covers the kernel class with the largest
share of the timed region's kernel time; ``bars`` reports the classes the
design targets are set on (decode attention and the small/medium-row GEMMs
against HBM, the large-row GEMMs against bf16 MFMA); ``run_roofline`` is the
whole run's roofline time (sum over every launch of max(bytes/8 TB/s,
flops/2.5 PF/s)) over the measured wall time; ``cpu_baseline`` times the fp64
oracle on a fixed slice of the same workload.
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
# per-step cost model of the schedule study: the decode streaming rate and
# the useful prefill rates this engine reaches on 8B shapes (large-M GEMM,
# causal prefill attention)
STUDY_BW = 5.0e12
STUDY_LIN = 4.7e14
STUDY_ATTN = 3.2e14
DEFAULT_STREAMS = 2


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_code_digest(path):
    """sha256/16 of a kernel source with its comments and blank lines taken
    out, so that a counter record stays valid across edits to comments only
    (the compiled kernels are the same) and lapses with any change to code."""
    import hashlib
    import re
    src = open(path, encoding="utf-8").read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    lines = [ln.rstrip() for ln in src.splitlines() if ln.strip()]
    return hashlib.sha256("\n".join(lines).encode()).hexdigest()[:16]


def measured_traffic(kernel, workload, streams=1):
    """HBM bytes per launch of ``kernel`` on ``workload`` from the committed
    rocprofv3 counter summaries, or None when none exists, the kernel source
    code changed since (kernel_code_digest), or the counters were taken with
    another number of model streams (which changes what one launch carries). The roofline's launches
    are those of the steps sampled for timing, which always run on one
    stream, so it asks for the one-stream counters."""
    import glob
    sha = kernel_code_digest(os.path.join(ROOT, "paper_2606_03014_amd", "csrc", "kernels.hip"))
    for path in glob.glob(os.path.join(ROOT, "profiles", "*traffic*.md")):
        for line in open(path):
            line = line.strip()
            if line.startswith("{") and '"traffic_bytes_per_launch"' in line:
                rec = json.loads(line)
                if (rec.get("kernel") == kernel and rec.get("kernels_code_sha256_16") == sha
                        and rec.get("workload") == workload and rec.get("model_streams", 1) == streams):
                    return rec["traffic_bytes_per_launch"]
    return None


def host_cpu():
    """The host's logical CPUs (nproc), the CPUs this process may run on, and
    the CPU model name from lscpu."""
    import subprocess
    model = None
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                model = line.split(":", 1)[1].strip()
                break
    except Exception:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except Exception:
        usable = os.cpu_count()
    return {"nproc": os.cpu_count(), "usable_cpus": usable, "model": model}


def oracle_threads():
    """Threads the oracle's BLAS calls use (its only parallel part)."""
    try:
        from threadpoolctl import threadpool_info
        return int(max([i.get("num_threads", 1) for i in threadpool_info()] or [1]))
    except Exception:
        return os.cpu_count()


def upcast_oracle(om, names):
    """Fill the oracle's float64 weight cache (setup, not timed). One tensor
    at a time: threads converting several tensors at once ran ten times
    slower here."""
    for name in names:
        om.W(name)


CPU_DECODE = 8          # decode steps of the oracle slice
CPU_PREFILL_MAX = 256   # prompt positions of the oracle slice at most


def cpu_baseline(cfg, wl, weights0):
    """The oracle, as it stands, on a fixed slice of the workload: the first
    call of model 0 (an expert call, or the first aggregator call when there
    are no experts). Its prompt (the first CPU_PREFILL_MAX positions of it at
    most) is prefilled at full depth in one pass, then CPU_DECODE greedy
    decode steps run with a KV cache; value = the slice's generated tokens /
    its wall time, on every BLAS thread. The decode steps are timed again on
    one thread (continuing the same call)."""
    from oracle import transformer as T
    om = T.OracleModel(cfg.model, weights0)
    upcast_oracle(om, list(weights0))
    reqs = [r for r in wl.expert_requests() if r[1] == 0]
    q, G = (reqs[0][0], reqs[0][2]) if reqs else (0, wl.agg_max_new)
    prompt = wl.prompts[q][:CPU_PREFILL_MAX]
    D = max(0, min(CPU_DECODE, G - 1))
    kv = T.ContiguousKV(cfg.model.n_layers, cfg.model.n_kv_heads, cfg.model.head_dim)
    threads = oracle_threads()
    t0 = time.perf_counter()
    lg = T.forward_chunk(om, prompt, 0, kv, bf16_kv=cfg.dtype == "bf16", want="last")[-1]
    t_pre = time.perf_counter() - t0
    toks = [T.argmax_lowest(lg)]
    for _ in range(D):
        lg = T.forward_chunk(om, [toks[-1]], len(prompt) + len(toks) - 1, kv, bf16_kv=cfg.dtype == "bf16")[-1]
        toks.append(T.argmax_lowest(lg))
    dt = time.perf_counter() - t0
    t_dec = dt - t_pre
    one = None
    try:
        from threadpoolctl import threadpool_limits
        n1 = 2
        with threadpool_limits(1):
            t1 = time.perf_counter()
            for _ in range(n1):
                lg = T.forward_chunk(om, [toks[-1]], len(prompt) + len(toks) - 1, kv,
                                     bf16_kv=cfg.dtype == "bf16")[-1]
                toks.append(T.argmax_lowest(lg))
            one = {"decode_tokens_per_s": n1 / (time.perf_counter() - t1), "threads": 1,
                   "sample": f"{n1} further decode steps of the same call on one BLAS thread"}
    except Exception as err:            # threadpoolctl missing: say so instead of guessing
        one = {"unavailable": str(err)}
    return {"value": (1 + D) / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": (f"the workload's first model-0 call (query {q}): its {len(prompt)}-token prompt "
                       f"prefilled at full depth in one pass ({t_pre:.1f} s, 1 token), then {D} greedy "
                       f"decode steps with a KV cache ({t_dec:.1f} s); fp64 numpy oracle, "
                       f"{1 + D} generated tokens in {dt:.1f} s"),
            "prefill_s": t_pre, "decode_tokens_per_s": D / t_dec if D else None,
            "host": host_cpu(), "single_thread": one}


def cpu_baseline_history(cfg, seed, weights0):
    """The oracle on the straggler workload's first sequence: its synthetic
    K/V history (bf16-rounded) in a contiguous cache, then CPU_DECODE decode
    steps (fewer if its remaining length is shorter)."""
    import numpy as np
    from moa_inputs import make_straggler_workload, synthetic_kv, f32_to_bf16_bits
    from moa_inputs.weights import bf16_bits_to_f32
    from oracle import transformer as T
    m = cfg.model
    om = T.OracleModel(m, weights0)
    upcast_oracle(om, list(weights0))
    L, tok, R = make_straggler_workload(seed).sequence(0)
    hist = bf16_bits_to_f32(f32_to_bf16_bits(synthetic_kv(seed, 0, m.n_layers, L, m.n_kv_heads, m.head_dim)))
    kv = T.ContiguousKV(m.n_layers, m.n_kv_heads, m.head_dim)
    for l in range(m.n_layers):
        kv.K[l] = hist[l, 0].astype(np.float64)
        kv.V[l] = hist[l, 1].astype(np.float64)
    del hist
    t0 = time.perf_counter()
    toks = [tok]
    while len(toks) <= min(R, CPU_DECODE):
        lg = T.forward_chunk(om, [toks[-1]], L + len(toks) - 1, kv, bf16_kv=True)[-1]
        toks.append(T.argmax_lowest(lg))
    dt = time.perf_counter() - t0
    n = len(toks) - 1
    return {"value": n / dt, "unit": "tokens/s", "cores": oracle_threads(), "kind": "oracle",
            "sample": (f"sequence 0 (KV history {L} positions, synthetic): {n} decode steps in {dt:.1f} s, "
                       f"fp64 numpy oracle with a KV cache"), "host": host_cpu()}


def kernel_summary(stats, workload, label="", streams=1):
    """Log per-class shares and rates; return the roofline object of the
    class with the largest timed share (None when nothing was timed). The
    GEMM views (every GEMM launch counted again by the kernel that ran it)
    are logged but never chosen and never summed."""
    from paper_2606_03014_amd.moa import VIEW_CLASSES
    real = {k: v for k, v in stats.items() if k not in VIEW_CLASSES}
    total_timed = sum(s["ms"] for s in real.values())
    if total_timed <= 0:
        return None
    for name, s in sorted(stats.items(), key=lambda kv: -kv[1]["ms"]):
        if s["launches"]:
            log(f"[bench] {label}{name:12s} {100 * s['ms'] / total_timed:5.1f}% of timed  "
                f"{s['ms'] / s['launches'] * 1e3:8.1f} us/launch  "
                f"{s['bytes'] / (s['ms'] * 1e-3) / 1e9:8.1f} GB/s  {s['flops'] / (s['ms'] * 1e-3) / 1e12:7.1f} TF/s")
    dom_name, dom = max(real.items(), key=lambda kv: kv[1]["ms"])
    roof = roof_of(dom)
    roof["traffic"] = measured_traffic(dom_name, workload, streams)
    roof["kernel"] = dom_name
    roof["launches_timed"] = dom["launches"]
    roof["us_per_launch"] = dom["ms"] / max(dom["launches"], 1) * 1e3
    roof["algorithmic_bytes_per_launch"] = dom["bytes"] / max(dom["launches"], 1)
    roof["algorithmic_flops_per_launch"] = dom["flops"] / max(dom["launches"], 1)
    roof["share_of_timed_kernel_time"] = dom["ms"] / total_timed
    return roof


def roof_of(s):
    """Achieved rate of one class against the roof its arithmetic intensity
    puts it under (HBM below the ridge point, bf16 MFMA above)."""
    if s["flops"] / max(s["bytes"], 1.0) > MFMA_BF16_PEAK / HBM_PEAK:
        achieved = s["flops"] / (s["ms"] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": MFMA_BF16_PEAK / 1e12, "unit": "TFLOP/s"}
    else:
        achieved = s["bytes"] / (s["ms"] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK / 1e9, "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    return roof


def design_bars(stats):
    """The classes the design targets are set on, each against its roof:
    decode attention and the small/medium-row GEMM kernel against 8 TB/s
    (target 70%), the large-row GEMM kernel against 2.5 PF/s of useful bf16
    flops (target 60%), and causal prefill attention against 2.5 PF/s."""
    out = {}
    for name, bound in (("attn", "hbm"), ("gemm_small_m", "hbm"), ("gemm_large_m", "mfma"),
                        ("prefill_attn", "mfma")):
        s = stats.get(name)
        if not s or not s["launches"] or s["ms"] <= 0:
            continue
        sec = s["ms"] * 1e-3
        frac = s["bytes"] / sec / HBM_PEAK if bound == "hbm" else s["flops"] / sec / MFMA_BF16_PEAK
        out[name] = {"bound": bound, "frac": round(frac, 4), "launches_timed": s["launches"],
                     "us_per_launch": round(s["ms"] / s["launches"] * 1e3, 2),
                     "target": 0.7 if bound == "hbm" else 0.6}
    return out


def class_rates(stats):
    """Per-class achieved rates against the HBM and MFMA peaks."""
    out = {}
    for name, s in stats.items():
        if s["launches"] and s["ms"] > 0:
            sec = s["ms"] * 1e-3
            out[name] = {"us_per_launch": round(s["ms"] / s["launches"] * 1e3, 2),
                         "hbm_frac": round(s["bytes"] / sec / HBM_PEAK, 4),
                         "mfma_frac": round(s["flops"] / sec / MFMA_BF16_PEAK, 4)}
    return out


class Progress:
    """Logs an engine-step progress line at most every ``every_s`` seconds."""

    def __init__(self, every_s=10.0):
        self.every_s = every_s
        self.reset()

    def reset(self):
        self.t0 = self.last = time.perf_counter()

    def __call__(self, info):
        now = time.perf_counter()
        if now - self.last >= self.every_s:
            self.last = now
            log(f"[bench]   engine step {info.step}: running {info.running}, pending {info.pending}, "
                f"{now - self.t0:.1f} s")


def load_models(eng, cfg, seed, n_models):
    """Generate and load each model's weights in turn (host copies freed as
    they go: an 8B-shape blob is 16 GB)."""
    from moa_inputs import generate_weights, pack_blob
    mids, first = [], None
    for m in range(n_models):
        t = time.perf_counter()
        w = generate_weights(cfg.model, cfg.dtype, seed, cfg.wid, m, threads=16)
        blob = pack_blob(w, cfg.model)
        mids.append(eng.load(blob))
        if m == 0:
            first = w
        del w, blob
        log(f"[bench] model {m} generated and loaded in {time.perf_counter() - t:.1f} s")
    return mids, first


def bench_feeder(args, cfg, eng, mids):
    """The workload's routed expert calls (and aggregator calls) through the
    feeder: each bench step is a block of args.block_steps engine steps of
    the one deterministic schedule (0: the whole batch, from submit to the
    last collect). Returns (tokens, seconds, config, extra, workload)."""
    import torch
    from moa_inputs import make_workload
    from paper_2606_03014_amd import Feeder
    wl = make_workload(cfg.name, args.seed, n_queries=args.queries)
    log(f"[bench] {cfg.name}: {wl.n_queries} queries, {len(wl.max_new)} expert calls, "
        f"{sum(len(p) for p in wl.prompts)} query prompt tokens")
    agg = mids[cfg.n_experts] if cfg.aggregator else -1
    prog = Progress()
    phase = {"prefill_steps": 0, "prefill_tokens": 0, "decode_rows": 0, "steps": 0, "models_rows": 0}

    def on_step(info):
        prog(info)
        phase["steps"] += 1
        phase["prefill_tokens"] += info.prefill_tokens
        phase["decode_rows"] += info.decode_rows
        phase["prefill_steps"] += 1 if info.prefill_tokens else 0

    gate = {}
    if args.gate_tau is not None:
        A = args.answer_options
        gate = dict(gate_tau=args.gate_tau, answer_of=lambda q, e, toks: int(toks[0]) % A)

    def new_feeder():
        return Feeder(eng, wl, mids[: cfg.n_experts], agg_model=agg, on_step=on_step, order=args.order,
                      window=args.window, **gate)

    block = args.block_steps if args.block_steps > 0 else None
    # one feeder across the blocks of the one schedule; for whole-batch steps
    # each bench step makes its own (a feeder submits its calls when made)
    feeder = new_feeder() if block else None

    def one_step():
        nonlocal feeder
        prog.reset()
        for k in phase:
            phase[k] = 0
        if block is None:                      # the whole batch, every bench step
            feeder = new_feeder()
        return feeder.advance(block)

    for i in range(args.warmup):
        t = time.perf_counter()
        n, tok = one_step()
        torch.cuda.synchronize()
        log(f"[bench] warmup {i}: {n} engine steps, {tok} tokens, {time.perf_counter() - t:.2f} s")
    first_timed = feeder.res.n_steps if block else 0
    eng.time_kernels(args.time_every, HBM_PEAK, MFMA_BF16_PEAK)
    torch.cuda.synchronize()
    tokens = steps = prefill_tokens = decode_rows = 0
    t0 = time.perf_counter()
    ns0 = time.monotonic_ns()
    for i in range(args.steps):
        t = time.perf_counter()
        n, tok = one_step()
        tokens += tok
        steps += n
        prefill_tokens += phase["prefill_tokens"]
        decode_rows += phase["decode_rows"]
        log(f"[bench] step {i}: {n} engine steps ({phase['prefill_steps']} with prefill), "
            f"{tok} tokens, {phase['prefill_tokens']} prompt tokens prefilled, "
            f"{phase['decode_rows'] / max(n, 1):.0f} decode rows per engine step, {time.perf_counter() - t:.2f} s (host)")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # the timed region on the monotonic clock a kernel trace is stamped with
    log(f"[bench] timed region monotonic_ns {ns0} {time.monotonic_ns()}")
    config = {"workload": cfg.name, "models": len(mids), "queries": wl.n_queries,
              "expert_calls": len(wl.max_new), "seed": args.seed, "parallelism": "single GPU",
              "order": args.order}
    if block:
        config["slice"] = (f"engine steps {first_timed}..{first_timed + steps - 1} of the workload's "
                           f"schedule (bench step = {block} engine steps; warm-up = steps 0..{first_timed - 1})")
        config["block_steps"] = block
        config["first_timed_engine_step"] = first_timed
    else:
        config["slice"] = "the whole batch per bench step"
    config["engine_steps_timed"] = steps
    config["generated_tokens_timed"] = tokens
    config["prefill_tokens_timed"] = prefill_tokens
    config["decode_rows_per_engine_step"] = round(decode_rows / max(steps, 1), 1)
    extra = {"prefill_tokens_per_s": prefill_tokens / wall}
    if block is None:
        extra["makespan_s"] = wall / args.steps
    if cfg.aggregator:
        r = feeder.res
        extra["aggregation"] = {"aggregator_calls_submitted": r.agg_calls, "skipped_by_gate": len(r.gated),
                                "gate_tau": args.gate_tau, "answer_options": args.answer_options if gate else None,
                                "answer": "first generated token mod answer_options" if gate else None}
    if args.window is not None:
        config["window"] = args.window
    return tokens, wall, config, extra, wl


def bench_straggler(args, cfg, eng, mids):
    """Long-reasoning straggler stress: a refill phase (every retired call is
    replaced at the next step) then a drain phase; both reported."""
    import torch
    from moa_inputs import make_straggler_workload
    from paper_2606_03014_amd import run_straggler
    sw = make_straggler_workload(args.seed, n_live=args.queries)
    prog = Progress()
    marks = {}

    def on_step(info):
        prog(info)
        rows = marks.setdefault("rows", [])
        rows.append(info.decode_rows)
        base = marks.setdefault("base", info.step)
        if info.step - base == sw.refill_steps:          # every refill-phase step has finished
            marks["t_refill_end"] = time.perf_counter()
            marks["tokens_refill"] = sum(rows[:-1])

    def one_step():
        prog.reset()
        marks.clear()
        return run_straggler(eng, sw, mids[0], on_step=on_step, after_collect=True)

    for i in range(args.warmup):
        t = time.perf_counter()
        tok, n, used = one_step()
        torch.cuda.synchronize()
        log(f"[bench] warmup {i}: {n} engine steps, {tok} tokens, {used} sequences, {time.perf_counter() - t:.2f} s")
    eng.time_kernels(args.time_every, HBM_PEAK, MFMA_BF16_PEAK)
    torch.cuda.synchronize()
    tokens = steps = 0
    phases = []
    ns0 = time.monotonic_ns()
    t0 = time.perf_counter()
    for i in range(args.steps):
        ts = time.perf_counter()
        tok, n, used = one_step()
        torch.cuda.synchronize()
        te = time.perf_counter()
        tokens += tok
        steps += n
        rows = marks["rows"]
        ta = marks["t_refill_end"] - ts
        ka = marks["tokens_refill"]
        phases.append({"refill": {"steps": sw.refill_steps, "tokens": ka, "s": ta, "tokens_per_s": ka / ta,
                                  "mean_live": ka / sw.refill_steps},
                       "drain": {"steps": n - sw.refill_steps, "tokens": tok - ka, "s": te - ts - ta,
                                 "tokens_per_s": (tok - ka) / (te - ts - ta),
                                 "mean_live": (tok - ka) / max(n - sw.refill_steps, 1)}})
        log(f"[bench] step {i}: {n} engine steps, {tok} tokens, {used} sequences; refill phase "
            f"{ka} tokens in {ta:.2f} s, drain {tok - ka} tokens in {te - ts - ta:.2f} s; rows "
            f"max {max(rows)} mean {sum(rows) / len(rows):.0f}")
    wall = time.perf_counter() - t0
    log(f"[bench] timed region monotonic_ns {ns0} {time.monotonic_ns()}")
    config = {"workload": cfg.name, "models": 1, "live_sequences": sw.n_live,
              "refill_steps": sw.refill_steps, "generated_tokens_per_step": tokens // args.steps,
              "engine_steps_per_step": steps // args.steps, "seed": args.seed,
              "kv_history": "device-filled synthetic K/V (hash of seed, layer, position)",
              "parallelism": "single GPU"}
    return tokens, wall, config, {"phases": phases}, None


def calibrate_placement(args, cfg):
    """Fit the session model T = t_step * O^max + t_token * N * Obar on this
    engine from three timed single-model sessions, then solve the placement
    ILP (Eq. 4-10) for the workload's experts on 1..8 workers (capacity 2),
    with the measured model-load time as l_m. Prints one JSON line."""
    import numpy as np
    import torch
    from moa_inputs import make_workload
    from paper_2606_03014_amd import Engine
    from paper_2606_03014_amd.placement import (ModelCost, fit_session_model, output_stats,
                                                session_time, solve_placement)
    from moa_inputs import generate_weights, pack_blob
    eng = Engine(cfg.model, cfg.dtype, cfg.engine, 1)
    blob = pack_blob(generate_weights(cfg.model, cfg.dtype, args.seed, cfg.wid, 0, threads=16), cfg.model)
    torch.cuda.synchronize()
    t = time.perf_counter()                    # l_m: host weights -> a ready expert on the GPU
    mids = [eng.load(blob)]
    torch.cuda.synchronize()
    load_s = time.perf_counter() - t
    del blob
    rng = np.random.default_rng([args.seed, 91])
    samples = []
    for n, G, P in ((8, 256, 128), (64, 128, 128), (16, 1024, 128)):
        prompts = [rng.integers(0, cfg.model.vocab, P).astype(np.int32) for _ in range(n)]
        torch.cuda.synchronize()
        t = time.perf_counter()
        for pr in prompts:
            eng.submit(pr, mids[0], G)
        while eng.step().step >= 0:
            pass
        eng.collect(-1)
        torch.cuda.synchronize()
        samples.append((n, float(G), float(G), time.perf_counter() - t))
        log(f"[bench] calibration session: {n} calls x {G} tokens in {samples[-1][3]:.2f} s")
    eng.close()
    t_step, t_token = fit_session_model(samples)
    wl = make_workload(cfg.name, args.seed, n_queries=args.queries)
    models = []
    for e in range(cfg.n_experts):
        lens = [G for (q, ee, G) in wl.expert_requests() if ee == e]
        om, ox = output_stats(lens)
        models.append(ModelCost(f"expert{e}", len(lens), load_s, session_time(len(lens), om, ox, t_step, t_token)))
    plans = {}
    for N in range(1, 9):
        try:
            p = solve_placement(models, N, 2)
            plans[N] = {"makespan_s": p.makespan, "Y": p.Y.tolist(), "X": p.X.tolist(), "replica_caps": p.caps}
        except ValueError as err:
            plans[N] = {"infeasible": str(err)}
    print(json.dumps({"calibration": {"t_step_s": t_step, "t_token_s": t_token, "load_s": load_s,
                                      "sessions": samples},
                      "experts": [{"name": m.name, "N_m": m.n_prompts, "T_hat_s": m.T_hat, "tau_s": m.tau}
                                  for m in models],
                      "placements_K2": plans, "workload": cfg.name}), flush=True)


def plan_cost(cfg):
    """Per-unit costs of the schedule cost model for cfg's model shape."""
    import numpy as np
    from moa_inputs.weights import tensor_shapes
    g = cfg.model
    esz = 2 if cfg.dtype == "bf16" else 4
    n_params = sum(int(np.prod(sh)) for _, sh in tensor_shapes(g))
    return {"streamed": (n_params - g.vocab * g.d_model) * esz,          # every matrix but the embedding
            "kv_per_ctx": 2 * g.n_layers * g.n_kv_heads * g.head_dim * esz,
            "lin_flops": 2.0 * (n_params - g.vocab * g.d_model),           # per prefill token
            "pair_flops": 4.0 * g.n_heads * g.head_dim * g.n_layers,       # per causal (q, k) pair
            "blob_bytes": n_params * esz}


def price_plan(eng, res, cost, nm):
    """Model time of a schedule planned by a plan-only engine (res: the
    feeder's FeedResult). Per step: the weights of every model with a row in
    the step and the K/V of every decode row's context at STUDY_BW, prefill
    tokens at the large-M GEMM rate and causal prefill pairs at the
    prefill-attention rate. Returns (model seconds, steps, generated tokens,
    mean models per step)."""
    import numpy as np
    S = res.n_steps
    active = np.zeros((S + 1, nm), bool)
    ctx = np.zeros(S + 1)
    pre = np.zeros(S + 1)
    pairs = 0.0
    gen = 0
    for (q, m), rid in res.rid_of.items():
        info = eng.request(rid)
        ch = eng.chunks(rid)
        for s, a, b in ch:
            pre[s] += b
            pairs += b * a + b * (b + 1) / 2
            active[s, m] = True
        d0 = max(s for s, a, b in ch) + 1       # decode steps d0..finish, at positions P..P+G-2
        d1 = info.finish_step
        if d1 >= d0:
            active[d0:d1 + 1, m] = True
            ctx[d0:d1 + 1] += info.prompt_len + 1 + np.arange(d1 - d0 + 1)
        gen += info.max_new_tokens
    t = (active.sum(axis=1) * cost["streamed"] + ctx * cost["kv_per_ctx"]) / STUDY_BW + pre * cost["lin_flops"] / STUDY_LIN
    model_s = float(t.sum() + pairs * cost["pair_flops"] / STUDY_ATTN)
    return model_s, S, gen, float(active[:S].sum(axis=1).mean())


def plan_only_run(cfg, wl, consts, order="first-seen", window=None, gate=None):
    """The workload's schedule on a plan-only engine (no GPU); gate: a dict
    of Feeder gate arguments. Returns price_plan's tuple."""
    import numpy as np
    from paper_2606_03014_amd import Engine, run_feeder
    nm = cfg.n_experts + (1 if cfg.aggregator else 0)
    cost = plan_cost(cfg)
    eng = Engine(cfg.model, cfg.dtype, consts, nm, plan_only=True)
    blob = np.zeros(cost["blob_bytes"], np.uint8)
    for _ in range(nm):
        eng.load(blob)
    r = run_feeder(eng, wl, list(range(cfg.n_experts)), agg_model=cfg.n_experts if cfg.aggregator else -1,
                   order=order, window=window, **(gate or {}))
    out = price_plan(eng, r, cost, nm)
    eng.close()
    return out + (r,)


def schedule_study(args, cfg):
    """Plan-only schedules of the workload under the feeder's policies
    (submission order x submission window x prefill budget), with no GPU: the
    engine's own scheduler plans every step, and a per-step cost model prices
    it (price_plan). Prints one JSON line."""
    import dataclasses
    from moa_inputs import make_workload
    wl = make_workload(cfg.name, args.seed, n_queries=args.queries)
    rows_out = []
    for order in ("first-seen", "longest-first"):
        for window in (None, 256, 64, 16):
            for budget in (4096, 16384, 32768):
                consts = dataclasses.replace(cfg.engine, max_prefill_tokens=budget)
                model_s, S, gen, act, _ = plan_only_run(cfg, wl, consts, order, window)
                rows_out.append({"order": order, "window": window, "prefill_budget": budget, "steps": S,
                                 "model_s": float(f"{model_s:.4g}"), "model_tokens_per_s": round(gen / model_s),
                                 "mean_active_models": round(act, 3)})
                log(f"[bench] {order:13s} window {str(window):5s} budget {budget:6d}: {S} steps, "
                    f"model {model_s:.1f} s")
    print(json.dumps({"schedule_study": rows_out, "workload": cfg.name, "queries": wl.n_queries,
                      "cost_model": {"stream_Bps": STUDY_BW, "prefill_linear_flops": STUDY_LIN,
                                     "prefill_attention_flops": STUDY_ATTN}}), flush=True)


# the feeder policies of the study: submission order, and the synthetic
# answer space of the confidence gate (None: no gate)
POLICIES = {"first-seen": ("first-seen", None), "longest-first": ("longest-first", None),
            "gate-A2": ("first-seen", 2), "gate-A8": ("first-seen", 8)}


def policy_study(args, cfg, eng, mids):
    """The feeder's policies measured on the GPU (Section "MOSAIC: Multi-Model
    Scheduling" for the order, Eq. 11 / Algorithm 1 for the gate): the same
    query slice run to completion under first-seen and longest-first
    submission, and under first-seen with the confidence gate at tau = 1
    for two synthetic answer spaces (an expert's answer is its first token
    mod A, so about 1/A of the two-expert queries agree). Each measured
    makespan stands beside the plan-only cost model's for the same schedule
    (for a gated run, planned with the GPU run's own answers). Prints one
    JSON line."""
    import torch
    from moa_inputs import make_workload
    from paper_2606_03014_amd import Feeder
    wl = make_workload(cfg.name, args.seed, n_queries=args.queries or 256)
    agg = mids[cfg.n_experts] if cfg.aggregator else -1
    rows = []
    for name, (order, A) in POLICIES.items():
        if args.policies and name not in args.policies.split(","):
            continue
        gate = {}
        if A:
            gate = dict(gate_tau=1, answer_of=lambda q, e, toks, A=A: int(toks[0]) % A)
        prog = Progress()
        f = Feeder(eng, wl, mids[: cfg.n_experts], agg_model=agg, on_step=prog, order=order, **gate)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        f.advance(None)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        r = f.res
        pgate = {}
        if A:
            ans = {(q, e): int(r.outputs[(q, mids[e])][0]) % A for q in range(wl.n_queries) for e in wl.experts[q]}
            pgate = dict(gate_tau=1, answer_of=lambda q, e, toks, ans=ans: ans[(q, e)])
        model_s, S, gen, act, pr = plan_only_run(cfg, wl, cfg.engine, order, None, pgate)
        assert S == r.n_steps and pr.agg_calls == r.agg_calls, "plan-only and GPU schedules differ"
        rows.append({"policy": name, "order": order, "gate": {"tau": 1, "answer_options": A} if A else None,
                     "makespan_s": wall, "engine_steps": r.n_steps, "generated_tokens": r.tokens,
                     "tokens_per_s": r.tokens / wall, "aggregator_calls": r.agg_calls,
                     "gated_queries": len(r.gated), "model_makespan_s": model_s,
                     "model_over_measured": model_s / wall})
        log(f"[bench] policy {order} gate A={A}: {r.n_steps} steps, {r.tokens} tokens, {wall:.1f} s "
            f"(model {model_s:.1f} s), aggregator calls {r.agg_calls}, gated {len(r.gated)}")
    print(json.dumps({"policy_study": rows, "workload": cfg.name, "queries": wl.n_queries, "seed": args.seed,
                      "model_streams": 1 if eng.cfg.flags & 2 else 2,
                      "cost_model": {"stream_Bps": STUDY_BW, "prefill_linear_flops": STUDY_LIN,
                                     "prefill_attention_flops": STUDY_ATTN}}), flush=True)


def main():
    t_start = time.perf_counter()
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20, help="timed bench steps")
    ap.add_argument("--warmup", type=int, default=5, help="untimed bench steps before them")
    ap.add_argument("--workload", default="moa-3+1x8b-bf16")
    ap.add_argument("--block-steps", type=int, default=128,
                    help="engine steps per bench step (0: the whole batch per bench step)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--queries", type=int, default=None, help="fewer queries (quick runs only)")
    ap.add_argument("--time-every", type=int, default=8, help="time the kernels of 1 step in N")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--gate-tau", type=float, default=None,
                    help="adaptive-aggregation gate threshold (skip the aggregator when the experts' vote share >= tau)")
    ap.add_argument("--answer-options", type=int, default=4,
                    help="synthetic answer space of the gate: an expert's answer is its first token mod this")
    ap.add_argument("--order", default="first-seen", choices=["first-seen", "longest-first"],
                    help="submission order of the expert calls")
    ap.add_argument("--calibrate-placement", action="store_true",
                    help="fit the per-model session cost on this engine and solve the placement ILP for 1..8 workers")
    ap.add_argument("--policy-study", action="store_true",
                    help="measure the feeder's policies (order, confidence gate) to completion on a query slice "
                         "(default 256 queries) beside the plan-only cost model")
    ap.add_argument("--policies", default=None,
                    help="comma-separated subset of the policy study's policies (" + ", ".join(POLICIES) + ")")
    ap.add_argument("--schedule-study", action="store_true",
                    help="plan-only schedules under each submission order, window and prefill budget, "
                         "priced by a per-step cost model (no GPU)")
    ap.add_argument("--window", type=int, default=None,
                    help="submission window of the feeder (default: every expert call up front)")
    ap.add_argument("--streams", type=int, default=None, choices=[1, 2],
                    help="model streams of a several-model bf16 batch: 1 runs every kernel on the "
                         "caller's stream, 2 splits each step's models over two overlapping streams "
                         f"(default: {DEFAULT_STREAMS})")
    ap.add_argument("--one-stream", action="store_true", help="same as --streams 1")
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
    if args.schedule_study:
        from moa_inputs import CONFIGS
        schedule_study(args, CONFIGS[args.workload])
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the engine has no "
              "multi-GPU path: it runs every model of the batch on one MI355X.", file=sys.stderr)
        sys.exit(2)

    import torch
    from moa_inputs import CONFIGS
    from paper_2606_03014_amd import Engine

    cfg = CONFIGS[args.workload]
    if args.calibrate_placement:
        calibrate_placement(args, cfg)
        return
    straggler = cfg.name.startswith("straggler")
    n_models = cfg.n_experts + (1 if cfg.aggregator else 0)
    want = 1 if args.one_stream else (args.streams or DEFAULT_STREAMS)
    eng = Engine(cfg.model, cfg.dtype, cfg.engine, n_models, one_stream=want == 1)
    streams = 1 if (want == 1 or n_models < 2 or cfg.dtype != "bf16") else 2
    log(f"[bench] {cfg.name}: {n_models} model(s); arena {eng.arena_bytes / 2**30:.1f} GiB")
    mids, weights0 = load_models(eng, cfg, args.seed, n_models)
    read_bps, mfma_fps = eng.measure_peaks()
    log(f"[bench] measured peaks: HBM read {read_bps / 1e12:.2f} TB/s, bf16 32x32x16 MFMA {mfma_fps / 1e15:.2f} PFLOP/s")
    if args.policy_study:
        policy_study(args, cfg, eng, mids)
        eng.close()
        return
    run = bench_straggler if straggler else bench_feeder
    tokens, wall, config, extra, wl = run(args, cfg, eng, mids)
    stats = eng.kernel_stats()
    roof = kernel_summary(stats, cfg.name, streams=1)
    config["model_streams"] = streams
    if roof is not None and streams > 1:
        roof["timed_steps"] = ("one engine step in --time-every runs every kernel on one stream and is the "
                               "one timed; the others split their models over two streams")
    from paper_2606_03014_amd.moa import VIEW_CLASSES
    real = {k: v for k, v in stats.items() if k not in VIEW_CLASSES}
    run_roof_ms = sum(s["roof_ms_all"] for s in real.values())
    # kernel time of every launch, estimated from the timed sample of each
    # class in proportion to its bytes (an untimed two-stream launch carries
    # about half the step's models)
    busy_ms = sum(s["ms"] * (s["bytes_all"] / s["bytes"] if s["bytes"] > 0 else s["launches_all"] / s["launches"])
                  for s in real.values() if s["launches"])

    out = {
        "metric": METRIC,
        "value": tokens / wall,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall * 1e3 / args.steps,
        "timed_wall_s": wall,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": config,
        "roofline": roof,
        "bars": design_bars(stats),
        "run_roofline": {"roof_ms": run_roof_ms / args.steps, "measured_ms": wall * 1e3 / args.steps,
                         "frac": run_roof_ms / (wall * 1e3),
                         "kernel_ms_est": busy_ms / args.steps, "gpu_busy_frac": busy_ms / (wall * 1e3)},
        "kernel_classes": class_rates(stats),
        # the same roofline against what this GPU sustains (per kernel class:
        # max(bytes / measured read bandwidth, useful flops / measured MFMA rate))
        "measured_peaks": {"hbm_read_GBps": read_bps / 1e9, "mfma_bf16_TFLOPs": mfma_fps / 1e12},
        "run_roofline_measured_peaks": {
            "roof_ms": sum(max(s["bytes_all"] / read_bps, s["flops_all"] / mfma_fps) for s in real.values()) * 1e3 / args.steps,
            "frac": sum(max(s["bytes_all"] / read_bps, s["flops_all"] / mfma_fps) for s in real.values()) / wall},
    }
    out.update(extra)
    eng.close()
    del eng
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        if straggler:
            out["cpu_baseline"] = cpu_baseline_history(cfg, args.seed, weights0)
        else:
            out["cpu_baseline"] = cpu_baseline(cfg, wl, weights0)
    log(f"[bench] whole run {time.perf_counter() - t_start:.1f} s (models, peaks, warm-up, timed steps, CPU leg)")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
