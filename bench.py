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
# per-step cost model of the schedule study: the decode streaming rate and
# the useful prefill rates this engine reaches on 8B shapes (large-M GEMM,
# causal prefill attention)
STUDY_BW = 5.0e12
STUDY_LIN = 4.7e14
STUDY_ATTN = 3.2e14


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def measured_traffic(kernel, workload, streams=1):
    """HBM bytes per launch of ``kernel`` on ``workload`` from the committed
    rocprofv3 counter summaries, or None when none exists, the kernel source
    changed since, or the counters were taken with another number of model
    streams (which changes what one launch carries)."""
    import glob
    import hashlib
    src = os.path.join(ROOT, "paper_2606_03014_amd", "csrc", "kernels.hip")
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    for path in glob.glob(os.path.join(ROOT, "profiles", "*traffic*.md")):
        for line in open(path):
            line = line.strip()
            if line.startswith("{") and '"traffic_bytes_per_launch"' in line:
                rec = json.loads(line)
                if (rec.get("kernel") == kernel and rec.get("kernels_source_sha256_16") == sha
                        and rec.get("workload") == workload and rec.get("model_streams", 1) == streams):
                    return rec["traffic_bytes_per_launch"]
    return None


def oracle_threads():
    try:
        from threadpoolctl import threadpool_info
        return int(max([i.get("num_threads", 1) for i in threadpool_info()] or [1]))
    except Exception:
        return os.cpu_count()


def cpu_baseline(cfg, wl, weights0, budget_s):
    """The oracle, as it stands, on the workload's first call of model 0 (an
    expert call, or the first aggregator call when there are no experts):
    prefill its prompt in chunks of 256 positions (stopping after half the
    budget if the prompt is that long), then decode until the budget runs out."""
    from oracle import transformer as T
    om = T.OracleModel(cfg.model, weights0)
    for name in weights0:                       # fp64 upcast of the weights: setup, not timed
        om.W(name)
    reqs = [r for r in wl.expert_requests() if r[1] == 0]
    q, G = (reqs[0][0], reqs[0][2]) if reqs else (0, wl.agg_max_new)
    prompt = wl.prompts[q]
    kv = T.ContiguousKV(cfg.model.n_layers, cfg.model.n_kv_heads, cfg.model.head_dim)
    t0 = time.perf_counter()
    pos = 0
    while pos < len(prompt):
        c = min(256, len(prompt) - pos)
        lg = T.forward_chunk(om, prompt[pos:pos + c], pos, kv, bf16_kv=True, want="last")[-1]
        pos += c
        if time.perf_counter() - t0 > budget_s / 2:
            break
    t_pre = time.perf_counter() - t0
    toks = [T.argmax_lowest(lg)]
    while len(toks) < G and time.perf_counter() - t0 < budget_s:
        lg = T.forward_chunk(om, [toks[-1]], pos + len(toks) - 1, kv, bf16_kv=True)[-1]
        toks.append(T.argmax_lowest(lg))
    dt = time.perf_counter() - t0
    return {"value": len(toks) / dt, "unit": "tokens/s", "cores": oracle_threads(), "kind": "oracle",
            "sample": (f"model-0 call of query {q}: prefill of {pos} of its {len(prompt)} prompt tokens "
                       f"({t_pre:.1f} s) plus {len(toks) - 1} decode steps ({len(toks)} generated tokens, "
                       f"{dt:.1f} s, fp64 numpy oracle with a KV cache)")}


def cpu_baseline_history(cfg, seed, weights0, budget_s):
    """The oracle on the straggler workload's first sequence: its synthetic
    K/V history (bf16-rounded) in a contiguous cache, then decode steps until
    the budget or its remaining length runs out."""
    import numpy as np
    from moa_inputs import make_straggler_workload, synthetic_kv, f32_to_bf16_bits
    from moa_inputs.weights import bf16_bits_to_f32
    from oracle import transformer as T
    m = cfg.model
    om = T.OracleModel(m, weights0)
    for name in weights0:
        om.W(name)
    L, tok, R = make_straggler_workload(seed).sequence(0)
    hist = bf16_bits_to_f32(f32_to_bf16_bits(synthetic_kv(seed, 0, m.n_layers, L, m.n_kv_heads, m.head_dim)))
    kv = T.ContiguousKV(m.n_layers, m.n_kv_heads, m.head_dim)
    for l in range(m.n_layers):
        kv.K[l] = hist[l, 0].astype(np.float64)
        kv.V[l] = hist[l, 1].astype(np.float64)
    del hist
    t0 = time.perf_counter()
    toks = [tok]
    while len(toks) <= R and time.perf_counter() - t0 < budget_s:
        lg = T.forward_chunk(om, [toks[-1]], L + len(toks) - 1, kv, bf16_kv=True)[-1]
        toks.append(T.argmax_lowest(lg))
    dt = time.perf_counter() - t0
    n = len(toks) - 1
    return {"value": n / dt, "unit": "tokens/s", "cores": oracle_threads(), "kind": "oracle",
            "sample": (f"sequence 0 (KV history {L} positions, synthetic): {n} decode steps in {dt:.1f} s, "
                       f"fp64 numpy oracle with a KV cache")}


def kernel_summary(stats, workload, label="", streams=1):
    """Log per-class shares and rates; return the roofline object of the
    class with the largest timed share (None when nothing was timed)."""
    total_timed = sum(s["ms"] for s in stats.values())
    if total_timed <= 0:
        return None
    for name, s in sorted(stats.items(), key=lambda kv: -kv[1]["ms"]):
        if s["launches"]:
            log(f"[bench] {label}{name:12s} {100 * s['ms'] / total_timed:5.1f}% of timed  "
                f"{s['ms'] / s['launches'] * 1e3:8.1f} us/launch  "
                f"{s['bytes'] / (s['ms'] * 1e-3) / 1e9:8.1f} GB/s  {s['flops'] / (s['ms'] * 1e-3) / 1e12:7.1f} TF/s")
    dom_name, dom = max(stats.items(), key=lambda kv: kv[1]["ms"])
    intensity = dom["flops"] / max(dom["bytes"], 1.0)
    if intensity > MFMA_BF16_PEAK / HBM_PEAK:
        achieved = dom["flops"] / (dom["ms"] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": MFMA_BF16_PEAK / 1e12, "unit": "TFLOP/s"}
    else:
        achieved = dom["bytes"] / (dom["ms"] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK / 1e9, "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = measured_traffic(dom_name, workload, streams)
    roof["kernel"] = dom_name
    roof["launches_timed"] = dom["launches"]
    roof["us_per_launch"] = dom["ms"] / max(dom["launches"], 1) * 1e3
    roof["algorithmic_bytes_per_launch"] = dom["bytes"] / max(dom["launches"], 1)
    roof["algorithmic_flops_per_launch"] = dom["flops"] / max(dom["launches"], 1)
    return roof


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
    """Every routed expert call (and aggregator call) of the workload, run to
    completion through the feeder; returns (tokens, seconds, extra)."""
    import torch
    from moa_inputs import make_workload
    from paper_2606_03014_amd import run_feeder
    wl = make_workload(cfg.name, args.seed, n_queries=args.queries)
    log(f"[bench] {cfg.name}: {wl.n_queries} queries, {len(wl.max_new)} expert calls, "
        f"{sum(len(p) for p in wl.prompts)} query prompt tokens")
    agg = mids[cfg.n_experts] if cfg.aggregator else -1
    prog = Progress()
    phase = {"prefill_steps": 0, "prefill_tokens": 0, "decode_rows": 0, "steps": 0}

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

    def one_step():
        prog.reset()
        for k in phase:
            phase[k] = 0
        return run_feeder(eng, wl, mids[: cfg.n_experts], agg_model=agg, on_step=on_step, order=args.order,
                          window=args.window, **gate)

    for i in range(args.warmup):
        t = time.perf_counter()
        r = one_step()
        torch.cuda.synchronize()
        log(f"[bench] warmup {i}: {r.n_steps} engine steps, {r.tokens} tokens, {time.perf_counter() - t:.2f} s")
    eng.time_kernels(args.time_every, HBM_PEAK, MFMA_BF16_PEAK)
    torch.cuda.synchronize()
    tokens = steps = prefill_tokens = 0
    t0 = time.perf_counter()
    r = None
    for i in range(args.steps):
        r = one_step()
        tokens += r.tokens
        steps += r.n_steps
        prefill_tokens += phase["prefill_tokens"]
        log(f"[bench] step {i}: {r.n_steps} engine steps ({phase['prefill_steps']} with prefill), "
            f"{r.tokens} tokens, {phase['prefill_tokens']} prompt tokens prefilled")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    config = {"workload": cfg.name, "models": len(mids), "queries": wl.n_queries,
              "expert_calls": len(wl.max_new), "generated_tokens_per_step": tokens // args.steps,
              "prefill_tokens_per_step": prefill_tokens // args.steps,
              "engine_steps_per_step": steps // args.steps, "seed": args.seed,
              "parallelism": "single GPU"}
    extra = {"prefill_tokens_per_s": prefill_tokens / wall, "makespan_s": wall / args.steps}
    if cfg.aggregator:
        extra["aggregation"] = {"aggregator_calls": r.agg_calls, "skipped_by_gate": len(r.gated),
                                "gate_tau": args.gate_tau, "answer_options": args.answer_options if gate else None,
                                "answer": "first generated token mod answer_options" if gate else None}
    config["order"] = args.order
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


def schedule_study(args, cfg):
    """Plan-only schedules of the workload under the feeder's policies
    (submission order x submission window x prefill budget), with no GPU: the
    engine's own scheduler plans every step, and a per-step cost model prices
    it. Per step: the weights of every model with a row in the step at
    STUDY_BW, the K/V of every decode row's context at STUDY_BW, prefill
    tokens at the measured large-M GEMM rate and causal prefill pairs at the
    measured prefill-attention rate. Prints one JSON line."""
    import dataclasses
    import numpy as np
    from moa_inputs import make_workload
    from moa_inputs.weights import tensor_shapes
    from paper_2606_03014_amd import Engine, run_feeder
    g = cfg.model
    esz = 2 if cfg.dtype == "bf16" else 4
    n_params = sum(int(np.prod(sh)) for _, sh in tensor_shapes(g))
    streamed = (n_params - g.vocab * g.d_model) * esz           # every matrix but the embedding
    kv_per_ctx = 2 * g.n_layers * g.n_kv_heads * g.head_dim * esz
    lin_flops = 2.0 * (n_params - g.vocab * g.d_model)           # per prefill token
    pair_flops = 4.0 * g.n_heads * g.head_dim * g.n_layers       # per causal (q, k) pair
    wl = make_workload(cfg.name, args.seed, n_queries=args.queries)
    nm = cfg.n_experts + (1 if cfg.aggregator else 0)
    blob = np.zeros(n_params * esz, np.uint8)
    rows_out = []
    for order in ("first-seen", "longest-first"):
        for window in (None, 256, 64, 16):
            for budget in (4096, 16384, 32768):
                consts = dataclasses.replace(cfg.engine, max_prefill_tokens=budget)
                eng = Engine(g, cfg.dtype, consts, nm, plan_only=True)
                for _ in range(nm):
                    eng.load(blob)
                r = run_feeder(eng, wl, list(range(cfg.n_experts)), agg_model=cfg.n_experts if cfg.aggregator else -1,
                               order=order, window=window)
                S = r.n_steps
                active = np.zeros((S + 1, nm), bool)
                ctx = np.zeros(S + 1)
                pre = np.zeros(S + 1)
                pairs = 0.0
                gen = 0
                for (q, m), rid in r.rid_of.items():
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
                t = (active.sum(axis=1) * streamed + ctx * kv_per_ctx) / STUDY_BW + pre * lin_flops / STUDY_LIN
                model_s = float(t.sum() + pairs * pair_flops / STUDY_ATTN)
                eng.close()
                rows_out.append({"order": order, "window": window, "prefill_budget": budget, "steps": S,
                                 "model_s": float(f"{model_s:.4g}"), "model_tokens_per_s": round(gen / model_s),
                                 "mean_active_models": round(float(active[:S].sum(axis=1).mean()), 3)})
                log(f"[bench] {order:13s} window {str(window):5s} budget {budget:6d}: {S} steps, "
                    f"model {model_s:.1f} s")
    print(json.dumps({"schedule_study": rows_out, "workload": cfg.name, "queries": wl.n_queries,
                      "cost_model": {"stream_Bps": STUDY_BW, "prefill_linear_flops": STUDY_LIN,
                                     "prefill_attention_flops": STUDY_ATTN}}), flush=True)


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
    ap.add_argument("--gate-tau", type=float, default=None,
                    help="adaptive-aggregation gate threshold (skip the aggregator when the experts' vote share >= tau)")
    ap.add_argument("--answer-options", type=int, default=4,
                    help="synthetic answer space of the gate: an expert's answer is its first token mod this")
    ap.add_argument("--order", default="first-seen", choices=["first-seen", "longest-first"],
                    help="submission order of the expert calls")
    ap.add_argument("--calibrate-placement", action="store_true",
                    help="fit the per-model session cost on this engine and solve the placement ILP for 1..8 workers")
    ap.add_argument("--schedule-study", action="store_true",
                    help="plan-only schedules under each submission order, window and prefill budget, "
                         "priced by a per-step cost model (no GPU)")
    ap.add_argument("--window", type=int, default=None,
                    help="submission window of the feeder (default: every expert call up front)")
    ap.add_argument("--one-stream", action="store_true",
                    help="run every kernel on one stream (default: a several-model batch splits its "
                         "models over two overlapping streams)")
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
    eng = Engine(cfg.model, cfg.dtype, cfg.engine, n_models, one_stream=args.one_stream)
    streams = 1 if (args.one_stream or n_models < 2 or cfg.dtype != "bf16") else 2
    log(f"[bench] {cfg.name}: {n_models} model(s); arena {eng.arena_bytes / 2**30:.1f} GiB")
    mids, weights0 = load_models(eng, cfg, args.seed, n_models)
    read_bps, mfma_fps = eng.measure_peaks()
    log(f"[bench] measured peaks: HBM read {read_bps / 1e12:.2f} TB/s, bf16 32x32x16 MFMA {mfma_fps / 1e15:.2f} PFLOP/s")
    run = bench_straggler if straggler else bench_feeder
    tokens, wall, config, extra, wl = run(args, cfg, eng, mids)
    stats = eng.kernel_stats()
    roof = kernel_summary(stats, cfg.name, streams=streams)
    config["model_streams"] = streams
    if roof is not None and streams > 1:
        roof["overlap"] = ("launch durations from two model streams whose kernels run concurrently: "
                           "each launch carries half the batch's models and shares the GPU with the "
                           "other stream's launches (--one-stream times them alone)")
    run_roof_ms = sum(s["roof_ms_all"] for s in stats.values())
    # kernel time of every launch, estimated from the timed sample of each class
    busy_ms = sum(s["ms"] / s["launches"] * s["launches_all"] for s in stats.values() if s["launches"])

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
        "config": config,
        "roofline": roof,
        "run_roofline": {"roof_ms": run_roof_ms / args.steps, "measured_ms": wall * 1e3 / args.steps,
                         "frac": run_roof_ms / (wall * 1e3),
                         "kernel_ms_est": busy_ms / args.steps, "gpu_busy_frac": busy_ms / (wall * 1e3)},
        "kernel_classes": class_rates(stats),
        # the same roofline against what this GPU sustains (per kernel class:
        # max(bytes / measured read bandwidth, useful flops / measured MFMA rate))
        "measured_peaks": {"hbm_read_GBps": read_bps / 1e9, "mfma_bf16_TFLOPs": mfma_fps / 1e12},
        "run_roofline_measured_peaks": {
            "roof_ms": sum(max(s["bytes_all"] / read_bps, s["flops_all"] / mfma_fps) for s in stats.values()) * 1e3 / args.steps,
            "frac": sum(max(s["bytes_all"] / read_bps, s["flops_all"] / mfma_fps) for s in stats.values()) / wall},
    }
    out.update(extra)
    eng.close()
    del eng
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        if straggler:
            out["cpu_baseline"] = cpu_baseline_history(cfg, args.seed, weights0, args.cpu_budget)
        else:
            out["cpu_baseline"] = cpu_baseline(cfg, wl, weights0, args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
