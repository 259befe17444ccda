"""bench.py's reading of committed counter records (CPU only)."""
import importlib.util
import json
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_traffic_records_match_source_workload_and_streams(tmp_path):
    """A traffic record applies only to the kernel source it was taken on,
    its workload and its number of model streams (which set what one launch
    carries); records without a stream count are one-stream records."""
    bench = _bench()
    src = tmp_path / "paper_2606_03014_amd" / "csrc"
    src.mkdir(parents=True)
    (src / "kernels.hip").write_text("// kernels\nint k;  // one\n/* block\n comment */\n")
    sha = bench.kernel_code_digest(str(src / "kernels.hip"))
    prof = tmp_path / "profiles"
    prof.mkdir()
    recs = [
        {"kernel": "gemm_gateup", "kernels_code_sha256_16": sha, "workload": "w", "model_streams": 2,
         "traffic_bytes_per_launch": 2.0},
        {"kernel": "gemm_gateup", "kernels_code_sha256_16": sha, "workload": "w",
         "traffic_bytes_per_launch": 1.0},
        {"kernel": "attn", "kernels_code_sha256_16": "0" * 16, "workload": "w", "model_streams": 1,
         "traffic_bytes_per_launch": 3.0},
    ]
    (prof / "traffic_w.md").write_text("# t\n\n```\n" + "\n".join(json.dumps(r) for r in recs) + "\n```\n")
    (prof / "kernels_w.md").write_text(json.dumps(dict(recs[0], traffic_bytes_per_launch=9.0)) + "\n")
    bench.ROOT = str(tmp_path)
    assert bench.measured_traffic("gemm_gateup", "w", 2) == 2.0
    assert bench.measured_traffic("gemm_gateup", "w", 1) == 1.0
    assert bench.measured_traffic("gemm_gateup", "other", 2) is None
    assert bench.measured_traffic("attn", "w", 1) is None          # another kernel source
    assert bench.measured_traffic("gemm_down", "w", 1) is None
    # comments and blank lines do not change the digest; code does
    (src / "kernels.hip").write_text("// other words\n\nint k;   /* note */\n")
    assert bench.measured_traffic("gemm_gateup", "w", 1) == 1.0
    (src / "kernels.hip").write_text("int k2;\n")
    assert bench.measured_traffic("gemm_gateup", "w", 1) is None


def test_bench_refuses_more_than_one_gpu():
    """The engine runs on one GPU: bench.py --gpus 2 exits with status 2 and
    says so, before touching a GPU."""
    import subprocess
    import sys
    out = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert out.returncode == 2
    assert "one GPU only" in out.stderr and out.stdout == ""


def _dry_engine(cfg, n_models):
    import numpy as np
    from paper_2606_03014_amd import Engine
    g = cfg.model
    qd, kd = g.n_heads * g.head_dim, g.n_kv_heads * g.head_dim
    n = 2 * g.vocab * g.d_model + g.d_model + g.n_layers * (
        2 * g.d_model + (qd + 2 * kd) * g.d_model + g.d_model * qd + 3 * g.ffn_dim * g.d_model)
    eng = Engine(g, cfg.dtype, cfg.engine, n_models, plan_only=True)
    mids = [eng.load(np.zeros(n * (2 if cfg.dtype == "bf16" else 4), dtype=np.uint8)) for _ in range(n_models)]
    return eng, mids


def test_whole_batch_bench_steps_each_run_the_batch_once(monkeypatch):
    """--block-steps 0: every bench step (warm-up and timed) runs the whole
    batch once through a feeder of its own, on a dry-run engine: each step
    generates exactly the workload's tokens (no step sees another's calls)."""
    import argparse
    import torch
    from moa_inputs import CONFIGS, make_workload
    bench = _bench()
    monkeypatch.setattr(torch.cuda, "synchronize", lambda *a, **k: None)
    cfg = CONFIGS["tiny-moa-fp32"]
    n_models = cfg.n_experts + (1 if cfg.aggregator else 0)
    eng, mids = _dry_engine(cfg, n_models)
    try:
        args = argparse.Namespace(seed=0, queries=None, gate_tau=None, answer_options=4, order="first-seen",
                                  window=None, block_steps=0, warmup=2, steps=2, time_every=8)
        tokens, wall, config, extra, wl = bench.bench_feeder(args, cfg, eng, mids)
    finally:
        eng.close()
    wl = make_workload(cfg.name, 0)
    per_batch = wl.total_expert_tokens() + wl.n_queries * wl.agg_max_new
    assert tokens == 2 * per_batch
    assert config["slice"] == "the whole batch per bench step"
    assert extra["aggregation"]["aggregator_calls_submitted"] == wl.n_queries


def test_bench_line_keeps_its_contract(monkeypatch, capsys):
    """The one JSON line bench.py prints, end to end on the CPU: a plan-only
    engine runs the tiny fp32 workload's schedule (the GPU-only calls, peak
    probes and kernel timing, are stubbed with fixed figures), and the CPU
    oracle leg runs for real. Every key the line promises is there, with the
    right type, and the roofline object is the dominant class's."""
    import sys
    import torch
    import paper_2606_03014_amd as pkg
    from paper_2606_03014_amd.moa import KERNEL_CLASSES
    bench = _bench()
    real_engine = pkg.Engine

    def plan_only_engine(shape, dtype, consts, max_models, **kw):
        kw.pop("plan_only", None)
        eng = real_engine(shape, dtype, consts, max_models, plan_only=True, **kw)
        eng.measure_peaks = lambda: (6.3e12, 2.0e15)
        # attention dominates the timed kernel time: 4 launches of 2 GB in 1 ms each
        stats = {n: {"launches": 0, "ms": 0.0, "bytes": 0.0, "flops": 0.0, "launches_all": 0,
                     "bytes_all": 0.0, "flops_all": 0.0, "roof_ms_all": 0.0} for n in KERNEL_CLASSES}
        stats["attn"].update(launches=4, ms=4.0, bytes=8e9, flops=1e9, launches_all=4, bytes_all=8e9,
                             flops_all=1e9, roof_ms_all=1.0)
        stats["gemm_qkv"].update(launches=4, ms=1.0, bytes=2e9, flops=4e11, launches_all=4, bytes_all=2e9,
                                 flops_all=4e11, roof_ms_all=0.25)
        eng.kernel_stats = lambda: stats
        return eng

    monkeypatch.setattr(pkg, "Engine", plan_only_engine)
    monkeypatch.setattr(torch.cuda, "synchronize", lambda *a, **k: None)
    monkeypatch.setattr(torch.cuda, "empty_cache", lambda *a, **k: None)
    monkeypatch.setattr(sys, "argv", ["bench.py", "--workload", "tiny-moa-fp32", "--steps", "2", "--warmup", "1",
                                      "--block-steps", "4"])
    bench.main()
    lines = [l for l in capsys.readouterr().out.splitlines() if l.strip()]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for k, t in (("metric", str), ("value", float), ("unit", str), ("n_gpus", int), ("steps", int),
                 ("warmup", int), ("ms_per_step", float), ("higher_is_better", bool), ("scaling", str),
                 ("dtype", str), ("data", str), ("config", dict), ("roofline", dict), ("cpu_baseline", dict)):
        assert isinstance(d[k], t), k
    assert d["n_gpus"] == 1 and d["steps"] == 2 and d["warmup"] == 1 and d["value"] > 0
    assert d["higher_is_better"] is True and d["scaling"] in ("weak", "strong") and d["vs_baseline"] is None
    assert d["data"] == "synthetic" and d["config"]["workload"] == "tiny-moa-fp32"
    assert abs(d["ms_per_step"] * d["steps"] / 1e3 - d["timed_wall_s"]) < 1e-9
    r = d["roofline"]
    assert {"bound", "achieved", "peak", "unit", "frac", "traffic"} <= set(r)
    assert r["kernel"] == "attn" and r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert abs(r["achieved"] - 2000.0) < 1e-6 and abs(r["frac"] - 0.25) < 1e-9
    assert r["traffic"] is None                      # no counter record for this workload
    c = d["cpu_baseline"]
    assert c["kind"] == "oracle" and c["unit"] == "tokens/s" and c["value"] > 0
    assert isinstance(c["cores"], int) and c["cores"] >= 1 and isinstance(c["sample"], str)
