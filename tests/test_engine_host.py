"""Host-side tests of the C-ABI library (no GPU): symbols, argument checks, and
the engine's step bookkeeping against the oracle scheduler (dry-run mode)."""
import json
import os
import re

import numpy as np
import pytest

from moa_inputs import CONFIGS, ModelShape, make_workload
from moa_inputs.configs import EngineConsts
from oracle.scheduler import OracleScheduler, run_feeder as oracle_feeder
from paper_2606_03014_amd import Engine, run_feeder
from paper_2606_03014_amd import moa as M

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLD = json.load(open(os.path.join(ROOT, "tests", "golden", "step_rule_examples.json")))
TOY = ModelShape(1, 256, 4, 2, 64, 256, 256)


def _blob_bytes(shape, dtype):
    return shape.n_params() * (2 if dtype == "bf16" else 4)


def _dry(shape, consts, n_models, dtype="bf16"):
    eng = Engine(shape, dtype, consts, max(n_models, 1), plan_only=True)
    for _ in range(n_models):
        eng.load(np.zeros(_blob_bytes(shape, dtype), dtype=np.uint8))
    return eng


def test_library_exports_every_declared_symbol():
    hdr = open(os.path.join(ROOT, "include", "moa.h")).read()
    hdr = re.sub(r"/\*.*?\*/", "", hdr, flags=re.S)
    declared = set(re.findall(r"\b(moa_[a-z_]+)\s*\(", hdr))
    assert len(declared) >= 14
    lib = M.lib()
    for name in declared:
        assert hasattr(lib, name), name
    assert declared == set(M.exported_symbols())


def test_binding_constants_match_the_header():
    """Every MOA_* enum value the header defines has the same value in the
    ctypes binding (flags, dtypes, status codes)."""
    hdr = open(os.path.join(ROOT, "include", "moa.h")).read()
    hdr = re.sub(r"/\*.*?\*/", "", hdr, flags=re.S)
    consts = {k: int(v) for k, v in re.findall(r"\b(MOA_[A-Z0-9_]+)\s*=\s*(-?\d+)", hdr)}
    for name in ("MOA_FLAG_PLAN_ONLY", "MOA_FLAG_ONE_STREAM", "MOA_F32", "MOA_BF16", "MOA_OK", "MOA_EINVAL"):
        assert name in consts, name
    for name, value in consts.items():
        if hasattr(M, name):
            assert getattr(M, name) == value, name
    assert consts["MOA_FLAG_PLAN_ONLY"] & consts["MOA_FLAG_ONE_STREAM"] == 0


def test_kernel_classes_follow_the_header_enum():
    """The binding's kernel-class names index moa_debug_kernel_stats' array in
    the order of the header's MOA_K_* enum, and the two GEMM views are last."""
    hdr = open(os.path.join(ROOT, "include", "moa.h")).read()
    hdr = re.sub(r"/\*.*?\*/", "", hdr, flags=re.S)
    body = hdr[hdr.index("MOA_K_EMBED = 0"):hdr.index("MOA_K_COUNT")]
    names = [n.lower() for n in re.findall(r"MOA_K_([A-Z_]+)", body)]
    assert [n.replace("_", "") for n in names] == [c.replace("_", "") for c in M.KERNEL_CLASSES]
    assert M.KERNEL_CLASSES[-2:] == list(M.VIEW_CLASSES)


def test_feeder_in_blocks_matches_one_run_and_counts_every_token():
    """Advancing the feeder a fixed number of engine steps at a time (the
    benchmark's timed blocks) gives the same schedule as one uninterrupted
    run, and the steps' emitted counts add up to every generated token."""
    from paper_2606_03014_amd import Feeder
    c = CONFIGS["moa-3+1x8b-bf16"]
    wl = make_workload(c.name, 0, n_queries=48)
    runs = []
    for block in (None, 7, 128):
        eng = _dry(c.model, c.engine, 4)
        f = Feeder(eng, wl, [0, 1, 2], agg_model=3)
        per_block = []
        while not f.done:
            per_block.append(f.advance(block))
        steps = eng.steps()
        eng.close()
        assert sum(n for n, _ in per_block) == f.res.n_steps == len(steps)
        if block is not None:
            assert all(n == block for n, _ in per_block[:-2])
        assert f.emitted == sum(t for _, t in per_block) == f.res.tokens
        assert f.res.tokens == wl.total_expert_tokens() + f.res.agg_calls * wl.agg_max_new
        runs.append((steps.tolist(), sorted(f.res.rid_of.items()), f.res.collects))
    assert runs[0] == runs[1] == runs[2]


def test_capture_logits_checks_its_capacity():
    """moa_debug_capture_logits takes the buffer's size in floats and refuses
    one below max_new_tokens * vocab (nothing registered), and refuses a
    request whose prefill has completed."""
    c = CONFIGS["tiny-moa-fp32"]
    eng = _dry(c.model, c.engine, 1, dtype="f32")
    rid = eng.submit(np.arange(10, dtype=np.int32), 0, 5)
    with pytest.raises(M.MoaError) as err:
        eng.capture_logits(rid, np.zeros(5 * c.model.vocab - 1, dtype=np.float32))
    assert err.value.code == M.MOA_EINVAL
    with pytest.raises(ValueError):
        eng.capture_logits(rid, np.zeros(5 * c.model.vocab, dtype=np.float64))
    buf = np.zeros(5 * c.model.vocab, dtype=np.float32)
    eng.capture_logits(rid, buf)
    eng.step()
    with pytest.raises(M.MoaError) as err:
        eng.capture_logits(rid, buf)
    assert err.value.code == M.MOA_ESTATE
    eng.close()


@pytest.mark.parametrize("field,value", [("vocab", 32016), ("n_kv_heads", 1), ("head_dim", 64)])
def test_bf16_widths_must_be_whole_128_column_tiles(field, value):
    """A bf16 engine takes only projection widths that are whole 128-column
    GEMM tiles (LM head = vocab, qkv = (heads + 2 kv heads) x head_dim):
    anything else is refused at moa_arena_bytes / moa_create."""
    from dataclasses import replace as rp
    from paper_2606_03014_amd.engine import engine_cfg
    c = CONFIGS["moa-4x1b-bf16"]
    base = ModelShape(n_layers=2, d_model=256, n_heads=5, n_kv_heads=2, head_dim=64, ffn_dim=512, vocab=1024) \
        if field != "vocab" else c.model
    if field == "vocab":
        shape = rp(base, vocab=value)
    elif field == "n_kv_heads":          # (5 + 2) * 64 = 448: not a multiple of 128
        shape = rp(base, n_heads=5, n_kv_heads=1)
    else:                                # (5 + 4) * 64 = 576
        shape = rp(base, n_heads=5, n_kv_heads=2)
    with pytest.raises(M.MoaError) as err:
        M.moa_arena_bytes(engine_cfg(shape, "bf16", c.engine, 1))
    assert err.value.code == M.MOA_EINVAL
    ok = rp(c.model, vocab=32000)
    assert M.moa_arena_bytes(engine_cfg(ok, "bf16", c.engine, 1)) > 0


def test_step_noalloc_plans_like_step_and_refuses_oversized_partials():
    """The allocation-free step plans exactly like moa_step (same bookkeeping
    on a dry run); an engine whose planned partials exceed the library's
    64 MiB scratch is refused with MOA_ENOMEM before anything changes."""
    c = CONFIGS["tiny-moa-fp32"]
    wl = make_workload(c.name, 0)
    traces = []
    for noalloc in (False, True):
        eng = _dry(c.model, c.engine, 3, dtype="f32")
        for q, e, G in wl.expert_requests():
            eng.submit(wl.prompts[q], e, G)
        while (eng.step_noalloc() if noalloc else eng.step()).step >= 0:
            pass
        traces.append(eng.steps().tolist())
        eng.close()
    assert traces[0] == traces[1] and len(traces[0]) > 10
    big = CONFIGS["moa-3+1x8b-bf16"]
    eng = _dry(big.model, big.engine, 4)
    eng.submit(np.arange(20, dtype=np.int32), 0, 3)
    with pytest.raises(M.MoaError) as err:
        eng.step_noalloc()
    assert err.value.code == M.MOA_ENOMEM
    assert len(eng.steps()) == 0
    assert eng.step().step == 0
    eng.close()


def test_second_model_stream_reserves_one_partial_buffer():
    """A bf16 engine reserves split-K partials for its second model stream in
    the arena; MOA_FLAG_ONE_STREAM drops exactly that buffer, and fp32
    engines (one stream) are unaffected by the flag."""
    from paper_2606_03014_amd.engine import engine_cfg
    c = CONFIGS["moa-4x1b-bf16"]
    two = M.moa_arena_bytes(engine_cfg(c.model, "bf16", c.engine, 4))
    one = M.moa_arena_bytes(engine_cfg(c.model, "bf16", c.engine, 4, one_stream=True))
    g, e = c.model, c.engine
    qkv = (g.n_heads + 2 * g.n_kv_heads) * g.head_dim
    tmax = e.max_prefill_tokens + e.max_num_seqs
    part = max(tmax, 8 * e.max_num_seqs) * max(qkv, g.d_model) * 4
    assert two - one == (part + 255) // 256 * 256
    f = CONFIGS["tiny-moa-fp32"]
    assert (M.moa_arena_bytes(engine_cfg(f.model, "f32", f.engine, 3))
            == M.moa_arena_bytes(engine_cfg(f.model, "f32", f.engine, 3, one_stream=True)))


def test_model_stream_shares_are_greedy_cost_balanced():
    """A plan-only bf16 engine plans the model-stream split of a two-stream
    GPU engine. On every step of a skewed four-expert batch: the shares
    partition the step's models, rows and LM rows into contiguous runs; each
    model's cost is its weight bytes times max(1, rows / 96) plus the K/V
    bytes its rows' attention reads; and the split is the greedy one (largest
    cost first, each to the share with the least cost so far)."""
    from paper_2606_03014_amd.engine import engine_cfg
    c = CONFIGS["moa-4x1b-bf16"]
    g = c.model
    model_bytes = (M.moa_arena_bytes(engine_cfg(g, "bf16", c.engine, 4))
                   - M.moa_arena_bytes(engine_cfg(g, "bf16", c.engine, 3)))
    kv_pos = g.n_layers * g.n_kv_heads * 2 * g.head_dim * 2
    eng = _dry(g, c.engine, 4)
    snaps = {}
    wl = make_workload(c.name, 0, n_queries=48)
    r = run_feeder(eng, wl, [0, 1, 2, 3], on_step=lambda info: snaps.__setitem__(info.step, eng.step_shares()))
    S = r.n_steps
    rows = np.zeros((S, 4), np.int64)
    lms = np.zeros((S, 4), np.int64)
    keys = np.zeros((S, 4), np.float64)
    for (q, m), rid in r.rid_of.items():
        info = eng.request(rid)
        P = info.prompt_len
        for s, a, b in eng.chunks(rid):
            rows[s, m] += b
            keys[s, m] += b * a + b * (b + 1) / 2          # positions a .. a+b-1 see pos+1 keys
            lms[s, m] += (a + b == P)
        d0 = max(s for s, a, b in eng.chunks(rid)) + 1
        for t in range(d0, info.finish_step + 1):
            rows[t, m] += 1
            lms[t, m] += 1
            keys[t, m] += P + 1 + (t - d0)
    eng.close()
    two = 0
    for s in range(S):
        sh = snaps[s]
        active = [m for m in range(4) if rows[s, m]]
        assert sorted(sh["models"]) == active
        assert len(sh["shares"]) == max(1, min(2, len(active)))
        assert [m for mods, _, _ in sh["shares"] for m in mods] == sh["models"]
        r0 = l0 = 0
        for mods, rr, ll in sh["shares"]:
            assert mods == sorted(mods)
            assert rr.start == r0 and len(rr) == sum(rows[s, m] for m in mods)
            assert ll.start == l0 and len(ll) == sum(lms[s, m] for m in mods)
            r0, l0 = rr.stop, ll.stop
        assert r0 == rows[s].sum() and l0 == lms[s].sum()
        cost = dict(zip(sh["models"], sh["cost"]))
        for m in active:
            want = model_bytes * max(1.0, rows[s, m] / 96.0) + kv_pos * keys[s, m]
            assert cost[m] == pytest.approx(want, rel=1e-12)
        if len(active) >= 2:
            two += 1
            load, sets = [0.0, 0.0], [[], []]
            for m in sorted(active, key=lambda m: -cost[m]):
                u = 0 if load[0] <= load[1] else 1
                load[u] += cost[m]
                sets[u].append(m)
            assert [sorted(x) for x in sets] == [mods for mods, _, _ in sh["shares"]]
    assert two > S // 2


def test_status_strings():
    for code in (0, -1, -2, -3, -4, -5):
        assert M.moa_status_str(code).startswith(M.STATUS_NAMES[code])


def test_config_validation_and_arena_size():
    c = CONFIGS["moa-4x1b-bf16"]
    from paper_2606_03014_amd.engine import engine_cfg
    good = engine_cfg(c.model, "bf16", c.engine, 4)
    n = M.moa_arena_bytes(good)
    weights = 4 * c.model.n_params() * 2
    kv = c.engine.num_kv_blocks * c.model.n_layers * c.model.n_kv_heads * 2 * 16 * c.model.head_dim * 2
    assert weights + kv < n < weights + kv + (8 << 30)
    for field, bad in [("kv_block_size", 32), ("max_models", 0), ("max_models", 9), ("dtype", 7)]:
        cfg = engine_cfg(c.model, "bf16", c.engine, 4)
        setattr(cfg, field, bad)
        with pytest.raises(M.MoaError) as e:
            M.moa_arena_bytes(cfg)
        assert e.value.code == M.MOA_EINVAL
    cfg = engine_cfg(c.model, "bf16", c.engine, 4)
    cfg.model.head_dim = 96
    with pytest.raises(M.MoaError):
        M.moa_arena_bytes(cfg)


def test_create_rejects_small_or_missing_arena():
    c = CONFIGS["tiny-moa-fp32"]
    from paper_2606_03014_amd.engine import engine_cfg
    cfg = engine_cfg(c.model, "f32", c.engine, 3)
    with pytest.raises(M.MoaError) as e:
        M.moa_create(cfg, None, 0, None)
    assert e.value.code == M.MOA_EINVAL
    with pytest.raises(M.MoaError) as e:
        M.moa_create(cfg, 1 << 20, 4096, None)          # never dereferenced: size check first
    assert e.value.code == M.MOA_ENOMEM


def test_submit_and_load_errors():
    consts = EngineConsts(num_kv_blocks=4, max_num_seqs=2, max_prefill_tokens=16, max_model_len=100)
    eng = _dry(TOY, consts, 1)
    with pytest.raises(M.MoaError) as e:
        eng.load(np.zeros(10, dtype=np.uint8))
    assert e.value.code == M.MOA_EINVAL
    for args, code in [(([1, 2], 1, 3), M.MOA_EINVAL), (([], 0, 3), M.MOA_EINVAL),
                       (([1, 2], 0, 0), M.MOA_EINVAL), (([1] * 60, 0, 6), M.MOA_ENOSPC),
                       (([1] * 90, 0, 20), M.MOA_EINVAL)]:
        with pytest.raises(M.MoaError) as e:
            eng.submit(*args)
        assert e.value.code == code, args
    assert eng.submit([1] * 60, 0, 5) == 0
    eng.step()
    with pytest.raises(M.MoaError) as e:
        eng.load(np.zeros(_blob_bytes(TOY, "bf16"), dtype=np.uint8))
    assert e.value.code == M.MOA_ESTATE


def test_collect_reports_required_capacity():
    consts = EngineConsts(num_kv_blocks=8, max_num_seqs=4, max_prefill_tokens=64, max_model_len=100)
    eng = _dry(TOY, consts, 1)
    for G in (3, 5):
        eng.submit([1, 2, 3], 0, G)
    while eng.step().step >= 0:
        pass
    import ctypes as C
    n = C.c_int32()
    res = (M.moa_result * 1)()
    buf = np.zeros(4, dtype=np.int32)
    code = M.lib().moa_collect(eng.h, -1, res, 1, C.byref(n), buf.ctypes.data_as(C.POINTER(C.c_int32)), 4)
    assert code == M.MOA_EINVAL and n.value == 2
    out = eng.collect()
    assert [r[0] for r in out] == [0, 1] and [len(r[3]) for r in out] == [3, 5]
    assert all((r[3] == -1).all() for r in out)          # a dry run computes no tokens
    assert eng.collect() == []


def test_hand_traced_example_matches():
    ex = GOLD["examples"][0]
    consts = EngineConsts(ex["num_blocks"], ex["max_num_seqs"], ex["max_prefill_tokens"], 1000)
    eng = _dry(TOY, consts, ex["n_models"])
    for kind, m, P, G in ex["submit"]:
        assert kind == "std"
        eng.submit(np.ones(P, dtype=np.int32), m, G)
    while eng.step().step >= 0:
        pass
    st = eng.steps()
    assert len(st) == ex["n_steps"]
    assert st[: len(ex["steps_head"])].tolist() == ex["steps_head"]
    for rid, want in enumerate(ex["requests"]):
        info = eng.request(rid)
        assert (info.admit_step, info.finish_step) == (want["admit"], want["finish"])
        assert eng.block_table(rid) == want["blocks"]
        assert [list(c) for c in eng.chunks(rid)] == want["chunks"]


def test_hand_traced_windowed_feeder_matches():
    """The engine's feeder with a submission window of one call reproduces
    the hand trace (aggregator calls overtake an unsubmitted expert call)."""
    f = GOLD["feeder_window"]
    consts = EngineConsts(f["num_blocks"], f["max_num_seqs"], f["max_prefill_tokens"], 1000)
    eng = _dry(TOY, consts, f["n_models"])
    nq = len(f["queries"])

    class W:
        prompts = [np.ones(q["P"], dtype=np.int32) for q in f["queries"]]
        experts = [tuple(e for e, _ in q["experts"]) for q in f["queries"]]
        max_new = {(qi, e): G for qi, q in enumerate(f["queries"]) for e, G in q["experts"]}
        n_experts = 2
        n_queries = nq
        agg_max_new = f["agg_G"]

        def expert_requests(self):
            return [(q, e, self.max_new[(q, e)]) for q in range(nq) for e in self.experts[q]]

    r = run_feeder(eng, W(), [0, 1], agg_model=f["aggregator"], window=f["window"])
    assert eng.steps().tolist() == f["steps"]
    assert [[a, list(b)] for a, b in r.collects] == f["collects"]
    for rid, want in enumerate(f["requests"]):
        info = eng.request(rid)
        assert (info.model_id, info.prompt_len, info.max_new_tokens, info.admit_step, info.finish_step) == (
            want["model"], want["P"], want["G"], want["admit"], want["finish"])
        assert eng.block_table(rid) == want["blocks"]
    eng.close()


def test_hand_traced_feeder_matches():
    f = GOLD["feeder"]
    consts = EngineConsts(f["num_blocks"], f["max_num_seqs"], f["max_prefill_tokens"], 1000)
    eng = _dry(TOY, consts, f["n_models"])

    class W:                                          # a two-query workload in the feeder's terms
        prompts = [np.ones(q["P"], dtype=np.int32) for q in f["queries"]]
        experts = [tuple(e for e, _ in q["experts"]) for q in f["queries"]]
        max_new = {(qi, e): G for qi, q in enumerate(f["queries"]) for e, G in q["experts"]}
        n_experts = 2
        n_queries = 2
        agg_max_new = f["agg_G"]

        def expert_requests(self):
            return [(q, e, self.max_new[(q, e)]) for q in range(2) for e in self.experts[q]]

    r = run_feeder(eng, W(), [0, 1], agg_model=f["aggregator"])
    assert eng.steps().tolist() == f["steps"]
    assert [[a, list(b)] for a, b in r.collects] == f["collects"]
    for rid, want in enumerate(f["requests"]):
        info = eng.request(rid)
        assert (info.model_id, info.prompt_len, info.max_new_tokens, info.admit_step, info.finish_step) == (
            want["model"], want["P"], want["G"], want["admit"], want["finish"])
        assert eng.block_table(rid) == want["blocks"]


def _compare_full(name, seed=0):
    c = CONFIGS[name]
    w = make_workload(name, seed)
    nm = c.n_experts + (1 if c.aggregator else 0)
    eng = _dry(c.model, c.engine, nm, c.dtype)
    agg = c.n_experts if c.aggregator else -1
    r = run_feeder(eng, w, list(range(c.n_experts)), agg_model=agg)
    s = OracleScheduler(c.engine.num_kv_blocks, c.engine.max_num_seqs, c.engine.max_prefill_tokens, nm,
                        max_model_len=c.engine.max_model_len)
    calls = [(q, e, len(w.prompts[q]), G) for q, e, G in w.expert_requests()]
    direct = [(q, 0, len(w.prompts[q]), w.agg_max_new) for q in range(w.n_queries)] if c.n_experts == 0 else []
    log, rid_of = oracle_feeder(s, calls, agg_model=agg if c.n_experts else -1, agg_G=w.agg_max_new,
                                query_len=[len(p) for p in w.prompts], query_experts=w.experts,
                                direct_calls=direct)
    assert np.array_equal(eng.steps(), np.array(s.steps, dtype=np.int64))
    assert [(a, list(b)) for a, b in r.collects] == [(a, list(b)) for a, b in log]
    for req in s.reqs[:: max(1, len(s.reqs) // 64)]:
        info = eng.request(req.rid)
        assert (info.model_id, info.prompt_len, info.max_new_tokens) == (req.expert, req.P, req.G)
        assert (info.admit_step, info.finish_step) == (req.admit_step, req.finish_step)
        assert eng.block_table(req.rid) == req.blocks
        assert [tuple(x) for x in eng.chunks(req.rid)] == [tuple(x) for x in req.chunks]
    return r


@pytest.mark.parametrize("name", ["tiny-moa-fp32", "moa-4x1b-bf16", "agg-prefill-8b-bf16"])
def test_full_workload_bookkeeping_is_bit_exact(name):
    _compare_full(name)


@pytest.mark.slow
def test_full_3p1x8b_bookkeeping_is_bit_exact():
    r = _compare_full("moa-3+1x8b-bf16")
    assert r.tokens == 5966555


@pytest.mark.parametrize("seed", range(25))
def test_random_small_workloads_bit_exact(seed):
    rng = np.random.default_rng(1000 + seed)
    consts = EngineConsts(int(rng.integers(4, 40)), int(rng.integers(1, 6)), int(rng.integers(1, 80)), 200)
    eng = _dry(TOY, consts, 3)
    s = OracleScheduler(consts.num_kv_blocks, consts.max_num_seqs, consts.max_prefill_tokens, 3,
                        max_model_len=200)
    for _ in range(int(rng.integers(1, 14))):
        m, P, G = int(rng.integers(0, 3)), int(rng.integers(1, 60)), int(rng.integers(1, 30))
        try:
            s.submit(m, P, G)
            ok = True
        except Exception:
            ok = False
        if ok:
            eng.submit(np.ones(P, dtype=np.int32), m, G)
        else:
            with pytest.raises(M.MoaError):
                eng.submit(np.ones(P, dtype=np.int32), m, G)
    while True:
        a = eng.step().step
        b = s.step()
        assert a == (-1 if b is None else b)
        if b is None:
            break
    assert np.array_equal(eng.steps(), np.array(s.steps, dtype=np.int64).reshape(-1, 6))
    for req in s.reqs:
        assert eng.block_table(req.rid) == req.blocks


def test_hand_traced_injected_history_matches():
    ex = GOLD["examples"][1]
    consts = EngineConsts(ex["num_blocks"], ex["max_num_seqs"], 16, 1000)
    eng = _dry(TOY, consts, ex["n_models"])
    for kind, m, L, R in ex["submit"]:
        assert kind == "inj"
        eng.submit_with_history(m, 1, L, R)
    while eng.step().step >= 0:
        pass
    st = eng.steps()
    assert len(st) == ex["n_steps"]
    assert st[: len(ex["steps_head"])].tolist() == ex["steps_head"]
    for rid, want in enumerate(ex["requests"]):
        info = eng.request(rid)
        assert (info.admit_step, info.finish_step) == (want["admit"], want["finish"])
        assert eng.block_table(rid) == want["blocks"]
        assert eng.chunks(rid) == []


def test_straggler_workload_bookkeeping_is_bit_exact():
    """The whole straggler workload -- refill phase (every retired call
    replaced at the next admission) then drain -- against the oracle
    scheduler driven the same way."""
    from moa_inputs import make_straggler_workload
    from paper_2606_03014_amd.engine import run_straggler
    c = CONFIGS["straggler-8b-bf16"]
    sw = make_straggler_workload(0)                   # the whole workload: 512 live, 512 refill steps
    eng = _dry(c.model, c.engine, 1, "bf16")
    tokens, steps, used = run_straggler(eng, sw)
    s = OracleScheduler(c.engine.num_kv_blocks, c.engine.max_num_seqs, c.engine.max_prefill_tokens, 1,
                        max_model_len=c.engine.max_model_len)
    nxt = 0
    for _ in range(sw.n_live):
        L, tok, R = sw.sequence(nxt)
        s.submit_injected(0, L, R)
        nxt += 1
    while True:
        st = s.step()
        if st is None:
            break
        if st < sw.refill_steps:
            for _ in range(s.steps[-1][4]):
                L, tok, R = sw.sequence(nxt)
                s.submit_injected(0, L, R)
                nxt += 1
    assert used == nxt and steps == len(s.steps)
    assert np.array_equal(eng.steps(), np.array(s.steps, dtype=np.int64))
    for req in s.reqs[::17]:
        info = eng.request(req.rid)
        assert (info.admit_step, info.finish_step) == (req.admit_step, req.finish_step)
        assert eng.block_table(req.rid) == req.blocks
    assert tokens == sum(r.G for r in s.reqs)


def test_straggler_refill_counts_from_the_runs_first_step():
    """A second drive of the same engine (a benchmark's timed pass after its
    warm-up) refills for the same number of its own steps as the first."""
    from moa_inputs import make_straggler_workload
    from paper_2606_03014_amd.engine import run_straggler
    c = CONFIGS["straggler-8b-bf16"]
    sw = make_straggler_workload(0, n_live=64, refill_steps=32)
    eng = _dry(c.model, c.engine, 1, "bf16")
    first = run_straggler(eng, sw)
    second = run_straggler(eng, sw)
    assert first == second
    assert first[2] > sw.n_live
