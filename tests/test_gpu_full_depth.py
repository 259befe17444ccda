"""GPU parity at full 8B depth (32 layers): calls of the 3+1x8B workload's
first expert, and one decode step of calls that arrive with long K/V
histories (the straggler workload's Pareto lengths up to 32,768).

Teacher-forced against the oracle (bf16 K/V cache): logits within 2e-2,
the distance to the exact-cache oracle within tests.gpu_helpers.PURE_TOL,
tokens identical unless the oracle's top-2 margin is below 1e-3. The 8B
weights and the oracle's float64 copy of them (64 GB of host memory) are
made once for the module.
"""
import numpy as np
import pytest

from moa_inputs import CONFIGS, generate_weights, make_workload, pack_blob, f32_to_bf16_bits
from moa_inputs.configs import EngineConsts
from moa_inputs.workload import synthetic_kv
from oracle import transformer as T
from paper_2606_03014_amd import Engine
from tests.gpu_helpers import PURE_TOL, check_tokens, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def expert0():
    import torch
    assert torch.cuda.is_available(), "GPU tests need the MI355X"
    c = CONFIGS["moa-3+1x8b-bf16"]
    say("full depth: generating the 3+1x8B workload's expert 0 (8B shape, 32 layers)")
    w = generate_weights(c.model, "bf16", 0, c.wid, 0, threads=16)
    blob = pack_blob(w, c.model)
    om = T.OracleModel(c.model, w)
    yield c, w, blob, om
    del om, blob, w


def _engine(c, consts, blob):
    eng = Engine(c.model, "bf16", consts, 1)
    mid = eng.load(blob)
    return eng, mid


def test_full_depth_8b_workload_calls(expert0):
    """Two calls of expert 0 from the 3+1x8B workload (its shortest prompts),
    four tokens each, through all 32 layers."""
    c, w, blob, om = expert0
    wl = make_workload(c.name, 0)
    calls = sorted(((len(wl.prompts[q]), q) for q, e, G in wl.expert_requests() if e == 0))[:2]
    consts = EngineConsts(num_kv_blocks=64, max_num_seqs=4, max_prefill_tokens=512, max_model_len=1024)
    eng, mid = _engine(c, consts, blob)
    G = 4
    try:
        rids, caps = [], []
        for _, q in calls:
            rid = eng.submit(wl.prompts[q], mid, G)
            caps.append(np.full(G * c.model.vocab, np.nan, dtype=np.float32))
            eng.capture_logits(rid, caps[-1])
            rids.append(rid)
        while eng.step().step >= 0:
            pass
        got = {r[0]: r[3] for r in eng.collect()}
    finally:
        eng.close()
    for (P, q), rid, cap in zip(calls, rids, caps):
        toks = got[rid]
        lg = cap.reshape(G, -1)
        ref = T.teacher_forced_logits(om, wl.prompts[q], toks, bf16_kv=True)
        pure = T.teacher_forced_logits(om, wl.prompts[q], toks)
        err, perr = float(np.abs(lg - ref).max()), float(np.abs(lg - pure).max())
        flips = check_tokens(ref, toks, f"query {q}")
        say(f"full depth query {q} P={P}: |engine - oracle| {err:.3e} (exact cache {perr:.3e}; the oracle's "
            f"own bf16-cache effect {float(np.abs(ref - pure).max()):.3e}) flips {flips}")
        assert err <= 2e-2 and perr <= PURE_TOL


def test_full_depth_8b_straggler_step(expert0):
    """Calls with K/V histories at the straggler workload's Pareto(1.2) x 256
    quantiles up to the 32,768 cap (bf16 histories through all 32 layers),
    two decode steps each, in one batch."""
    c, w, blob, om = expert0
    g = c.model
    Ls = [0, 255, 256, 1051, 4000, 16383, 32768]
    R = 2
    need = sum((L + R + 15) // 16 for L in Ls)
    consts = EngineConsts(num_kv_blocks=need + 64, max_num_seqs=16, max_prefill_tokens=64, max_model_len=32800)
    rng = np.random.default_rng(17)
    seeds = [int(x) for x in rng.integers(0, g.vocab, len(Ls))]
    eng, mid = _engine(c, consts, blob)
    hist = []
    try:
        rids, caps = [], []
        for i, (L, tok) in enumerate(zip(Ls, seeds)):
            kvb = f32_to_bf16_bits(synthetic_kv(3, i, g.n_layers, L, g.n_kv_heads, g.head_dim)) if L else None
            hist.append(kvb)
            rid = eng.submit_with_history(mid, tok, L, R, kvb)
            caps.append(np.full(R * g.vocab, np.nan, dtype=np.float32))
            eng.capture_logits(rid, caps[-1])
            rids.append(rid)
        say("full depth straggler: histories submitted")
        steps = []
        while True:
            info = eng.step()
            if info.step < 0:
                break
            steps.append(info.decode_rows)
        got = {r[0]: r[3] for r in eng.collect()}
    finally:
        eng.close()
    assert steps[0] == len(Ls)
    for i, (L, tok) in enumerate(zip(Ls, seeds)):
        toks = got[rids[i]]
        kv = T.ContiguousKV(g.n_layers, g.n_kv_heads, g.head_dim)
        if L:
            for layer in range(g.n_layers):
                kv.K[layer] = T.to_f64(hist[i][layer, 0])
                kv.V[layer] = T.to_f64(hist[i][layer, 1])
        seq = [tok] + [int(t) for t in toks[:-1]]
        ref = T.forward_chunk(om, seq, L, kv, bf16_kv=True)
        err = float(np.abs(caps[i].reshape(R, -1) - ref).max())
        flips = check_tokens(ref, toks, f"history L={L}")
        say(f"full depth history L={L}: |engine - oracle| {err:.3e} flips {flips}")
        assert err <= 2e-2
        hist[i] = None
