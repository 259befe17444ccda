"""moa_step_noalloc (the allocation-free step) against moa_step, on the GPU.

Two engines with the same models run the same calls, one through moa_step
and one through moa_step_noalloc, twice in a row (the second batch smaller,
so the library's scratch array holds the first run's partials when the
second starts): tokens and captured logits must be bit-identical (same plan,
same kernels; only where the partial sums live differs). The bf16 case has
two models, so both model streams' split-K partials sit in the scratch.
"""
import numpy as np
import pytest

from moa_inputs import CONFIGS, ModelShape, generate_weights, pack_blob
from moa_inputs.configs import EngineConsts
from paper_2606_03014_amd import Engine
from paper_2606_03014_amd import moa as M

pytestmark = pytest.mark.gpu

SMALL_BF16 = ModelShape(n_layers=2, d_model=256, n_heads=8, n_kv_heads=2, head_dim=64, ffn_dim=512, vocab=1024)


def _run(eng, mids, reqs, vocab, noalloc):
    caps, rids = {}, []
    for toks, m, G in reqs:
        rid = eng.submit(np.asarray(toks, dtype=np.int32), mids[m], G)
        caps[rid] = np.full(G * vocab, np.nan, dtype=np.float32)
        eng.capture_logits(rid, caps[rid])
        rids.append(rid)
    while True:
        info = eng.step_noalloc() if noalloc else eng.step()
        if info.step < 0:
            break
    got = {r[0]: r[3] for r in eng.collect()}
    return [got[r] for r in rids], [caps[r] for r in rids]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_step_noalloc_matches_step_twice_in_a_row(dtype):
    import torch
    assert torch.cuda.is_available()
    if dtype == "f32":
        c = CONFIGS["tiny-moa-fp32"]
        shape, consts = c.model, EngineConsts(num_kv_blocks=128, max_num_seqs=8, max_prefill_tokens=64,
                                              max_model_len=512)
        ws = [generate_weights(shape, "f32", 5, c.wid, m) for m in range(2)]
    else:
        shape = SMALL_BF16
        consts = EngineConsts(num_kv_blocks=256, max_num_seqs=8, max_prefill_tokens=96, max_model_len=512)
        ws = [generate_weights(shape, "bf16", 5, 99, m) for m in range(2)]
    rng = np.random.default_rng(3)
    big = [(rng.integers(0, shape.vocab, n), i % 2, G)
           for i, (n, G) in enumerate([(1, 30), (70, 12), (300, 25), (33, 40), (128, 8), (250, 20)])]
    small = [(rng.integers(0, shape.vocab, n), i % 2, G) for i, (n, G) in enumerate([(17, 9), (5, 14)])]
    engines = [Engine(shape, dtype, consts, 2) for _ in range(2)]
    try:
        mids = [[eng.load(pack_blob(w, shape)) for w in ws] for eng in engines]
        for batch, name in ((big, "first (6 calls)"), (small, "second (2 calls)")):
            ref_t, ref_l = _run(engines[0], mids[0], batch, shape.vocab, noalloc=False)
            got_t, got_l = _run(engines[1], mids[1], batch, shape.vocab, noalloc=True)
            for i in range(len(batch)):
                assert np.array_equal(ref_t[i], got_t[i]), f"{dtype} {name} call {i}: tokens differ"
                assert np.array_equal(ref_l[i], got_l[i], equal_nan=True), f"{dtype} {name} call {i}: logits differ"
                assert np.all(np.isfinite(got_l[i]))
            print(f"{dtype} {name}: moa_step_noalloc bit-identical to moa_step", flush=True)
    finally:
        for eng in engines:
            eng.close()


def test_step_noalloc_refuses_partials_beyond_the_scratch_on_a_gpu_engine():
    """An engine whose planned partials exceed the 64 MiB scratch gets
    MOA_ENOMEM and is left as it was: moa_step then runs its steps."""
    import torch
    assert torch.cuda.is_available()
    shape = SMALL_BF16
    consts = EngineConsts(num_kv_blocks=256, max_num_seqs=512, max_prefill_tokens=16384, max_model_len=512)
    eng = Engine(shape, "bf16", consts, 2)
    try:
        mid = eng.load(pack_blob(generate_weights(shape, "bf16", 5, 99, 0), shape))
        eng.submit(np.arange(20, dtype=np.int32), mid, 3)
        with pytest.raises(M.MoaError) as err:
            eng.step_noalloc()
        assert err.value.code == M.MOA_ENOMEM
        assert len(eng.steps()) == 0
        n = 0
        while eng.step().step >= 0:
            n += 1
        assert n == 3 and len(eng.collect()[0][3]) == 3
    finally:
        eng.close()
