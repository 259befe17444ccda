"""Pins for the oracle's whole-model paths (forward, caches, greedy decoding)."""
import numpy as np
import pytest

from moa_inputs import CONFIGS, ModelShape, generate_weights
from oracle import transformer as T
from tests.torch_reference import torch_logits

MINI = ModelShape(n_layers=2, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16,
                  ffn_dim=128, vocab=97)


def _model(shape=MINI, dtype="f32", seed=0, model_id=0, scale=None):
    w = generate_weights(shape, dtype, seed, 99, model_id)
    if scale is not None:                        # larger weights: sharper attention
        w = {k: (v * scale if not k.endswith("norm") else v) for k, v in w.items()}
    return T.OracleModel(shape, w), w


def _tokens(n, V, seed=0):
    return np.random.default_rng([77, seed]).integers(0, V, n)


@pytest.mark.parametrize("scale", [1.0, 25.0])
def test_forward_matches_torch_functional_model(scale):
    om, w = _model(scale=scale)
    toks = _tokens(29, MINI.vocab)
    np.testing.assert_allclose(T.forward_full(om, toks), torch_logits(MINI, w, toks),
                               rtol=1e-10, atol=1e-12)


def test_forward_matches_torch_on_tiny_workload_shape():
    shape = CONFIGS["tiny-moa-fp32"].model
    om, w = _model(shape, seed=3)
    toks = _tokens(40, shape.vocab, 1)
    np.testing.assert_allclose(T.forward_full(om, toks), torch_logits(shape, w, toks),
                               rtol=1e-10, atol=1e-12)


def test_zero_layer_model_is_closed_form():
    """With no layers the model is logits = Wlm . rmsnorm(E[t])."""
    om, w = _model()
    om.n_layers = 0
    toks = _tokens(5, MINI.vocab)
    E = w["embed"].astype(np.float64)
    x = E[toks]
    xn = x / np.sqrt((x * x).mean(-1, keepdims=True) + MINI.rms_eps)
    np.testing.assert_allclose(T.forward_full(om, toks), xn @ w["lm_head"].astype(np.float64).T,
                               rtol=1e-12, atol=1e-14)


def test_zero_output_projections_reduce_to_closed_form():
    """With Wo = Wdown = 0 every layer is the identity on the residual."""
    om, w = _model()
    for l in range(MINI.n_layers):
        w[f"layers.{l}.wo"] = np.zeros_like(w[f"layers.{l}.wo"])
        w[f"layers.{l}.w_down"] = np.zeros_like(w[f"layers.{l}.w_down"])
    om = T.OracleModel(MINI, w)
    toks = _tokens(6, MINI.vocab, 2)
    om0 = T.OracleModel(MINI, w, n_layers=0)
    np.testing.assert_allclose(T.forward_full(om, toks), T.forward_full(om0, toks), rtol=0, atol=0)


def test_cached_decode_equals_brute_force_prefix():
    om, _ = _model(scale=10.0)
    prompt = _tokens(7, MINI.vocab, 3)
    out, lg = T.greedy_generate(om, prompt, 6, return_logits=True)
    seq = np.concatenate([prompt, out[:-1]])
    bf = T.brute_force_prefix_logits(om, seq)
    np.testing.assert_allclose(lg, bf[len(prompt) - 1:], rtol=1e-11, atol=1e-12)
    for j, t in enumerate(out):
        assert t == T.argmax_lowest(bf[len(prompt) - 1 + j])


def test_prefill_logits_equal_decode_logits():
    """Logits at position t from a whole-sequence prefill equal those of a
    decode step after prefilling t tokens."""
    om, _ = _model(scale=5.0)
    toks = _tokens(12, MINI.vocab, 4)
    full = T.forward_full(om, toks)
    for t in (1, 5, 11):
        kv = T.ContiguousKV(om.n_layers, MINI.n_kv_heads, MINI.head_dim)
        T.forward_chunk(om, toks[:t], 0, kv)
        lg = T.forward_chunk(om, toks[t:t + 1], t, kv)[-1]
        np.testing.assert_allclose(lg, full[t], rtol=1e-11, atol=1e-12)


def test_paged_equals_contiguous_bit_exact():
    om, _ = _model(scale=5.0)
    prompt = _tokens(21, MINI.vocab, 5)
    G = 14
    contiguous = T.greedy_generate(om, prompt, G, return_logits=True)
    bs = 4
    nblk = -(-(len(prompt) + G - 1) // bs)
    pool = T.PagedKV.make_pool(40, om.n_layers, MINI.n_kv_heads, MINI.head_dim, bs)
    table = list(np.random.default_rng(5).permutation(40)[:nblk])   # scattered blocks
    paged = T.greedy_generate(om, prompt, G, kv=T.PagedKV(pool, table, bs), return_logits=True)
    assert contiguous[0] == paged[0]
    assert np.array_equal(contiguous[1], paged[1])


def test_teacher_forced_logits_reproduce_free_run():
    om, _ = _model(scale=5.0)
    prompt = _tokens(9, MINI.vocab, 6)
    out, lg = T.greedy_generate(om, prompt, 8, return_logits=True)
    tf = T.teacher_forced_logits(om, prompt, out)
    np.testing.assert_allclose(tf, lg, rtol=1e-11, atol=1e-12)


def test_decode_from_history_matches_prefill():
    om, _ = _model(scale=5.0)
    toks = _tokens(10, MINI.vocab, 7)
    kv = T.ContiguousKV(om.n_layers, MINI.n_kv_heads, MINI.head_dim)
    T.forward_chunk(om, toks[:9], 0, kv)
    lg = T.decode_from_history(om, kv.K, kv.V, toks[9], 9)
    np.testing.assert_allclose(lg, T.forward_full(om, toks)[9], rtol=1e-11, atol=1e-12)


def test_bf16_kv_rounds_only_the_cache():
    """bf16_kv changes the logits only through the stored K/V: a model whose
    K/V projections produce bf16-representable values is unaffected, and the
    bf16 weights themselves are read exactly."""
    shape = MINI
    w = generate_weights(shape, "bf16", 0, 99, 0)
    om = T.OracleModel(shape, w)
    toks = _tokens(16, shape.vocab, 8)
    a = T.forward_full(om, toks)
    b = T.forward_full(om, toks, bf16_kv=True)
    err = np.abs(a - b).max()
    assert 0 < err < 5e-2 * np.abs(a).max()
    np.testing.assert_allclose(a, torch_logits(shape, w, toks), rtol=1e-10, atol=1e-12)
    # the rounding points themselves: torch's own bf16 cast of k after RoPE
    # and of v (never q), at the exact same places
    np.testing.assert_allclose(b, torch_logits(shape, w, toks, bf16_kv=True), rtol=0, atol=1e-12)
    w2 = dict(w)
    for l in range(shape.n_layers):       # zero K/V projections: stored values are exact zeros
        w2[f"layers.{l}.wk"] = np.zeros_like(w[f"layers.{l}.wk"])
        w2[f"layers.{l}.wv"] = np.zeros_like(w[f"layers.{l}.wv"])
    om2 = T.OracleModel(shape, w2)
    assert np.array_equal(T.forward_full(om2, toks), T.forward_full(om2, toks, bf16_kv=True))


@pytest.mark.parametrize("scale", [1.0, 25.0])
def test_bf16_kv_cache_matches_torch_bfloat16_cache(scale):
    """The bf16 K/V reading, pinned against torch: an independent decoder whose
    cache holds torch.bfloat16(float32(k after RoPE)) and the same of v gives
    the oracle's bf16_kv logits to 1e-12 (rounding k before RoPE, rounding q,
    or skipping the float32 step each move them by far more)."""
    om, w = _model(scale=scale, seed=4)
    toks = _tokens(33, MINI.vocab, 9)
    got = T.forward_full(om, toks, bf16_kv=True)
    np.testing.assert_allclose(got, torch_logits(MINI, w, toks, bf16_kv=True), rtol=0, atol=1e-12)
    assert np.abs(got - torch_logits(MINI, w, toks)).max() > 1e-6     # the rounding is really there
