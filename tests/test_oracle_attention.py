"""Pins for the oracle's attention, RoPE, RMSNorm, argmax and bf16 rounding."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import transformer as T


def _rng(i=0):
    return np.random.default_rng([1234, i])


def test_single_key_returns_v_exactly():
    r = _rng(1)
    q = r.standard_normal((8, 16))
    K = r.standard_normal((1, 2, 16))
    V = r.standard_normal((1, 2, 16))
    out = T.attend(q, K, V)
    for h in range(8):
        assert np.array_equal(out[h], V[0, h // 4])


def test_identical_keys_average_v():
    r = _rng(2)
    q = r.standard_normal((4, 32))
    k = r.standard_normal((1, 1, 32))
    K = np.repeat(k, 37, axis=0)
    V = r.standard_normal((37, 1, 32))
    out = T.attend(q, K, V)
    for h in range(4):
        np.testing.assert_allclose(out[h], V[:, 0].mean(axis=0), rtol=0, atol=1e-14)


def test_softmax_rows_sum_to_one():
    r = _rng(3)
    s = r.standard_normal((50, 300)) * 30
    p = T.softmax(s)
    assert np.all(p >= 0)
    assert np.max(np.abs(p.sum(-1) - 1.0)) <= 1e-12


@pytest.mark.parametrize("n_h,n_kv", [(4, 4), (8, 2), (32, 8)])
def test_attend_matches_torch_sdpa_gqa(n_h, n_kv):
    """Library pin: torch's grouped-query SDPA (query head h reads KV head
    h // (n_h / n_kv)) on one query row against ctx keys."""
    r = _rng(4 + n_h)
    hd, ctx = 16, 23
    q = r.standard_normal((n_h, hd))
    K = r.standard_normal((ctx, n_kv, hd))
    V = r.standard_normal((ctx, n_kv, hd))
    ref = F.scaled_dot_product_attention(
        torch.from_numpy(q)[None, :, None, :],
        torch.from_numpy(K).permute(1, 0, 2)[None],
        torch.from_numpy(V).permute(1, 0, 2)[None], enable_gqa=True)[0, :, 0, :].numpy()
    np.testing.assert_allclose(T.attend(q, K, V), ref, rtol=0, atol=1e-13)


@pytest.mark.parametrize("start,T_,n_h,n_kv,block", [(0, 1, 4, 4, 512), (0, 37, 8, 2, 512),
                                                     (11, 37, 8, 2, 5), (300, 9, 32, 8, 4)])
def test_causal_attention_equals_attend_per_position(start, T_, n_h, n_kv, block):
    """The chunk attention of forward_chunk: row t against keys
    0..start+t, exactly attend() on that prefix (blocks of query rows and a
    chunk starting mid-sequence included)."""
    r = _rng(40 + start + T_)
    hd = 16
    q = r.standard_normal((T_, n_h, hd)) * 3
    K = r.standard_normal((start + T_, n_kv, hd))
    V = r.standard_normal((start + T_, n_kv, hd))
    got = T.causal_attention(q, K, V, start, block=block)
    for t in range(T_):
        np.testing.assert_allclose(got[t], T.attend(q[t], K[: start + t + 1], V[: start + t + 1]),
                                   rtol=0, atol=1e-13)


def test_causal_attention_first_position_returns_v():
    r = _rng(41)
    q = r.standard_normal((1, 8, 16))
    K = r.standard_normal((1, 2, 16))
    V = r.standard_normal((1, 2, 16))
    out = T.causal_attention(q, K, V, 0)
    for h in range(8):
        assert np.array_equal(out[0, h], V[0, h // 4])


def test_rope_identity_at_position_zero():
    r = _rng(5)
    x = r.standard_normal((1, 3, 64))
    c, s = T.rope_cos_sin([0], 64, 1e4)
    assert np.array_equal(T.apply_rope(x, c, s), x)


def test_rope_preserves_norm():
    r = _rng(6)
    x = r.standard_normal((5, 2, 128))
    c, s = T.rope_cos_sin([1, 7, 100, 5000, 37000], 128, 1e4)
    y = T.apply_rope(x, c, s)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)


def test_rope_scores_depend_on_relative_position_only():
    r = _rng(7)
    q = r.standard_normal((1, 1, 64))
    k = r.standard_normal((1, 1, 64))

    def score(m, n):
        cm, sm = T.rope_cos_sin([m], 64, 1e4)
        cn, sn = T.rope_cos_sin([n], 64, 1e4)
        return float(np.sum(T.apply_rope(q, cm, sm) * T.apply_rope(k, cn, sn)))

    assert abs(score(5, 2) - score(1003, 1000)) < 1e-11
    assert abs(score(9, 9) - float(np.sum(q * k))) < 1e-12
    assert abs(score(5, 2) - score(2, 5)) > 1e-3      # not symmetric in m - n


def test_rope_pairing_and_frequencies_closed_form():
    """Rotate-half pairs element i with i + hd/2 and turns pair i by
    pos * theta^(-2i/hd): unit vectors trace known circles."""
    hd, theta, p = 4, 1e4, 3.0
    c, s = T.rope_cos_sin([p], hd, theta)
    e0 = np.array([[[1.0, 0, 0, 0]]])
    e1 = np.array([[[0, 1.0, 0, 0]]])
    np.testing.assert_allclose(T.apply_rope(e0, c, s)[0, 0], [np.cos(p), 0, np.sin(p), 0], atol=1e-15)
    w = theta ** (-2.0 / hd)
    np.testing.assert_allclose(T.apply_rope(e1, c, s)[0, 0], [0, np.cos(w * p), 0, np.sin(w * p)], atol=1e-15)
    e2 = np.array([[[0, 0, 1.0, 0]]])
    np.testing.assert_allclose(T.apply_rope(e2, c, s)[0, 0], [-np.sin(p), 0, np.cos(p), 0], atol=1e-15)


def test_rmsnorm_matches_torch():
    r = _rng(8)
    x = r.standard_normal((6, 48)) * 3
    g = r.standard_normal(48)
    ref = F.rms_norm(torch.from_numpy(x), (48,), weight=torch.from_numpy(g), eps=1e-5).numpy()
    np.testing.assert_allclose(T.rmsnorm(x, g, 1e-5), ref, rtol=1e-14, atol=1e-14)


def test_silu_matches_torch():
    x = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(T.silu(x), F.silu(torch.from_numpy(x)).numpy(), rtol=1e-14, atol=1e-300)


def test_argmax_ties_to_lowest_id():
    assert T.argmax_lowest(np.zeros(4096)) == 0
    v = np.array([0.5, 2.0, -1.0, 2.0, 2.0])
    assert T.argmax_lowest(v) == 1
    v = np.full(10, -3.0)
    v[7] = -2.0
    assert T.argmax_lowest(v) == 7


def test_bf16_round_matches_torch():
    r = _rng(9)
    x = np.concatenate([r.standard_normal(10000) * 10.0 ** r.integers(-6, 6, 10000),
                        [0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.0e38]])
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(T.bf16_round(x), ref)
