"""An independent float64 decoder built from torch library primitives.

Used only to pin the oracle: attention is torch's scaled_dot_product_attention
(causal, grouped-query), RMSNorm is torch.nn.functional.rms_norm, SiLU is
torch.nn.functional.silu, and RoPE is written as a complex rotation
(pairs (i, i + hd/2) viewed as one complex number multiplied by
exp(1j * pos * theta^(-2i/hd))), a different formulation from the oracle's
real-valued rotate-half. With bf16_kv the cache values go through
torch.bfloat16 (via float32), torch's own rounding.
"""
import numpy as np
import torch
import torch.nn.functional as F


def _t(a):
    if a.dtype == np.uint16:
        a = (a.astype(np.uint32) << 16).view(np.float32)
    return torch.from_numpy(np.ascontiguousarray(a)).to(torch.float64)


def _rope_complex(x, pos, theta):
    # x: [H, T, hd]
    hd = x.shape[-1]
    half = hd // 2
    freqs = theta ** (-(torch.arange(0, hd, 2, dtype=torch.float64)) / hd)
    ang = torch.outer(pos.to(torch.float64), freqs)               # [T, half]
    rot = torch.polar(torch.ones_like(ang), ang)                  # e^{i ang}
    z = torch.complex(x[..., :half], x[..., half:]) * rot
    return torch.cat([z.real, z.imag], dim=-1)


def _bf16(x):
    """Round to bf16 through float32, both nearest-even, back to float64."""
    return x.to(torch.float32).to(torch.bfloat16).to(torch.float64)


def torch_logits(shape, weights, tokens, n_layers=None, bf16_kv=False):
    """Logits at every position. bf16_kv: the K/V cache holds bf16 values --
    k after RoPE and v are rounded to bf16 once, q never."""
    L = shape.n_layers if n_layers is None else n_layers
    d, nh, nkv, hd = shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim
    eps = shape.rms_eps
    tok = torch.as_tensor(np.asarray(tokens, dtype=np.int64))
    T = tok.shape[0]
    pos = torch.arange(T)
    x = _t(weights["embed"])[tok]
    for l in range(L):
        W = lambda n: _t(weights[f"layers.{l}.{n}"])
        xn = F.rms_norm(x, (d,), weight=W("attn_norm"), eps=eps)
        q = (xn @ W("wq").T).view(T, nh, hd).transpose(0, 1)
        k = (xn @ W("wk").T).view(T, nkv, hd).transpose(0, 1)
        v = (xn @ W("wv").T).view(T, nkv, hd).transpose(0, 1)
        q = _rope_complex(q, pos, shape.rope_theta)
        k = _rope_complex(k, pos, shape.rope_theta)
        if bf16_kv:
            k, v = _bf16(k), _bf16(v)
        a = F.scaled_dot_product_attention(q[None], k[None], v[None], is_causal=True,
                                           enable_gqa=True)[0]
        h = x + a.transpose(0, 1).reshape(T, nh * hd) @ W("wo").T
        hn = F.rms_norm(h, (d,), weight=W("mlp_norm"), eps=eps)
        x = h + (F.silu(hn @ W("w_gate").T) * (hn @ W("w_up").T)) @ W("w_down").T
    xf = F.rms_norm(x, (d,), weight=_t(weights["final_norm"]), eps=eps)
    return (xf @ _t(weights["lm_head"]).T).numpy()
