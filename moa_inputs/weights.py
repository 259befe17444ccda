"""Seeded random-init weights and the packed weight blob layout.

Every matrix (embedding and LM head included) is drawn i.i.d. N(0, 0.02^2),
one independent numpy stream per tensor keyed by
(seed, workload id, model id, tensor index). For bf16 workloads the fp32 draw
is rounded to bf16 with round-to-nearest-even; RMSNorm gains are exactly 1.

Blob layout (what the engine's weight loader accepts): tensors in the order
of ``TENSOR_NAMES``, each row-major ``[out, in]`` like ``nn.Linear.weight``,
packed back to back with no padding, every element in the storage dtype
(fp32: 4 bytes, bf16: 2 bytes, little endian).
"""
from concurrent.futures import ThreadPoolExecutor
import numpy as np

LAYER_TENSORS = ("attn_norm", "wq", "wk", "wv", "wo",
                 "mlp_norm", "w_gate", "w_up", "w_down")


def TENSOR_NAMES(n_layers):
    names = ["embed"]
    for l in range(n_layers):
        names += [f"layers.{l}.{t}" for t in LAYER_TENSORS]
    names += ["final_norm", "lm_head"]
    return names


def tensor_shapes(m):
    """(name, shape) in blob order for a ModelShape ``m``."""
    d, hd = m.d_model, m.head_dim
    per = {
        "attn_norm": (d,), "wq": (m.n_heads * hd, d), "wk": (m.n_kv_heads * hd, d),
        "wv": (m.n_kv_heads * hd, d), "wo": (d, m.n_heads * hd), "mlp_norm": (d,),
        "w_gate": (m.ffn_dim, d), "w_up": (m.ffn_dim, d), "w_down": (d, m.ffn_dim),
    }
    out = [("embed", (m.vocab, d))]
    for l in range(m.n_layers):
        out += [(f"layers.{l}.{t}", per[t]) for t in LAYER_TENSORS]
    out += [("final_norm", (d,)), ("lm_head", (m.vocab, d))]
    return out


def f32_to_bf16_bits(a):
    """Round float32 array to bf16 (round to nearest, ties to even); uint16 bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    rounding = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + rounding) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b):
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _draw(seed, wid, model_id, idx, name, shape, dtype):
    if name.endswith("norm"):
        a = np.ones(shape, dtype=np.float32)
    else:
        rng = np.random.default_rng([seed, wid, model_id, idx])
        a = rng.standard_normal(shape, dtype=np.float32)
        a *= np.float32(0.02)
    if dtype == "bf16":
        return f32_to_bf16_bits(a)
    return a


def generate_weights(model_shape, dtype, seed, wid, model_id, n_layers=None, threads=8):
    """Dict name -> array (float32, or uint16 bf16 bits). ``n_layers`` may
    truncate the depth (same streams for the layers that remain)."""
    m = model_shape
    shapes = tensor_shapes(m)
    if n_layers is not None and n_layers != m.n_layers:
        from dataclasses import replace
        m2 = replace(m, n_layers=n_layers)
        keep = {n for n, _ in tensor_shapes(m2)}
        # final_norm / lm_head keep their full-depth tensor index so the head
        # is the same matrix whatever the depth.
        shapes = [(n, s) for n, s in shapes if n in keep]
    index = {n: i for i, (n, _) in enumerate(tensor_shapes(m))}
    with ThreadPoolExecutor(max_workers=threads) as ex:
        futs = {n: ex.submit(_draw, seed, wid, model_id, index[n], n, s, dtype)
                for n, s in shapes}
        return {n: futs[n].result() for n, _ in shapes}


def pack_blob(weights, model_shape, n_layers=None):
    """Concatenate tensors in blob order into one contiguous numpy byte array."""
    from dataclasses import replace
    m = model_shape if n_layers is None else replace(model_shape, n_layers=n_layers)
    parts = [weights[n].reshape(-1).view(np.uint8) for n, _ in tensor_shapes(m)]
    return np.concatenate(parts)
