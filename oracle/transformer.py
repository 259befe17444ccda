"""Oracle transformer: plain, slow, fp64 CPU reference of what each expert call computes.

TEST INFRASTRUCTURE ONLY. Nothing in the product path (the HIP engine and
its Python binding) may import this module; only the tests, the package's
smoke check and the CPU-baseline leg of the benchmark do.

What is computed. In the paper's setting (Section "Problem Setting") every
routed (query, expert) pair is an independent model call, and the aggregator
call runs the same way on the query followed by the expert outputs (Section
"MOSAIC: Adaptive Aggregation", Eq. 11's Aggregator(q, {a_i})). Batching,
paging and chunking are the engine's performance devices, not part of the
result. So the oracle is the per-request definition: greedy decoding of
exactly G tokens by a Llama-style pre-norm decoder,

    x   = E[tok]
    h   = x + Wo . Attn(RoPE(Wq n(x)), RoPE(Wk n(x)), Wv n(x))
    x'  = h + Wdown . (silu(Wgate n(h)) * Wup n(h))
    logits = Wlm . n(x_L)

with n() RMSNorm (unit gain stored in the weights), causal softmax attention
scaled by 1/sqrt(head_dim), grouped-query attention (query head h reads KV
head floor(h / (n_heads / n_kv_heads))), rotate-half RoPE with angles
pos * theta^(-2i/head_dim), and argmax with ties broken to the lowest id.

All arithmetic is float64 (weights are upcast from their fp32 or bf16
storage). ``bf16_kv=True`` models a model state whose KV cache is stored in
bf16: k (after RoPE) and v are rounded to bf16 (nearest-even) when they are
written to the cache, exactly once; everything else stays float64.

Parity pins (tests/test_oracle_*.py): single-key attention returns V, equal
keys average V, softmax rows sum to 1, the blockwise causal attention of a
chunk equals attend() position by position, RoPE is the identity at position 0 and
norm-preserving with relative-position scores, paged == contiguous KV bit for
bit, cached decode == brute-force prefix recompute, the zero-layer model
equals the closed form Wlm . n(E[t]), and a torch float64 functional model
built from library primitives (scaled_dot_product_attention) agrees.
"""
import numpy as np


# ----------------------------------------------------------------- helpers

def bf16_round(a):
    """Round float64 values to the nearest bf16 (ties to even), returned as float64.
    Goes through float32 first (the engine rounds fp32 values)."""
    f = np.ascontiguousarray(a, dtype=np.float32)
    u = f.view(np.uint32)
    r = ((u >> 16) & 1) + np.uint32(0x7FFF)
    out = ((u + r) & np.uint32(0xFFFF0000)).view(np.float32)
    return out.astype(np.float64)


def to_f64(arr):
    """Upcast a stored tensor (float32, or uint16 holding bf16 bits) to float64."""
    if arr.dtype == np.uint16:
        return (arr.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(arr, dtype=np.float64)


def rmsnorm(x, g, eps):
    """y = x / sqrt(mean(x^2) + eps) * g over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope_cos_sin(positions, head_dim, theta):
    """cos/sin of pos * theta^(-2i/head_dim), i < head_dim/2, in float64."""
    half = head_dim // 2
    inv = theta ** (-(2.0 * np.arange(half, dtype=np.float64)) / head_dim)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv[None, :]
    return np.cos(ang), np.sin(ang)


def apply_rope(x, cos, sin):
    """Rotate-half RoPE. x: [T, H, hd]; cos/sin: [T, hd/2]. Pairs (i, i + hd/2)."""
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def softmax(s):
    """Row softmax over the last axis (max-subtracted)."""
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def attend(q, K, V):
    """One query position against ctx keys.
    q: [n_h, hd]; K, V: [ctx, n_kv, hd] -> out [n_h, hd]."""
    n_h, hd = q.shape
    n_kv = K.shape[1]
    group = n_h // n_kv
    out = np.empty_like(q)
    for h in range(n_h):
        kv = h // group
        s = K[:, kv, :] @ q[h] / np.sqrt(hd)
        p = softmax(s)
        out[h] = p @ V[:, kv, :]
    return out


def causal_attention(q, K, V, start, block=512):
    """Causal attention of a chunk of query positions, all heads at once.

    q: [T, n_h, hd] at positions start .. start + T - 1; K, V: the cache,
    [start + T, n_kv, hd]. Row t attends to keys 0 .. start + t (the same
    masked softmax(q . k / sqrt(hd)) . v as attend(), which defines it;
    evaluated one block of query rows and one head at a time, so long
    prompts cost a few library matmuls instead of a Python loop per
    position). Returns [T, n_h, hd]."""
    T, n_h, hd = q.shape
    n_kv = K.shape[1]
    group = n_h // n_kv
    out = np.empty_like(q)
    for b0 in range(0, T, block):
        b1 = min(T, b0 + block)
        kmax = start + b1                                    # keys this block can see
        pos = start + np.arange(b0, b1)                      # query positions
        future = np.arange(kmax)[None, :] > pos[:, None]     # key index past the query's position
        for h in range(n_h):
            kv = h // group
            s = q[b0:b1, h, :] @ K[:kmax, kv, :].T / np.sqrt(hd)
            s[future] = -np.inf
            out[b0:b1, h, :] = softmax(s) @ V[:kmax, kv, :]
    return out


def silu(x):
    return x / (1.0 + np.exp(-x))


def argmax_lowest(logits):
    """Greedy token: the largest logit, ties to the lowest token id."""
    return int(np.argmax(logits))       # numpy returns the first maximal index


# ------------------------------------------------------------------- model

class OracleModel:
    """Holds one model's weights (storage dtype) and upcasts on use.

    ``weights`` maps blob tensor names to arrays (float32 or uint16 bf16 bits).
    With ``cache=True`` the float64 copies are kept (fast for small models)."""

    def __init__(self, shape, weights, n_layers=None, cache=True):
        self.shape = shape
        self.n_layers = shape.n_layers if n_layers is None else n_layers
        self.w = weights
        self.cache = cache
        self._f64 = {}

    def W(self, name):
        if name in self._f64:
            return self._f64[name]
        a = to_f64(self.w[name])
        if self.cache:
            self._f64[name] = a
        return a


class ContiguousKV:
    """Per-layer K/V history in position order: [ctx, n_kv, hd] float64."""

    def __init__(self, n_layers, n_kv, hd):
        self.K = [np.zeros((0, n_kv, hd)) for _ in range(n_layers)]
        self.V = [np.zeros((0, n_kv, hd)) for _ in range(n_layers)]

    def write(self, layer, start, k, v):
        assert start == self.K[layer].shape[0], "contiguous cache grows in order"
        self.K[layer] = np.concatenate([self.K[layer], k], axis=0)
        self.V[layer] = np.concatenate([self.V[layer], v], axis=0)

    def read(self, layer, ctx):
        return self.K[layer][:ctx], self.V[layer][:ctx]


class PagedKV:
    """K/V in fixed-size blocks of ``block_size`` slots taken from a shared pool;
    position p lives in block ``table[p // block_size]`` at slot ``p % block_size``
    (the paged layout of the engine, written out plainly)."""

    def __init__(self, pool, table, block_size):
        self.pool = pool                  # [NB, n_layers, 2, block_size, n_kv, hd]
        self.table = list(table)
        self.bs = block_size

    @staticmethod
    def make_pool(num_blocks, n_layers, n_kv, hd, block_size):
        return np.full((num_blocks, n_layers, 2, block_size, n_kv, hd), np.nan)

    def write(self, layer, start, k, v):
        for i in range(k.shape[0]):
            p = start + i
            b = self.table[p // self.bs]
            self.pool[b, layer, 0, p % self.bs] = k[i]
            self.pool[b, layer, 1, p % self.bs] = v[i]

    def read(self, layer, ctx):
        K = np.stack([self.pool[self.table[p // self.bs], layer, 0, p % self.bs] for p in range(ctx)])
        V = np.stack([self.pool[self.table[p // self.bs], layer, 1, p % self.bs] for p in range(ctx)])
        return K, V


def forward_chunk(model, tokens, start, kv, bf16_kv=False, want="all"):
    """Run positions [start, start + len(tokens)) through the model, appending
    their K/V to ``kv`` (whose first ``start`` positions must already hold the
    history). Each position attends causally to positions <= itself.
    Returns logits [len(tokens), vocab]; ``want="last"`` returns only the last
    row, an integer ``want=j`` only rows j.. (the others are not computed)."""
    m = model.shape
    n_h, n_kv, hd = m.n_heads, m.n_kv_heads, m.head_dim
    store = bf16_round if bf16_kv else (lambda a: a)
    toks = np.asarray(tokens, dtype=np.int64)
    T = toks.shape[0]
    pos = np.arange(start, start + T)
    cos, sin = rope_cos_sin(pos, hd, m.rope_theta)
    E = model.W("embed")
    x = E[toks].copy()
    for l in range(model.n_layers):
        p = f"layers.{l}."
        xn = rmsnorm(x, model.W(p + "attn_norm"), m.rms_eps)
        q = (xn @ model.W(p + "wq").T).reshape(T, n_h, hd)
        k = (xn @ model.W(p + "wk").T).reshape(T, n_kv, hd)
        v = (xn @ model.W(p + "wv").T).reshape(T, n_kv, hd)
        q = apply_rope(q, cos, sin)
        k = store(apply_rope(k, cos, sin))
        v = store(v)
        kv.write(l, start, k, v)
        K, V = kv.read(l, start + T)
        att = causal_attention(q, K, V, start).reshape(T, n_h * hd)
        h = x + att @ model.W(p + "wo").T
        hn = rmsnorm(h, model.W(p + "mlp_norm"), m.rms_eps)
        g = hn @ model.W(p + "w_gate").T
        u = hn @ model.W(p + "w_up").T
        a = silu(g) * u
        x = h + a @ model.W(p + "w_down").T
    if want == "last":
        x = x[-1:]
    elif not isinstance(want, str):
        x = x[want:]
    xf = rmsnorm(x, model.W("final_norm"), m.rms_eps)
    return xf @ model.W("lm_head").T


def forward_full(model, tokens, bf16_kv=False, first=0):
    """Logits at positions first.. of ``tokens`` computed from scratch (no prior cache)."""
    kv = ContiguousKV(model.n_layers, model.shape.n_kv_heads, model.shape.head_dim)
    return forward_chunk(model, tokens, 0, kv, bf16_kv, want=first)


def brute_force_prefix_logits(model, tokens, bf16_kv=False):
    """Logits at position t recomputed from tokens[0..t] alone, for every t
    (quadratic cost; tiny inputs only)."""
    return np.stack([forward_full(model, tokens[: t + 1], bf16_kv)[-1]
                     for t in range(len(tokens))])


def greedy_generate(model, prompt, G, kv=None, bf16_kv=False, return_logits=False):
    """Greedy decoding of exactly G tokens (no end-of-sequence token).
    The prompt is prefilled in one chunk; each later token is one decode step."""
    m = model.shape
    if kv is None:
        kv = ContiguousKV(model.n_layers, m.n_kv_heads, m.head_dim)
    P = len(prompt)
    lg = forward_chunk(model, prompt, 0, kv, bf16_kv, want="last")[-1]
    out, logits = [argmax_lowest(lg)], [lg]
    for j in range(1, G):
        lg = forward_chunk(model, [out[-1]], P + j - 1, kv, bf16_kv)[-1]
        out.append(argmax_lowest(lg))
        logits.append(lg)
    if return_logits:
        return out, np.stack(logits)
    return out


def teacher_forced_logits(model, prompt, outputs, bf16_kv=False):
    """Logits that produce each of ``outputs`` when the history is the prompt
    followed by the given outputs (so a flip never cascades): rows are the
    positions P-1 .. P+G-2 of prompt ++ outputs[:-1]."""
    seq = np.concatenate([np.asarray(prompt, dtype=np.int64),
                          np.asarray(outputs[:-1], dtype=np.int64)])
    return forward_full(model, seq, bf16_kv, first=len(prompt) - 1)


def decode_from_history(model, K_hist, V_hist, token, pos, bf16_kv=False):
    """One decode step for a sequence whose K/V at positions [0, pos) is given
    (per layer [pos, n_kv, hd]); returns the logits of ``token`` at ``pos``."""
    m = model.shape
    kv = ContiguousKV(model.n_layers, m.n_kv_heads, m.head_dim)
    for l in range(model.n_layers):
        kv.K[l] = np.asarray(K_hist[l], dtype=np.float64)
        kv.V[l] = np.asarray(V_hist[l], dtype=np.float64)
    return forward_chunk(model, [token], pos, kv, bf16_kv)[-1]
