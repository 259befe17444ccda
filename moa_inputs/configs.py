"""The five synthetic MoA workloads: model geometry, engine constants, draws.

Every workload is named by what it is. The integer ``wid`` only keys the
random streams so that two workloads never share a draw.

Readings fixed here (the paper states none of them, it runs trained
checkpoints under vLLM):
  * decoder: pre-norm, RMSNorm with unit gain, no biases, untied LM head,
    rotate-half RoPE with theta = 1e4, SwiGLU MLP, eps = 1e-5;
  * KV block = 16 token slots in every workload;
  * lognormal lengths are clip(rint(median * exp(sigma * z)), lo, hi) with
    sigma = 1 (the paper gives means and ranges, not a shape).
"""
from dataclasses import dataclass, field, asdict


@dataclass(frozen=True)
class ModelShape:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rope_theta: float = 10000.0
    rms_eps: float = 1e-5

    @property
    def qkv_dim(self):
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    def n_params(self):
        d, L = self.d_model, self.n_layers
        per_layer = (2 * d + d * self.qkv_dim + self.n_heads * self.head_dim * d
                     + 3 * d * self.ffn_dim)
        return 2 * self.vocab * d + L * per_layer + d


@dataclass(frozen=True)
class EngineConsts:
    num_kv_blocks: int
    max_num_seqs: int
    max_prefill_tokens: int
    max_model_len: int
    kv_block_size: int = 16


TINY = ModelShape(2, 256, 4, 4, 64, 1024, 4096)
LLAMA_1B = ModelShape(16, 2048, 32, 8, 64, 8192, 32000)
LLAMA_8B = ModelShape(32, 4096, 32, 8, 128, 14336, 128256)


@dataclass(frozen=True)
class WorkloadConfig:
    name: str
    wid: int
    dtype: str                 # "f32" or "bf16": storage/compute type of the engine
    model: ModelShape
    n_experts: int             # expert models (ids 0..n_experts-1)
    aggregator: bool           # an extra model (id n_experts) aggregates
    agg_max_new: int
    n_queries: int
    prompt: tuple              # ("uniform", lo, hi) | ("lognormal", median, sigma, lo, hi)
    route: tuple               # ("all",) | ("zipf_top2", s)
    gen: tuple                 # mixture spec, see workload.py
    engine: EngineConsts
    extra: dict = field(default_factory=dict)

    def as_dict(self):
        d = asdict(self)
        return d


CONFIGS = {
    "tiny-moa-fp32": WorkloadConfig(
        name="tiny-moa-fp32", wid=1, dtype="f32", model=TINY,
        n_experts=2, aggregator=True, agg_max_new=32, n_queries=16,
        prompt=("uniform", 16, 64), route=("all",),
        gen=(("uniform", 1.0, 8, 64),),
        engine=EngineConsts(num_kv_blocks=128, max_num_seqs=16,
                            max_prefill_tokens=256, max_model_len=256)),
    "moa-4x1b-bf16": WorkloadConfig(
        name="moa-4x1b-bf16", wid=2, dtype="bf16", model=LLAMA_1B,
        n_experts=4, aggregator=False, agg_max_new=0, n_queries=256,
        prompt=("lognormal", 200, 1.0, 32, 2048), route=("zipf_top2", 1.2),
        gen=(("uniform", 0.7, 64, 512), ("lognormal", 0.3, 2048, 1.0, 1, 8192)),
        engine=EngineConsts(num_kv_blocks=262144, max_num_seqs=512,
                            max_prefill_tokens=16384, max_model_len=10240)),
    "moa-3+1x8b-bf16": WorkloadConfig(
        name="moa-3+1x8b-bf16", wid=3, dtype="bf16", model=LLAMA_8B,
        n_experts=3, aggregator=True, agg_max_new=512, n_queries=1024,
        prompt=("lognormal", 512, 1.0, 64, 4096), route=("zipf_top2", 1.0),
        gen=(("uniform", 0.6, 128, 1024), ("lognormal", 0.4, 4096, 1.0, 1, 16384)),
        engine=EngineConsts(num_kv_blocks=100000, max_num_seqs=1024,
                            max_prefill_tokens=16384, max_model_len=37376)),
    "straggler-8b-bf16": WorkloadConfig(
        name="straggler-8b-bf16", wid=4, dtype="bf16", model=LLAMA_8B,
        n_experts=1, aggregator=False, agg_max_new=0, n_queries=512,
        prompt=("pareto", 1.2, 256, 32768), route=("all",),
        gen=(("uniform", 1.0, 1, 512),),
        engine=EngineConsts(num_kv_blocks=120000, max_num_seqs=512,
                            max_prefill_tokens=0, max_model_len=33280),
        extra={"refill_steps": 512}),
    "agg-prefill-8b-bf16": WorkloadConfig(
        name="agg-prefill-8b-bf16", wid=5, dtype="bf16", model=LLAMA_8B,
        n_experts=0, aggregator=True, agg_max_new=256, n_queries=64,
        prompt=("segments", 256, 4, 512, 8192), route=("none",),
        gen=(),
        engine=EngineConsts(num_kv_blocks=120000, max_num_seqs=64,
                            max_prefill_tokens=16384, max_model_len=33280)),
}


def config(name):
    return CONFIGS[name]
