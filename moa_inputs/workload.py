"""Seeded synthetic MoA workloads (stand-ins for the paper's benchmark suites).

The paper measures on multiple-choice benchmark suites that are not shipped
here; none of their items is reproduced. What these draws keep from the paper
is the *shape* of its workload (Sections "Motivation" and "Workload
Characterisation"): every query goes to several experts chosen by a skewed
popularity (Observation 2), and reasoning-style experts emit far longer and
heavier-tailed outputs than instruction-style ones (Observation 1).

Each quantity has its own stream keyed by (seed, workload id, stream id), so a
change in one draw never shifts another.
"""
from dataclasses import dataclass
import numpy as np

from .configs import CONFIGS

_S_PLEN, _S_TOK, _S_ROUTE, _S_GEN, _S_SEG = 1, 2, 3, 4, 5


def _lognormal_len(rng, median, sigma, lo, hi):
    z = rng.standard_normal()
    return int(np.clip(np.rint(median * np.exp(sigma * z)), lo, hi))


def _draw_len(rng, spec):
    kind = spec[0]
    if kind == "uniform":
        return int(rng.integers(spec[1], spec[2] + 1))
    if kind == "lognormal":
        return _lognormal_len(rng, *spec[1:])
    raise ValueError(spec)


def _draw_gen(rng, mixture):
    """mixture: tuple of ("uniform", weight, lo, hi) | ("lognormal", weight, median, sigma, lo, hi)."""
    u = rng.random()
    acc = 0.0
    for comp in mixture:
        acc += comp[1]
        if u < acc or comp is mixture[-1]:
            if comp[0] == "uniform":
                return int(rng.integers(comp[2], comp[3] + 1))
            return _lognormal_len(rng, *comp[2:])
    raise AssertionError


@dataclass
class Workload:
    """Queries, their experts (ascending ids) and per-(query, expert) budgets."""
    name: str
    seed: int
    prompts: list                   # list of int32 arrays
    experts: list                   # list of tuples of expert ids, ascending
    max_new: dict                   # (q, e) -> G
    n_experts: int
    aggregator_id: int = -1         # model id of the aggregator, -1 if none
    agg_max_new: int = 0

    @property
    def n_queries(self):
        return len(self.prompts)

    def expert_requests(self):
        """(q, e, G) in first-seen order: queries ascending, experts ascending."""
        return [(q, e, self.max_new[(q, e)]) for q in range(self.n_queries)
                for e in self.experts[q]]

    def total_expert_tokens(self):
        return sum(self.max_new.values())


def make_workload(name, seed=0, n_queries=None):
    c = CONFIGS[name]
    nq = c.n_queries if n_queries is None else n_queries
    V = c.model.vocab
    r_len = np.random.default_rng([seed, c.wid, _S_PLEN])
    r_tok = np.random.default_rng([seed, c.wid, _S_TOK])
    r_route = np.random.default_rng([seed, c.wid, _S_ROUTE])
    r_gen = np.random.default_rng([seed, c.wid, _S_GEN])

    prompts, experts = [], []
    for q in range(nq):
        if c.prompt[0] == "segments":
            head, nseg, lo, hi = c.prompt[1:]
            P = head + sum(int(r_len.integers(lo, hi + 1)) for _ in range(nseg))
        else:
            P = _draw_len(r_len, c.prompt)
        prompts.append(r_tok.integers(0, V, size=P, dtype=np.int32))
        if c.route[0] == "all":
            experts.append(tuple(range(c.n_experts)))
        elif c.route[0] == "zipf_top2":
            s = c.route[1]
            w = np.arange(1, c.n_experts + 1, dtype=np.float64) ** (-s)
            w /= w.sum()
            pick = r_route.choice(c.n_experts, 2, replace=False, p=w)
            experts.append(tuple(sorted(int(x) for x in pick)))
        elif c.route[0] == "none":
            experts.append(())
        else:
            raise ValueError(c.route)
    max_new = {}
    for q in range(nq):
        for e in experts[q]:
            max_new[(q, e)] = _draw_gen(r_gen, c.gen)
    return Workload(name=name, seed=seed, prompts=prompts, experts=experts,
                    max_new=max_new, n_experts=c.n_experts,
                    aggregator_id=c.n_experts if c.aggregator else -1,
                    agg_max_new=c.agg_max_new)


@dataclass
class StragglerWorkload:
    """Long-reasoning straggler stress: sequences that arrive with a KV
    history already in place and decode their remaining budget.

    Sequence ``i`` has a KV length L ~ min(floor(256 * (1 + Pareto(1.2))), 32768)
    (classical Pareto with scale 256, clipped at 32768), a seed token uniform
    over the vocabulary and a remaining budget R ~ U[1, 512]."""
    name: str
    seed: int
    n_live: int
    refill_steps: int
    vocab: int
    alpha: float = 1.2
    scale: int = 256
    cap: int = 32768
    r_lo: int = 1
    r_hi: int = 512
    wid: int = 4

    def sequence(self, i):
        rng = np.random.default_rng([self.seed, self.wid, _S_SEG, i])
        L = int(min(np.floor(self.scale * (1.0 + rng.pareto(self.alpha))), self.cap))
        tok = int(rng.integers(0, self.vocab))
        R = int(rng.integers(self.r_lo, self.r_hi + 1))
        return L, tok, R


def make_straggler_workload(seed=0, n_live=None, refill_steps=None):
    c = CONFIGS["straggler-8b-bf16"]
    return StragglerWorkload(name=c.name, seed=seed,
                             n_live=c.n_queries if n_live is None else n_live,
                             refill_steps=c.extra["refill_steps"] if refill_steps is None else refill_steps,
                             vocab=c.model.vocab, alpha=c.prompt[1], scale=c.prompt[2],
                             cap=c.prompt[3], r_lo=c.gen[0][2], r_hi=c.gen[0][3], wid=c.wid)


def synthetic_kv(seed, seq_index, n_layers, ctx, n_kv, head_dim):
    """Seeded N(0,1) K/V history for an injected sequence, float32
    [n_layers, 2, ctx, n_kv, head_dim] (K then V). Callers round to the
    storage type."""
    rng = np.random.default_rng([seed, 4, 6, seq_index])
    return rng.standard_normal((n_layers, 2, ctx, n_kv, head_dim), dtype=np.float32)
