"""Adaptive aggregation (Eq. 11, Algorithm 1) and the submission order of the
host feeder: the confidence statistic against the values the paper states,
and the gated / reordered schedules against the oracle scheduler."""
from fractions import Fraction

import numpy as np
import pytest

from moa_inputs import CONFIGS, make_workload
from oracle.scheduler import OracleScheduler, c_vote, run_feeder as oracle_feeder
from paper_2606_03014_amd import run_feeder
from paper_2606_03014_amd.engine import expert_order, plurality
from tests.test_engine_host import _dry


# The paper's buckets for k = 3: 3:0 -> C = 1, 2:1 -> C = 2/3, 1:1:1 -> C = 1/3;
# k = 2 (top-2 routing): agreement -> 1, disagreement -> 1/2.
BUCKETS = [([7, 7, 7], Fraction(1)), ([7, 7, 2], Fraction(2, 3)), ([2, 7, 7], Fraction(2, 3)),
           ([1, 2, 3], Fraction(1, 3)), ([4, 4], Fraction(1)), ([4, 5], Fraction(1, 2)), ([9], Fraction(1))]


@pytest.mark.parametrize("answers,conf", BUCKETS)
def test_vote_confidence_buckets(answers, conf):
    assert c_vote(answers) == conf
    got, majority = plurality(answers)
    assert got == conf
    assert answers.count(majority) == max(answers.count(a) for a in answers)


def test_gate_thresholds_select_the_stated_buckets():
    """tau = 1 gates only unanimous votes; tau = 2/3 gates 3:0 and 2:1 (k = 3)."""
    votes = {"3:0": [1, 1, 1], "2:1": [1, 1, 0], "1:1:1": [0, 1, 2]}
    for tau, gated in ((1, {"3:0"}), (Fraction(2, 3), {"3:0", "2:1"}), (2 / 3, {"3:0", "2:1"})):
        tau_f = Fraction(tau).limit_denominator(64)
        assert {b for b, v in votes.items() if c_vote(v) >= tau_f} == gated
        assert {b for b, v in votes.items() if plurality(v)[0] >= tau_f} == gated


def _answers(name, nq, A, seed=3):
    """A seeded synthetic answer per (query, expert) in [0, A)."""
    rng = np.random.default_rng([seed, A])
    c = CONFIGS[name]
    return {(q, e): int(rng.integers(0, A)) for q in range(nq) for e in range(c.n_experts)}


def _gated_pair(name, nq, tau, A, order):
    c = CONFIGS[name]
    w = make_workload(name, 0, n_queries=nq)
    nm = c.n_experts + 1
    ans = _answers(name, w.n_queries, A)
    eng = _dry(c.model, c.engine, nm, c.dtype)
    r = run_feeder(eng, w, list(range(c.n_experts)), agg_model=c.n_experts, gate_tau=tau,
                   answer_of=lambda q, e, toks: ans[(q, e)], order=order)
    s = OracleScheduler(c.engine.num_kv_blocks, c.engine.max_num_seqs, c.engine.max_prefill_tokens, nm,
                        max_model_len=c.engine.max_model_len)
    calls = [(q, e, len(w.prompts[q]), G) for q, e, G in w.expert_requests()]
    if order == "longest-first":
        calls = [calls[i] for i in sorted(range(len(calls)), key=lambda i: (-calls[i][3], i))]
    log, rid_of = oracle_feeder(s, calls, agg_model=c.n_experts, agg_G=w.agg_max_new,
                                query_len=[len(p) for p in w.prompts], query_experts=w.experts,
                                gate_tau=tau, answers=ans)
    return w, ans, eng, r, s, log, rid_of


@pytest.mark.parametrize("name,nq,tau,A", [("tiny-moa-fp32", 16, 1, 2), ("moa-3+1x8b-bf16", 96, 1, 3),
                                           ("moa-3+1x8b-bf16", 96, 2 / 3, 3)])
def test_gated_schedule_matches_oracle(name, nq, tau, A):
    w, ans, eng, r, s, log, rid_of = _gated_pair(name, nq, tau, A, "first-seen")
    c = CONFIGS[name]
    assert np.array_equal(eng.steps(), np.array(s.steps, dtype=np.int64))
    assert [(a, list(b)) for a, b in r.collects] == [(a, list(b)) for a, b in log]
    agg = c.n_experts
    oracle_called = {q for (q, m) in rid_of if m == agg}
    engine_called = {q for (q, m) in r.rid_of if m == agg}
    assert engine_called == oracle_called
    assert r.agg_calls == len(engine_called)
    # the gate's own definition, query by query
    for q in range(w.n_queries):
        votes = [ans[(q, e)] for e in w.experts[q]]
        skipped = Fraction(max(votes.count(v) for v in votes), len(votes)) >= Fraction(tau).limit_denominator(64)
        assert (q in r.gated) == skipped and (q in engine_called) == (not skipped)
        if skipped:
            assert votes.count(r.gated[q]) == max(votes.count(v) for v in votes)
    assert 0 < len(r.gated) < w.n_queries


def test_longest_first_order_schedule_matches_oracle():
    w, ans, eng, r, s, log, rid_of = _gated_pair("moa-3+1x8b-bf16", 96, None, 3, "longest-first")
    assert np.array_equal(eng.steps(), np.array(s.steps, dtype=np.int64))
    assert [(a, list(b)) for a, b in r.collects] == [(a, list(b)) for a, b in log]
    Gs = [G for _, _, G in expert_order(w, "longest-first")]
    assert Gs == sorted(Gs, reverse=True)
