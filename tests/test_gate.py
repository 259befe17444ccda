"""Adaptive aggregation (Eq. 11, Algorithm 1) and the submission order of the
host feeder: the confidence statistic against the values the paper states,
and the gated / reordered schedules against the oracle scheduler."""
import dataclasses
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


def _gated_pair(name, nq, tau, A, order, window=None, consts=None, on_step=None):
    c = CONFIGS[name]
    consts = consts or c.engine
    w = make_workload(name, 0, n_queries=nq)
    nm = c.n_experts + 1
    ans = _answers(name, w.n_queries, A)
    eng = _dry(c.model, consts, nm, c.dtype)
    r = run_feeder(eng, w, list(range(c.n_experts)), agg_model=c.n_experts, gate_tau=tau,
                   answer_of=lambda q, e, toks: ans[(q, e)], order=order, window=window, on_step=on_step)
    s = OracleScheduler(consts.num_kv_blocks, consts.max_num_seqs, consts.max_prefill_tokens, nm,
                        max_model_len=consts.max_model_len)
    calls = [(q, e, len(w.prompts[q]), G) for q, e, G in w.expert_requests()]
    if order == "longest-first":
        calls = [calls[i] for i in sorted(range(len(calls)), key=lambda i: (-calls[i][3], i))]
    log, rid_of = oracle_feeder(s, calls, agg_model=c.n_experts, agg_G=w.agg_max_new,
                                query_len=[len(p) for p in w.prompts], query_experts=w.experts,
                                gate_tau=tau, answers=ans, window=window)
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


# A KV pool of 12,000 blocks holds only ~55 of the 3+1x8B calls at once, so
# admission is the bottleneck and the submission window decides which calls
# wait: the schedule pressure of the full workload at a size the CPU plans fast.
def _tight(name):
    return dataclasses.replace(CONFIGS[name].engine, num_kv_blocks=12000)


@pytest.mark.parametrize("window", [1, 7, 64])
@pytest.mark.parametrize("order", ["first-seen", "longest-first"])
def test_windowed_feeder_schedule_matches_oracle(window, order):
    """The submission window (aggregator calls overtake expert calls not yet
    submitted): every step's bookkeeping, every collect and every request id
    agree with the oracle scheduler's feeder."""
    pend = []
    w, ans, eng, r, s, log, rid_of = _gated_pair("moa-3+1x8b-bf16", 96, None, 3, order, window=window,
                                                 consts=_tight("moa-3+1x8b-bf16"),
                                                 on_step=lambda info: pend.append(info.pending))
    assert np.array_equal(eng.steps(), np.array(s.steps, dtype=np.int64))
    assert [(a, list(b)) for a, b in r.collects] == [(a, list(b)) for a, b in log]
    assert r.rid_of == rid_of
    assert r.agg_calls == w.n_queries and len(rid_of) == 3 * w.n_queries
    # after a step's admissions, what still waits is at most the window plus
    # the aggregator calls submitted since the previous top-up
    assert max(pend) <= window + w.n_queries


def test_window_lets_aggregation_overtake_the_expert_backlog():
    """Under admission pressure a window admits aggregator calls long before
    the expert backlog drains: with every call submitted up front the first
    aggregator waits behind all expert calls, with W = 8 it does not."""
    first_agg = {}
    for window in (None, 8):
        w, ans, eng, r, s, log, rid_of = _gated_pair("moa-3+1x8b-bf16", 96, None, 3, "first-seen",
                                                     window=window, consts=_tight("moa-3+1x8b-bf16"))
        agg = [eng.request(rid).admit_step for (q, m), rid in r.rid_of.items() if m == 3]
        last_expert = max(eng.request(rid).admit_step for (q, m), rid in r.rid_of.items() if m != 3)
        first_agg[window] = (min(agg), last_expert)
    assert first_agg[None][0] > first_agg[None][1]        # FIFO: after the last expert admission
    assert first_agg[8][0] < first_agg[8][1]              # window: well before it


def test_schedule_study_runs_without_a_gpu():
    """bench.py --schedule-study plans every (order, window, budget) with the
    engine's scheduler and no device; its window-free first-seen row is the
    plain feeder's schedule."""
    import json
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    out = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--workload", "tiny-moa-fp32",
                          "--schedule-study"], capture_output=True, text=True, timeout=300, cwd=root)
    assert out.returncode == 0, out.stderr
    d = json.loads(out.stdout.strip().splitlines()[-1])
    rows = d["schedule_study"]
    assert len(rows) == 2 * 4 * 3
    c = CONFIGS["tiny-moa-fp32"]
    w = make_workload("tiny-moa-fp32", 0)
    eng = _dry(c.model, dataclasses.replace(c.engine, max_prefill_tokens=16384), c.n_experts + 1, c.dtype)
    r = run_feeder(eng, w, list(range(c.n_experts)), agg_model=c.n_experts)
    base = [x for x in rows if x["order"] == "first-seen" and x["window"] is None and x["prefill_budget"] == 16384]
    assert base[0]["steps"] == r.n_steps
    assert all(x["model_s"] > 0 and x["steps"] > 0 for x in rows)
