"""Pins for the oracle scheduler: hand traces, invariants, workload identities."""
import json
import os

import numpy as np
import pytest

from moa_inputs import CONFIGS, make_workload
from oracle.scheduler import OracleScheduler, SchedError, run_feeder

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "step_rule_examples.json")))


def _run_example(ex):
    s = OracleScheduler(ex["num_blocks"], ex["max_num_seqs"], ex["max_prefill_tokens"], ex["n_models"])
    for kind, m, a, b in ex["submit"]:
        (s.submit if kind == "std" else s.submit_injected)(m, a, b)
    while s.step() is not None:
        pass
    return s


@pytest.mark.parametrize("ex", GOLD["examples"], ids=lambda e: e["name"])
def test_hand_traced_examples(ex):
    s = _run_example(ex)
    assert len(s.steps) == ex["n_steps"]
    assert [list(t) for t in s.steps[: len(ex["steps_head"])]] == ex["steps_head"]
    for r, want in zip(s.reqs, ex["requests"]):
        assert r.admit_step == want["admit"]
        assert r.finish_step == want["finish"]
        assert r.blocks == want["blocks"]
        assert [list(c) for c in r.chunks] == want["chunks"]
    if "last_slot" in ex:
        ls = ex["last_slot"]
        r = s.reqs[ls["request"]]
        assert r.P + r.G - 2 == ls["position"]
        assert r.blocks[ls["position"] // 16] == ls["block"] and ls["position"] % 16 == ls["offset"]


def test_hand_traced_feeder():
    f = GOLD["feeder"]
    s = OracleScheduler(f["num_blocks"], f["max_num_seqs"], f["max_prefill_tokens"], f["n_models"])
    calls = [(q, e, qq["P"], G) for q, qq in enumerate(f["queries"]) for e, G in qq["experts"]]
    log, _ = run_feeder(s, calls, agg_model=f["aggregator"], agg_G=f["agg_G"],
                        query_len=[qq["P"] for qq in f["queries"]],
                        query_experts=[tuple(e for e, _ in qq["experts"]) for qq in f["queries"]])
    assert [list(t) for t in s.steps] == f["steps"]
    assert [[a, list(b)] for a, b in log] == f["collects"]
    for r, want in zip(s.reqs, f["requests"]):
        assert (r.expert, r.P, r.G, r.admit_step, r.finish_step, r.blocks) == (
            want["model"], want["P"], want["G"], want["admit"], want["finish"], want["blocks"])


def test_hand_traced_windowed_feeder():
    """The feeder's submission window, traced by hand: with W = 1 the
    aggregator calls of q0 and q1 overtake q2's unsubmitted expert call."""
    f = GOLD["feeder_window"]
    s = OracleScheduler(f["num_blocks"], f["max_num_seqs"], f["max_prefill_tokens"], f["n_models"])
    calls = [(q, e, qq["P"], G) for q, qq in enumerate(f["queries"]) for e, G in qq["experts"]]
    log, _ = run_feeder(s, calls, agg_model=f["aggregator"], agg_G=f["agg_G"],
                        query_len=[qq["P"] for qq in f["queries"]],
                        query_experts=[tuple(e for e, _ in qq["experts"]) for qq in f["queries"]],
                        window=f["window"])
    assert [list(t) for t in s.steps] == f["steps"]
    assert [[a, list(b)] for a, b in log] == f["collects"]
    assert len(s.reqs) == len(f["requests"])
    for r, want in zip(s.reqs, f["requests"]):
        assert (r.expert, r.P, r.G, r.admit_step, r.finish_step, r.blocks) == (
            want["model"], want["P"], want["G"], want["admit"], want["finish"], want["blocks"])


def test_submit_validation():
    s = OracleScheduler(4, 2, 16, 2)
    for bad in [(2, 5, 3), (-1, 5, 3), (0, 0, 3), (0, 5, 0)]:
        with pytest.raises(SchedError) as e:
            s.submit(*bad)
        assert e.value.code == "EINVAL"
    with pytest.raises(SchedError) as e:
        s.submit(0, 60, 6)                      # needs 5 blocks of 16 > 4
    assert e.value.code == "ENOSPC"
    s.submit(0, 60, 5)                          # exactly 64 slots: fits


def _random_run(seed, injected=False):
    rng = np.random.default_rng(seed)
    NB = int(rng.integers(4, 40))
    s = OracleScheduler(NB, int(rng.integers(1, 6)), int(rng.integers(1, 80)), 3)
    n = int(rng.integers(1, 12))
    for _ in range(n):
        m = int(rng.integers(0, 3))
        try:
            if injected and rng.random() < 0.5:
                s.submit_injected(m, int(rng.integers(0, 60)), int(rng.integers(1, 20)))
            else:
                s.submit(m, int(rng.integers(1, 60)), int(rng.integers(1, 20)))
        except SchedError as e:
            assert e.code == "ENOSPC"
    owner = {}
    steps = 0
    while True:
        before = {r.rid for r in s.running}
        st = s.step()
        if st is None:
            break
        steps += 1
        owned = [b for r in s.running for b in r.blocks]
        assert len(owned) == len(set(owned)), "a block has two owners"
        assert len(owned) + len(s.free) == NB, "blocks are conserved"
        assert set(owned).isdisjoint(set(s.free))
        assert steps < 10000
    for r in s.reqs:
        if r.admit_step < 0:
            continue
        written_last = (r.injected_ctx + r.G - 1) if r.injected_ctx >= 0 else (r.P + r.G - 2)
        assert written_last < len(r.blocks) * 16, "every written slot lies in the request's blocks"
        assert r.blocks == sorted(r.blocks)
        assert r.finish_step >= r.admit_step
    return s


@pytest.mark.parametrize("seed", range(60))
def test_invariants_on_random_workloads(seed):
    _random_run(seed, injected=seed % 2 == 1)


def test_uncontended_request_retires_after_G_steps():
    """Enough blocks, seats and prefill budget: admitted at s, prompt done at s,
    one token per step after that, so it retires at s + G - 1."""
    s = OracleScheduler(1000, 100, 10 ** 6, 1)
    Gs = [1, 2, 7, 30]
    for i, G in enumerate(Gs):
        s.submit(0, 5 + 17 * i, G)
    while s.step() is not None:
        pass
    for r, G in zip(s.reqs, Gs):
        assert r.admit_step == 0 and r.finish_step == G - 1


def test_queries_times_fanout_equals_total_slots():
    """Sum over experts of N_m equals k * questions (the paper's per-expert slot
    table satisfies this identity: 3 slots per question)."""
    for name, k in [("moa-4x1b-bf16", 2), ("moa-3+1x8b-bf16", 2), ("tiny-moa-fp32", 2)]:
        w = make_workload(name, 0)
        assert len(w.expert_requests()) == k * w.n_queries
        assert all(len(set(e)) == len(e) == k for e in w.experts)


@pytest.mark.slow
def test_full_trace_of_4x1b_workload_is_plausible():
    c = CONFIGS["moa-4x1b-bf16"]
    w = make_workload(c.name, 0)
    e = c.engine
    s = OracleScheduler(e.num_kv_blocks, e.max_num_seqs, e.max_prefill_tokens, c.n_experts,
                        max_model_len=e.max_model_len)
    calls = [(q, m, len(w.prompts[q]), G) for q, m, G in w.expert_requests()]
    log, _ = run_feeder(s, calls)
    assert sum(len(b) for _, b in log) == len(calls)
    assert sum(t[3] for t in s.steps) + sum(1 for _ in calls) == w.total_expert_tokens()
    assert max(r.finish_step for r in s.reqs) >= max(w.max_new.values()) - 1
