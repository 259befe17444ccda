"""Oracle scheduler: an independent, plain simulation of the engine's step rule.

TEST INFRASTRUCTURE ONLY (see oracle/transformer.py).

The paper runs each expert session under vLLM's continuous batching (Section
"Evaluation Methodology"; appendix "Pitfalls of Data Concurrency": peak
tokens/s needs enough prompts in flight) and leaves the step rule to that
engine. The engine here fixes one rule so that its bookkeeping is a pure
function of request lengths (there is no end-of-sequence token, so every
finish is known in advance); this module re-implements that rule from its
statement, sharing nothing with the engine:

  need(r)   = ceil((P + G - 1) / 16)  block slots; an injected request (KV
              history of L positions already present, R tokens to emit)
              needs ceil((L + R) / 16)
  step s:
    1 admit   while the FIFO head fits (|running| < max_num_seqs and
              need <= free blocks): give it the need() smallest free block
              ids, ascending. Head-of-line blocking, no preemption.
    2 prefill budget = max_prefill_tokens tokens; running requests in
              admission order take min(remaining prompt, budget) positions;
              the one that completes its prompt emits token 0 this step and
              is "fresh" (it does not decode in the same step).
    3 decode  every running, fully prefilled, non-fresh request with
              gen < G feeds its last token at position P + gen - 1 and
              emits token gen. An injected request feeds its seed token
              first, at position L, and emits R tokens.
    4 retire  requests with gen == G free their blocks (in admission order)
              and join the done queue; fresh flags clear.
  feeder:   expert calls are submitted in first-seen order (queries
            ascending, experts ascending); after step s is enqueued the
            feeder collects everything retired at steps <= s - 1, and for
            each query whose experts are now all done (ascending q) submits
            the aggregator call on query ++ outputs (experts ascending).
"""
import heapq
from dataclasses import dataclass, field


class SchedError(Exception):
    def __init__(self, code, msg):
        super().__init__(msg)
        self.code = code        # "EINVAL" | "ENOSPC"


@dataclass
class Req:
    rid: int
    expert: int
    P: int                      # prompt length (injected: L + 1, seed included)
    G: int
    injected_ctx: int = -1      # L for an injected request, else -1
    need: int = 0
    pre: int = 0
    gen: int = 0
    fresh: bool = False
    blocks: list = field(default_factory=list)
    admit_step: int = -1
    finish_step: int = -1
    chunks: list = field(default_factory=list)     # (step, start, length)
    decode_steps: int = 0


class OracleScheduler:
    def __init__(self, num_blocks, max_num_seqs, max_prefill_tokens, n_models,
                 block_size=16, max_model_len=1 << 30):
        self.NB = num_blocks
        self.max_seqs = max_num_seqs
        self.max_prefill = max_prefill_tokens
        self.n_models = n_models
        self.bs = block_size
        self.max_len = max_model_len
        self.free = list(range(num_blocks))        # a heap of free block ids
        self.pending = []
        self.running = []
        self.done = []                             # (finish_step, Req)
        self.reqs = []
        self.step_idx = 0
        self.steps = []                            # per-step summary tuples

    # ------------------------------------------------------------ submit
    def submit(self, expert, P, G):
        if P < 1 or G < 1 or not (0 <= expert < self.n_models) or P + G - 1 > self.max_len:
            raise SchedError("EINVAL", "bad request")
        need = -(-(P + G - 1) // self.bs)
        if need > self.NB:
            raise SchedError("ENOSPC", "request can never fit the KV pool")
        r = Req(len(self.reqs), expert, P, G, need=need)
        self.reqs.append(r)
        self.pending.append(r)
        return r.rid

    def submit_injected(self, expert, L, R):
        if L < 0 or R < 1 or not (0 <= expert < self.n_models) or L + R > self.max_len:
            raise SchedError("EINVAL", "bad request")
        need = -(-(L + R) // self.bs)
        if need > self.NB:
            raise SchedError("ENOSPC", "request can never fit the KV pool")
        r = Req(len(self.reqs), expert, L + 1, R, injected_ctx=L, need=need)
        r.pre = r.P                                # no prompt to prefill
        self.reqs.append(r)
        self.pending.append(r)
        return r.rid

    def idle(self):
        return not self.pending and not self.running

    # -------------------------------------------------------------- step
    def step(self):
        """Plan one step. Returns None when there is nothing to run."""
        if self.idle():
            return None
        s = self.step_idx
        admitted = 0
        while (self.pending and len(self.running) < self.max_seqs
               and self.pending[0].need <= len(self.free)):
            r = self.pending.pop(0)
            r.blocks = [heapq.heappop(self.free) for _ in range(r.need)]
            r.admit_step = s
            self.running.append(r)
            admitted += 1
        budget = self.max_prefill
        n_pre = 0
        for r in self.running:
            if budget <= 0:
                break
            if r.pre < r.P:
                c = min(r.P - r.pre, budget)
                r.chunks.append((s, r.pre, c))
                r.pre += c
                budget -= c
                n_pre += c
                if r.pre == r.P:
                    r.gen = 1
                    r.fresh = True
        n_dec = 0
        for r in self.running:
            if r.pre == r.P and not r.fresh and r.gen < r.G:
                r.gen += 1
                r.decode_steps += 1
                n_dec += 1
        retired = []
        keep = []
        for r in self.running:
            if r.gen == r.G:
                for b in r.blocks:
                    heapq.heappush(self.free, b)
                r.finish_step = s
                self.done.append(r)
                retired.append(r.rid)
            else:
                keep.append(r)
            r.fresh = False
        self.running = keep
        self.steps.append((s, admitted, n_pre, n_dec, len(retired), len(self.free)))
        self.step_idx += 1
        return s

    def collect(self, upto_step):
        out = [r for r in self.done if r.finish_step <= upto_step]
        self.done = [r for r in self.done if r.finish_step > upto_step]
        return out


def c_vote(answers):
    """Plurality fraction of the adaptive-aggregation gate (Section "MOSAIC:
    Adaptive Aggregation", Eq. 11 and Algorithm 1): the largest number of
    experts that gave one same answer, divided by the number of experts k."""
    from collections import Counter
    from fractions import Fraction
    return Fraction(max(Counter(answers).values()), len(answers))


def run_feeder(sched, expert_calls, agg_model=-1, agg_G=0, query_len=None,
               query_experts=None, direct_calls=(), gate_tau=None, answers=None, window=None):
    """Drive ``sched`` the way the engine's feeder drives the engine.

    expert_calls: [(q, e, P, G)] in first-seen order. direct_calls: [(q, model,
    P, G)] submitted up front after the expert calls (no experts to wait for).
    Aggregator calls have prompt length query_len[q] + sum of the G of its
    experts. Returns (collect_log, rid_of) with collect_log a list of
    (after_step, [rids]) and rid_of[(q, model)] -> rid.

    gate_tau: Algorithm 1's threshold. When a query's experts are all done,
    its aggregator call is made only if c_vote of answers[(q, e)] over its
    experts is below gate_tau; otherwise no call (the majority answer stands).

    window: None submits every expert call up front; an integer W submits
    the next expert calls (in the given order) only while fewer than W
    requests wait in the scheduler's pending queue, checked after every step
    once that step's collect has been handled (aggregator calls are submitted
    when ready, whatever the queue holds)."""
    rid_of = {}
    calls = list(expert_calls)
    nxt = [0]

    def top_up():
        n = 0
        while nxt[0] < len(calls) and (window is None or len(sched.pending) < window):
            q, e, P, G = calls[nxt[0]]
            nxt[0] += 1
            rid = sched.submit(e, P, G)
            rid_of[(q, e)] = rid
            by_rid[rid] = (q, e)
            n += 1
        return n

    by_rid = {}
    top_up()
    for q, mdl, P, G in direct_calls:
        rid_of[(q, mdl)] = sched.submit(mdl, P, G)
    remaining = {}
    gsum = {}
    if agg_model >= 0 and query_experts is not None:
        for q, ex in enumerate(query_experts):
            if ex:
                remaining[q] = len(ex)
                gsum[q] = 0
    for (q, m), rid in rid_of.items():
        by_rid[rid] = (q, m)
    log = []
    last = -1

    def handle(done, after):
        if done:
            log.append((after, [r.rid for r in done]))
        ready = []
        for r in done:
            q, m = by_rid[r.rid]
            if q in remaining and m != agg_model:
                remaining[q] -= 1
                gsum[q] += r.G
                if remaining[q] == 0:
                    ready.append(q)
        for q in sorted(ready):
            if gate_tau is not None:
                from fractions import Fraction
                if c_vote([answers[(q, e)] for e in query_experts[q]]) >= Fraction(gate_tau).limit_denominator(64):
                    del remaining[q]
                    continue
            rid = sched.submit(agg_model, query_len[q] + gsum[q], agg_G)
            rid_of[(q, agg_model)] = rid
            by_rid[rid] = (q, agg_model)
            del remaining[q]
        return len(ready)

    while True:
        s = sched.step()
        if s is None:
            n = handle(sched.collect(last), last)
            m = top_up()
            if n == 0 and m == 0 and sched.idle():
                break
            continue
        last = s
        if s >= 1:
            handle(sched.collect(s - 1), s - 1)
        top_up()
    return log, rid_of
