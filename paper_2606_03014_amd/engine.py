"""Python-side handle on the C-ABI engine plus the host feeder.

PyTorch only supplies the device arena and the stream. The feeder is the
plain host-side policy of the paper's setting (Section "Problem Setting": a
fixed batch of routed calls; Section "MOSAIC: Adaptive Aggregation": the
aggregator runs on the query plus the expert outputs): it submits the expert
calls in first-seen order (queries ascending, experts ascending) and, after
each step, collects what retired one step earlier and submits the aggregator
call of every query whose experts are all done (ascending query id), on
query ++ outputs in ascending expert order.
"""
from fractions import Fraction

import numpy as np

from . import moa as M


def model_cfg(shape):
    return M.moa_model_cfg(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads,
                           shape.head_dim, shape.ffn_dim, shape.vocab, shape.rope_theta, shape.rms_eps)


def engine_cfg(shape, dtype, consts, max_models, plan_only=False, token_store=0, block_store=0,
               one_stream=False):
    flags = (M.MOA_FLAG_PLAN_ONLY if plan_only else 0) | (M.MOA_FLAG_ONE_STREAM if one_stream else 0)
    return M.moa_engine_cfg(model_cfg(shape), M.MOA_BF16 if dtype == "bf16" else M.MOA_F32,
                            consts.kv_block_size, consts.num_kv_blocks, consts.max_num_seqs,
                            consts.max_prefill_tokens, consts.max_model_len, max_models,
                            flags, token_store, block_store)


class Engine:
    """Owns one moa_engine and (unless plan_only) its torch-allocated arena."""

    def __init__(self, shape, dtype, consts, max_models, plan_only=False, device="cuda:0",
                 token_store=0, block_store=0, one_stream=False):
        self.shape = shape
        self.cfg = engine_cfg(shape, dtype, consts, max_models, plan_only, token_store, block_store, one_stream)
        self.arena_bytes = M.moa_arena_bytes(self.cfg)
        self.plan_only = plan_only
        self.arena = None
        if plan_only:
            self.h = M.moa_create(self.cfg, None, 0, None)
        else:
            import torch
            if not torch.cuda.is_available():
                raise RuntimeError("the HIP engine needs a GPU (torch.cuda.is_available() is False)")
            self.device = torch.device(device)
            self.arena = torch.empty(self.arena_bytes, dtype=torch.uint8, device=self.device)
            self.stream = torch.cuda.current_stream(self.device)
            self.h = M.moa_create(self.cfg, self.arena.data_ptr(), self.arena_bytes, self.stream.cuda_stream)

    def load(self, blob):
        return M.moa_load_expert(self.h, self.cfg.model, np.ascontiguousarray(blob))

    def submit(self, tokens, model_id, max_new):
        return M.moa_submit(self.h, tokens, model_id, max_new)

    def submit_with_history(self, model_id, seed_token, ctx_len, max_new, host_kv=None):
        return M.moa_submit_with_history(self.h, model_id, seed_token, ctx_len, max_new, host_kv)

    def step(self):
        return M.moa_step(self.h)

    def step_noalloc(self):
        return M.moa_step_noalloc(self.h)

    def collect(self, upto=-1):
        return M.moa_collect(self.h, upto)

    def sync(self):
        M.moa_sync(self.h)

    def steps(self):
        return M.moa_debug_steps(self.h)

    def request(self, rid):
        return M.moa_debug_request(self.h, rid)

    def block_table(self, rid):
        return M.moa_debug_block_table(self.h, rid)

    def chunks(self, rid):
        return M.moa_debug_chunks(self.h, rid)

    def time_kernels(self, every, peak_bw=8.0e12, peak_flops=2.5e15):
        M.moa_debug_time_kernels(self.h, every, peak_bw, peak_flops)

    def kernel_stats(self):
        return M.moa_debug_kernel_stats(self.h)

    def measure_peaks(self):
        return M.moa_debug_measure_peaks(self.h)

    def step_shares(self):
        return M.moa_debug_step_shares(self.h, self.cfg.max_models)

    def capture_logits(self, rid, arr):
        M.moa_debug_capture_logits(self.h, rid, arr)

    def close(self):
        if getattr(self, "h", None) is not None:
            M.moa_destroy(self.h)
            self.h = None
        self.arena = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class FeedResult:
    def __init__(self):
        self.outputs = {}        # (q, model_id) -> np.int32 tokens
        self.rid_of = {}         # (q, model_id) -> request id
        self.collects = []       # (after_step, [request ids])
        self.n_steps = 0
        self.tokens = 0
        self.gated = {}          # q -> majority answer, for queries whose aggregator call the gate skipped
        self.agg_calls = 0       # aggregator calls submitted


def plurality(answers):
    """Confidence of a set of expert answers as in the adaptive-aggregation
    gate (Eq. 11): the share of the most frequent answer among the k answers,
    as an exact fraction, and that answer (the smallest one if several tie)."""
    counts = {}
    for a in answers:
        counts[a] = counts.get(a, 0) + 1
    top = max(counts.values())
    return Fraction(top, len(answers)), min(a for a, c in counts.items() if c == top)


def expert_order(workload, order):
    """Expert calls (q, e, G) in submission order. "first-seen": queries
    ascending, experts ascending. "longest-first": largest max_new_tokens
    first (ties in first-seen order) -- with every call's generation length
    known up front, a longest-processing-time order starts the calls that
    set the makespan before the short ones."""
    calls = list(workload.expert_requests())
    if order == "first-seen":
        return calls
    if order == "longest-first":
        return sorted(calls, key=lambda c: -c[2])
    raise ValueError(order)


class Feeder:
    """The host feeder of one workload, resumable: ``advance(n)`` runs at most
    n engine steps, so a caller can time a fixed window of the schedule.

    expert_models[e] is the engine model id of expert e; agg_model is the
    aggregator's model id (-1: none). A workload without experts sends every
    query straight to the aggregator.

    gate_tau: the confidence gate of the adaptive aggregation (Eq. 11,
    Algorithm 1). When the last expert of a query finishes, its answers
    answer_of(q, e, tokens) (experts ascending) are scored by plurality();
    if the score is >= gate_tau the aggregator call is skipped and the
    majority answer recorded in FeedResult.gated, else the aggregator call
    is submitted as usual. order: see expert_order().

    window: None submits every expert call up front. An integer W keeps at
    most W submitted-but-unadmitted calls in the engine: expert calls are
    submitted as admissions make room, while aggregator calls are submitted
    the moment their experts finish, so they overtake the expert calls not
    yet submitted (aggregation fills the gaps of the expert tail instead of
    queueing behind every expert call).

    Each engine step collects what retired one step earlier, so the schedule
    (and when aggregator calls are submitted) is a function of step indices
    only, whatever the caller's step windows are."""

    def __init__(self, eng, workload, expert_models, agg_model=-1, on_step=None, gate_tau=None,
                 answer_of=None, order="first-seen", window=None, on_submit=None):
        if window is not None and window < 1:
            raise ValueError("window must be >= 1")
        self.eng, self.wl, self.experts, self.agg = eng, workload, list(expert_models), agg_model
        self.on_step = on_step
        self.on_submit = on_submit    # on_submit(request id, query, model id, max_new) after each submit
        self.answer_of = answer_of
        self.tau = None if gate_tau is None else Fraction(gate_tau).limit_denominator(64)
        self.window = window
        self.res = FeedResult()
        self.who = {}
        self.queue = list(expert_order(workload, order))
        self.nxt = 0
        self.submitted = self.admitted = 0
        self.last = -1
        self.emitted = 0         # tokens produced by the engine steps run so far
        self.done = False
        self._top_up()
        self.remaining = ({q: len(ex) for q, ex in enumerate(workload.experts) if ex}
                          if agg_model >= 0 else {})
        if agg_model >= 0 and workload.n_experts == 0:
            for q in range(workload.n_queries):
                self._submit(q, workload.prompts[q], agg_model, -1, workload.agg_max_new)
                self.res.agg_calls += 1

    def _submit(self, q, tokens, model, e, G):
        rid = self.eng.submit(tokens, model, G)
        self.res.rid_of[(q, model)] = rid
        self.who[rid] = (q, model, e)
        self.submitted += 1
        if self.on_submit is not None:
            self.on_submit(rid, q, model, G)

    def _top_up(self):
        n = 0
        while self.nxt < len(self.queue) and (self.window is None or
                                              self.submitted - self.admitted < self.window):
            q, e, G = self.queue[self.nxt]
            self.nxt += 1
            self._submit(q, self.wl.prompts[q], self.experts[e], e, G)
            n += 1
        return n

    def _handle(self, done, after):
        res, wl = self.res, self.wl
        if done:
            res.collects.append((after, [d[0] for d in done]))
        ready = []
        for rid, mdl, fin, toks in done:
            q, m, e = self.who[rid]
            res.outputs[(q, m)] = toks
            res.tokens += len(toks)
            if q in self.remaining and e >= 0:
                self.remaining[q] -= 1
                if self.remaining[q] == 0:
                    ready.append(q)
        for q in sorted(ready):
            del self.remaining[q]
            if self.tau is not None:
                conf, majority = plurality([self.answer_of(q, e, res.outputs[(q, self.experts[e])])
                                            for e in wl.experts[q]])
                if conf >= self.tau:
                    res.gated[q] = majority
                    continue
            parts = [wl.prompts[q]] + [res.outputs[(q, self.experts[e])] for e in wl.experts[q]]
            self._submit(q, np.concatenate(parts).astype(np.int32), self.agg, -1, wl.agg_max_new)
            res.agg_calls += 1
        return len(ready)

    def advance(self, max_steps=None):
        """Run engine steps until the workload is done or max_steps steps ran;
        returns (engine steps run, tokens those steps produced)."""
        steps = tokens = 0
        eng = self.eng
        while not self.done and (max_steps is None or steps < max_steps):
            info = eng.step()
            if info.step < 0:
                n = self._handle(eng.collect(self.last), self.last)
                m = self._top_up()
                if n == 0 and m == 0:
                    self.done = True
                continue
            self.last = info.step
            self.admitted += info.admitted
            self.res.n_steps += 1
            steps += 1
            tokens += info.emitted
            if self.on_step is not None:
                self.on_step(info)
            if self.last >= 1:
                self._handle(eng.collect(self.last - 1), self.last - 1)
            self._top_up()
        self.emitted += tokens
        return steps, tokens


def run_feeder(eng, workload, expert_models, agg_model=-1, on_step=None, max_steps=None,
               gate_tau=None, answer_of=None, order="first-seen", window=None, on_submit=None):
    """Drive ``eng`` through ``workload`` (a moa_inputs.Workload) to the end,
    or for at most max_steps engine steps; see Feeder for the arguments."""
    f = Feeder(eng, workload, expert_models, agg_model, on_step, gate_tau, answer_of, order, window,
               on_submit)
    f.advance(max_steps)
    return f.res


def run_straggler(eng, sw, model_id=0, host_kv_fn=None, on_step=None, after_collect=False):
    """Drive the long-reasoning straggler workload: ``sw.n_live`` calls that
    arrive with a KV history are submitted up front; for the first
    ``sw.refill_steps`` steps every call that retires is replaced by a new one
    (admitted at the next step), then the batch drains. host_kv_fn(i, L) may
    return the K/V history of sequence i (None: device fill).
    on_step(info) runs after each step is enqueued, or, with after_collect,
    once the previous step has finished and been collected.
    Returns (tokens generated, engine steps, sequences used)."""
    nxt = 0

    def submit_one():
        nonlocal nxt
        L, tok, R = sw.sequence(nxt)
        kv = host_kv_fn(nxt, L) if host_kv_fn is not None else None
        eng.submit_with_history(model_id, tok, L, R, kv)
        nxt += 1
        return R

    tokens = 0
    for _ in range(sw.n_live):
        tokens += submit_one()
    steps = 0
    first = None
    while True:
        info = eng.step()
        if info.step < 0:
            break
        first = info.step if first is None else first
        steps += 1
        if on_step is not None and not after_collect:
            on_step(info)
        if info.step - first < sw.refill_steps:
            for _ in range(info.finished):
                tokens += submit_one()
        eng.collect(info.step - 1)
        if on_step is not None and after_collect:
            on_step(info)
    eng.collect(-1)
    return tokens, steps, nxt
