"""Shared helpers for the GPU parity tests (engine run + oracle comparison)."""
import sys

import numpy as np

from moa_inputs import pack_blob
from oracle import transformer as T
from paper_2606_03014_amd import Engine

MARGIN = 1e-3          # a token may differ only where the oracle's top-2 margin is below this


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def run_requests(shape, dtype, consts, weights_list, requests, capture=True, repeat=1, one_stream=False):
    """requests: [(tokens, model_index, G)]. Returns (tokens by request, logits by request)."""
    eng = Engine(shape, dtype, consts, len(weights_list), one_stream=one_stream)
    try:
        mids = [eng.load(pack_blob(w, shape)) for w in weights_list]
        outs, caps = [], []
        for _ in range(repeat):
            cap = {}
            rids = []
            for toks, m, G in requests:
                rid = eng.submit(np.asarray(toks, dtype=np.int32), mids[m], G)
                rids.append(rid)
                if capture:
                    cap[rid] = np.full(G * shape.vocab, np.nan, dtype=np.float32)
                    eng.capture_logits(rid, cap[rid])
            while eng.step().step >= 0:
                pass
            got = {r[0]: r[3] for r in eng.collect()}
            outs.append([got[r] for r in rids])
            caps.append([cap[r].reshape(-1, shape.vocab) for r in rids] if capture else None)
    finally:
        eng.close()
    if repeat == 1:
        return outs[0], caps[0]
    return outs, caps


def check_tokens(ref_logits, toks, what=""):
    """Every emitted token is the oracle argmax, or the oracle's top-2 margin
    at that position is below MARGIN and the token is within it."""
    flips = []
    for j, t in enumerate(toks):
        lg = ref_logits[j]
        best = int(np.argmax(lg))
        if t != best:
            gap = float(lg[best] - lg[t])
            assert gap < MARGIN, f"{what} position {j}: token {t} vs oracle {best}, gap {gap:.3e}"
            flips.append((j, gap))
    return flips


def compare(shape, weights, prompt, toks, logits, bf16_kv, logit_tol, n_layers=None, what="",
            report_pure=True):
    """Teacher-forced oracle on the engine's own history; returns (max logit err, flips).

    A bf16 engine stores its KV cache in bf16, so its oracle stores K/V in
    bf16 too (``bf16_kv``); logits and tokens are judged against that oracle.
    The distance to the oracle with an exact cache is reported, not bounded."""
    om = T.OracleModel(shape, weights, n_layers=n_layers, cache=False)
    ref = T.teacher_forced_logits(om, prompt, toks, bf16_kv=bf16_kv)
    assert logits is None or np.all(np.isfinite(logits)), f"{what}: non-finite logits"
    err = float(np.abs(logits - ref).max()) if logits is not None else 0.0
    msg = f"{what}: |engine - oracle| {err:.3e}"
    if bf16_kv and report_pure and logits is not None:
        pure = T.teacher_forced_logits(om, prompt, toks)
        msg += f"  (vs oracle with an exact KV cache: {float(np.abs(logits - pure).max()):.3e})"
    say(msg)
    assert err <= logit_tol, f"{what}: max |logit - oracle| = {err:.3e} > {logit_tol}"
    flips = check_tokens(ref, toks, what)
    return err, flips
