"""ctypes binding of include/moa.h: the same names, argument marshalling only.

Every computation happens in libmoa.so (HIP kernels for gfx950 plus the
engine's host bookkeeping). Loading fails loudly when the library has not
been built; there is no fallback implementation.
"""
import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmoa.so")

MOA_OK, MOA_EINVAL, MOA_ENOMEM, MOA_ENOSPC, MOA_ESTATE, MOA_EHIP = 0, -1, -2, -3, -4, -5
MOA_F32, MOA_BF16 = 0, 1
MOA_FLAG_PLAN_ONLY = 1
MOA_FLAG_ONE_STREAM = 2
STATUS_NAMES = {0: "MOA_OK", -1: "MOA_EINVAL", -2: "MOA_ENOMEM", -3: "MOA_ENOSPC",
                -4: "MOA_ESTATE", -5: "MOA_EHIP"}


class moa_model_cfg(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn_dim", C.c_int32),
                ("vocab", C.c_int32), ("rope_theta", C.c_float), ("rms_eps", C.c_float)]


class moa_engine_cfg(C.Structure):
    _fields_ = [("model", moa_model_cfg), ("dtype", C.c_int32), ("kv_block_size", C.c_int32),
                ("num_kv_blocks", C.c_int32), ("max_num_seqs", C.c_int32),
                ("max_prefill_tokens", C.c_int32), ("max_model_len", C.c_int32),
                ("max_models", C.c_int32), ("flags", C.c_int32),
                ("token_store", C.c_int64), ("block_store", C.c_int64)]


class moa_step_info(C.Structure):
    _fields_ = [("step", C.c_int64), ("admitted", C.c_int32), ("prefill_tokens", C.c_int32),
                ("decode_rows", C.c_int32), ("finished", C.c_int32), ("running", C.c_int32),
                ("pending", C.c_int32), ("free_blocks", C.c_int32), ("emitted", C.c_int32)]


class moa_result(C.Structure):
    _fields_ = [("request_id", C.c_int64), ("model_id", C.c_int32), ("n_tokens", C.c_int32),
                ("tok_offset", C.c_int64), ("finish_step", C.c_int64)]


class moa_request_info(C.Structure):
    _fields_ = [("model_id", C.c_int32), ("prompt_len", C.c_int32), ("max_new_tokens", C.c_int32),
                ("n_blocks", C.c_int32), ("admit_step", C.c_int64), ("finish_step", C.c_int64),
                ("n_chunks", C.c_int32), ("state", C.c_int32)]


class moa_kernel_stats(C.Structure):
    _fields_ = [("launches", C.c_int64), ("ms", C.c_double), ("bytes", C.c_double), ("flops", C.c_double),
                ("launches_all", C.c_int64), ("bytes_all", C.c_double), ("flops_all", C.c_double),
                ("roof_ms_all", C.c_double)]


KERNEL_CLASSES = ["embed", "norm", "gemm_qkv", "rope_kv", "attn", "attn_reduce", "gemm_o",
                  "gemm_gateup", "gemm_down", "gemm_lmhead", "argmax", "prefill_attn",
                  "gemm_small_m", "gemm_large_m"]
# views: every GEMM launch is counted again in one of these (leave them out of sums over classes)
VIEW_CLASSES = ("gemm_small_m", "gemm_large_m")

P = C.POINTER
_SIGS = {
    "moa_arena_bytes": (C.c_int, [P(moa_engine_cfg), P(C.c_size_t)]),
    "moa_create": (C.c_int, [P(moa_engine_cfg), C.c_void_p, C.c_size_t, C.c_void_p, P(C.c_void_p)]),
    "moa_load_expert": (C.c_int, [C.c_void_p, P(moa_model_cfg), C.c_void_p, C.c_size_t, P(C.c_int32)]),
    "moa_submit": (C.c_int, [C.c_void_p, P(C.c_int32), C.c_int32, C.c_int32, C.c_int32, P(C.c_int64)]),
    "moa_submit_with_history": (C.c_int, [C.c_void_p, C.c_int32, C.c_int32, C.c_int32, C.c_void_p, C.c_int32,
                                          P(C.c_int64)]),
    "moa_step": (C.c_int, [C.c_void_p, P(moa_step_info)]),
    "moa_step_noalloc": (C.c_int, [C.c_void_p, P(moa_step_info)]),
    "moa_collect": (C.c_int, [C.c_void_p, C.c_int64, P(moa_result), C.c_int32, P(C.c_int32),
                              P(C.c_int32), C.c_int64]),
    "moa_sync": (C.c_int, [C.c_void_p]),
    "moa_destroy": (None, [C.c_void_p]),
    "moa_status_str": (C.c_char_p, [C.c_int]),
    "moa_debug_request": (C.c_int, [C.c_void_p, C.c_int64, P(moa_request_info)]),
    "moa_debug_block_table": (C.c_int, [C.c_void_p, C.c_int64, P(C.c_int32), C.c_int32, P(C.c_int32)]),
    "moa_debug_chunks": (C.c_int, [C.c_void_p, C.c_int64, P(C.c_int64), C.c_int32, P(C.c_int32)]),
    "moa_debug_steps": (C.c_int, [C.c_void_p, P(C.c_int64), C.c_int64, P(C.c_int64)]),
    "moa_debug_capture_logits": (C.c_int, [C.c_void_p, C.c_int64, P(C.c_float), C.c_int64]),
    "moa_debug_time_kernels": (C.c_int, [C.c_void_p, C.c_int32, C.c_double, C.c_double]),
    "moa_debug_kernel_stats": (C.c_int, [C.c_void_p, P(moa_kernel_stats)]),
    "moa_debug_measure_peaks": (C.c_int, [C.c_void_p, P(C.c_double), P(C.c_double)]),
    "moa_debug_step_shares": (C.c_int, [C.c_void_p, P(C.c_int32), P(C.c_int32), P(C.c_int32), P(C.c_double),
                                        P(C.c_int32), P(C.c_int32), P(C.c_int32)]),
}

_lib = None


def lib():
    """The loaded libmoa.so (raises if it was not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it first (python -c "
                               "'import __graft_entry__ as g; g.build()')")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


class MoaError(RuntimeError):
    def __init__(self, code, where):
        self.code = code
        super().__init__(f"{where}: {STATUS_NAMES.get(code, code)}")


def check(code, where):
    if code != MOA_OK:
        raise MoaError(code, where)
    return code


def exported_symbols():
    return list(_SIGS)


# thin same-name wrappers -----------------------------------------------------

def moa_arena_bytes(cfg):
    n = C.c_size_t()
    check(lib().moa_arena_bytes(C.byref(cfg), C.byref(n)), "moa_arena_bytes")
    return n.value


def moa_create(cfg, dev_arena, arena_bytes, hip_stream):
    h = C.c_void_p()
    check(lib().moa_create(C.byref(cfg), dev_arena, arena_bytes, hip_stream, C.byref(h)), "moa_create")
    return h


def moa_load_expert(eng, mcfg, blob):
    mid = C.c_int32()
    ptr = blob.ctypes.data_as(C.c_void_p)
    check(lib().moa_load_expert(eng, C.byref(mcfg), ptr, blob.nbytes, C.byref(mid)), "moa_load_expert")
    return mid.value


def moa_submit(eng, tokens, model_id, max_new_tokens):
    import numpy as np
    t = np.ascontiguousarray(tokens, dtype=np.int32)
    rid = C.c_int64()
    check(lib().moa_submit(eng, t.ctypes.data_as(P(C.c_int32)), len(t), model_id, max_new_tokens,
                           C.byref(rid)), "moa_submit")
    return rid.value


def moa_submit_with_history(eng, model_id, seed_token, ctx_len, max_new_tokens, host_kv=None):
    """host_kv: None (device fill) or a contiguous numpy array of
    [n_layers, 2, ctx_len, n_kv_heads, head_dim] in the engine dtype."""
    import numpy as np
    rid = C.c_int64()
    ptr = None
    if host_kv is not None:
        host_kv = np.ascontiguousarray(host_kv)
        ptr = host_kv.ctypes.data_as(C.c_void_p)
    check(lib().moa_submit_with_history(eng, model_id, seed_token, ctx_len, ptr, max_new_tokens, C.byref(rid)),
          "moa_submit_with_history")
    return rid.value


def moa_step(eng):
    info = moa_step_info()
    check(lib().moa_step(eng, C.byref(info)), "moa_step")
    return info


def moa_step_noalloc(eng):
    info = moa_step_info()
    check(lib().moa_step_noalloc(eng, C.byref(info)), "moa_step_noalloc")
    return info


def moa_collect(eng, upto_step=-1):
    """Returns [(request_id, model_id, finish_step, np.int32 tokens)] in retirement order."""
    import numpy as np
    L = lib()
    n = C.c_int32()
    code = L.moa_collect(eng, upto_step, None, 0, C.byref(n), None, 0)
    if code == MOA_OK:
        return []                      # nothing ready
    if code != MOA_EINVAL:
        raise MoaError(code, "moa_collect")
    cap = n.value
    res = (moa_result * cap)()
    tok_cap = 1 << 16
    while True:
        buf = np.empty(tok_cap, dtype=np.int32)
        code = L.moa_collect(eng, upto_step, res, cap, C.byref(n), buf.ctypes.data_as(P(C.c_int32)), tok_cap)
        if code == MOA_OK:
            break
        if code != MOA_EINVAL or tok_cap > (1 << 34):
            raise MoaError(code, "moa_collect")
        if n.value > cap:
            cap = n.value
            res = (moa_result * cap)()
        tok_cap *= 4
    return [(res[i].request_id, res[i].model_id, res[i].finish_step,
             buf[res[i].tok_offset: res[i].tok_offset + res[i].n_tokens].copy()) for i in range(n.value)]


def moa_sync(eng):
    check(lib().moa_sync(eng), "moa_sync")


def moa_destroy(eng):
    lib().moa_destroy(eng)


def moa_status_str(code):
    return lib().moa_status_str(code).decode()


def moa_debug_request(eng, rid):
    info = moa_request_info()
    check(lib().moa_debug_request(eng, rid, C.byref(info)), "moa_debug_request")
    return info


def moa_debug_block_table(eng, rid):
    import numpy as np
    n = C.c_int32()
    info = moa_debug_request(eng, rid)
    buf = np.zeros(max(info.n_blocks, 1), dtype=np.int32)
    check(lib().moa_debug_block_table(eng, rid, buf.ctypes.data_as(P(C.c_int32)), len(buf), C.byref(n)),
          "moa_debug_block_table")
    return buf[: n.value].tolist()


def moa_debug_chunks(eng, rid):
    import numpy as np
    info = moa_debug_request(eng, rid)
    n = C.c_int32()
    buf = np.zeros(3 * max(info.n_chunks, 1), dtype=np.int64)
    check(lib().moa_debug_chunks(eng, rid, buf.ctypes.data_as(P(C.c_int64)), max(info.n_chunks, 1),
                                 C.byref(n)), "moa_debug_chunks")
    return [tuple(int(v) for v in buf[3 * i: 3 * i + 3]) for i in range(n.value)]


def moa_debug_steps(eng):
    import numpy as np
    n = C.c_int64()
    L = lib()
    code = L.moa_debug_steps(eng, None, 0, C.byref(n))   # the count (MOA_EINVAL once there are steps)
    if code not in (MOA_OK, MOA_EINVAL) or (code == MOA_EINVAL and n.value == 0):
        raise MoaError(code, "moa_debug_steps")
    if n.value == 0:
        return np.zeros((0, 6), dtype=np.int64)
    buf = np.zeros(6 * n.value, dtype=np.int64)
    check(L.moa_debug_steps(eng, buf.ctypes.data_as(P(C.c_int64)), n.value, C.byref(n)), "moa_debug_steps")
    return buf.reshape(-1, 6)


def moa_debug_capture_logits(eng, rid, host_array):
    """host_array: contiguous float32 numpy array of at least max_new_tokens *
    vocab elements, kept alive by the caller until the request is collected."""
    import numpy as np
    if host_array.dtype != np.float32 or not host_array.flags.c_contiguous:
        raise ValueError("capture buffer must be a contiguous float32 array")
    check(lib().moa_debug_capture_logits(eng, rid, host_array.ctypes.data_as(P(C.c_float)), host_array.size),
          "moa_debug_capture_logits")


def moa_debug_time_kernels(eng, every, peak_bw=8.0e12, peak_flops=2.5e15):
    check(lib().moa_debug_time_kernels(eng, every, peak_bw, peak_flops), "moa_debug_time_kernels")


def moa_debug_kernel_stats(eng):
    """{class name: dict of the moa_kernel_stats fields}."""
    out = (moa_kernel_stats * len(KERNEL_CLASSES))()
    check(lib().moa_debug_kernel_stats(eng, out), "moa_debug_kernel_stats")
    return {n: {f: getattr(out[i], f) for f, _ in moa_kernel_stats._fields_}
            for i, n in enumerate(KERNEL_CLASSES)}


def moa_debug_step_shares(eng, max_models):
    """How the last step split its models over the model streams:
    {"models": [...], "cost": [...], "shares": [(models, rows, lm_rows), ...]}
    with each share's models as a list and its rows / LM rows as ranges."""
    ns, nm = C.c_int32(), C.c_int32()
    models = (C.c_int32 * max_models)()
    cost = (C.c_double * max_models)()
    m0, r0, l0 = (C.c_int32 * 5)(), (C.c_int32 * 5)(), (C.c_int32 * 5)()
    check(lib().moa_debug_step_shares(eng, C.byref(ns), C.byref(nm), models, cost, m0, r0, l0),
          "moa_debug_step_shares")
    mods = list(models[:nm.value])
    shares = [(mods[m0[u]:m0[u + 1]], range(r0[u], r0[u + 1]), range(l0[u], l0[u + 1]))
              for u in range(ns.value)]
    return {"models": mods, "cost": list(cost[:nm.value]), "shares": shares}


def moa_debug_measure_peaks(eng):
    """(HBM read bytes/s, bf16 32x32x16 MFMA flop/s) measured on the engine's stream."""
    r, f = C.c_double(), C.c_double()
    check(lib().moa_debug_measure_peaks(eng, C.byref(r), C.byref(f)), "moa_debug_measure_peaks")
    return r.value, f.value
