"""ctypes binding of libjet.so (the C ABI declared in include/jet.h).

Argument marshalling only: every step of the scoring path runs in the HIP
library. Functions keep the C names. Arrays may be numpy arrays (host) or
torch tensors (host or, where jet.h allows device memory, on the model's
GPU). Loading fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libjet.so")

JET_OK, JET_E_INVALID, JET_E_CAPACITY, JET_E_OOM, JET_E_DEVICE, JET_E_IO = range(6)
JET_BF16, JET_FP32, JET_BF16_SINGLE, JET_F16, JET_F16P = 0, 1, 2, 3, 4
JET_CHOICE, JET_BINARY, JET_ORDINAL = 0, 1, 2
JET_FLAG_KERNEL_TIMING = 1
JET_FLAG_RECORD_ROUTES = 2
JET_NOALLOC_SCRATCH_BYTES = 64 << 20
KERNEL_CLASSES = ["gemm_qkv", "gemm_o", "gemm_gateup", "gemm_down", "lmhead", "attn_prefix",
                  "attn_cand", "gdn", "other"]
ERROR_NAMES = {1: "JET_E_INVALID", 2: "JET_E_CAPACITY", 3: "JET_E_OOM", 4: "JET_E_DEVICE", 5: "JET_E_IO"}

# every symbol include/jet.h declares
EXPORTS = ["jet_model_load", "jet_prefill_prefix", "jet_generate_trace", "jet_score_candidates",
           "jet_score_candidates_noalloc", "jet_decide",
           "jet_answer_classes", "jet_evaluate", "jet_candidate_layout", "jet_stats_get", "jet_stats_reset", "jet_model_info",
           "jet_routes_get", "jet_prefix_free", "jet_model_free", "jet_last_error"]


class JetError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERROR_NAMES.get(code, code)}: {msg}")
        self.code = code


class jet_load_opts(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("device", ctypes.c_int32), ("max_ctx", ctypes.c_int64),
                ("prefill_token_budget", ctypes.c_int64), ("wave_token_budget", ctypes.c_int64),
                ("max_device_bytes", ctypes.c_int64), ("hip_stream", ctypes.c_void_p),
                ("flags", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class jet_stats(ctypes.Structure):
    _fields_ = [("prefix_tokens", ctypes.c_int64), ("prefix_evals", ctypes.c_int64),
                ("cand_body_tokens", ctypes.c_int64), ("scored_tokens", ctypes.c_int64),
                ("lm_rows", ctypes.c_int64), ("prefill_waves", ctypes.c_int64),
                ("score_waves", ctypes.c_int64), ("kernel_launches", ctypes.c_int64 * 9),
                ("kernel_ms", ctypes.c_double * 9), ("kernel_flops", ctypes.c_double * 9),
                ("kernel_bytes", ctypes.c_double * 9)]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        # torch ships its own HIP runtime under the same soname
        # (libamdhip64.so.7). Loading torch first makes the process use one
        # runtime for both, so device pointers and streams can be shared; if
        # libjet came first, torch could not initialise its runtime later.
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2609_33874_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        L.jet_model_load.argtypes = [ctypes.c_char_p, ctypes.POINTER(jet_load_opts), ctypes.POINTER(P)]
        L.jet_prefill_prefix.argtypes = [P, I32, P, P, ctypes.POINTER(P)]
        L.jet_generate_trace.argtypes = [P, P, I32, ctypes.c_float, ctypes.c_uint64, P]
        L.jet_score_candidates.argtypes = [P, P, P, P, P, P, P]
        L.jet_score_candidates_noalloc.argtypes = [P, P, P, P, P, P, P]
        L.jet_decide.argtypes = [I32, I32, P, P, P, P, P]
        L.jet_answer_classes.argtypes = [I32, P, P, P, P]
        L.jet_evaluate.argtypes = [I32, P, P, P, P, P, P, P, P]
        L.jet_candidate_layout.argtypes = [I32, P, P, P, I64, I64, P, P, P, P, P, P]
        L.jet_stats_get.argtypes = [P, ctypes.POINTER(jet_stats)]
        L.jet_stats_reset.argtypes = [P]
        L.jet_model_info.argtypes = [P, P, P, P, P, P]
        L.jet_routes_get.argtypes = [P, I32, P, P, P, P, I64]
        L.jet_prefix_free.argtypes = [P]
        L.jet_prefix_free.restype = None
        L.jet_model_free.argtypes = [P]
        L.jet_model_free.restype = None
        L.jet_last_error.restype = ctypes.c_char_p
        for n in EXPORTS:
            if n not in ("jet_prefix_free", "jet_model_free", "jet_last_error"):
                getattr(L, n).restype = ctypes.c_int
        _lib = L
    return _lib


def jet_last_error() -> str:
    return lib().jet_last_error().decode()


def _check(code: int) -> None:
    if code != JET_OK:
        raise JetError(code, jet_last_error())


def _ptr(x, dtype):
    """(pointer, keepalive) for a numpy array or torch tensor of `dtype`."""
    if x is None:
        return None, None
    if hasattr(x, "data_ptr"):  # torch tensor, host or device
        import torch
        want = {np.int32: torch.int32, np.int64: torch.int64, np.float32: torch.float32}[dtype]
        if x.dtype != want or not x.is_contiguous():
            raise TypeError(f"tensor must be contiguous {want}")
        return ctypes.c_void_p(x.data_ptr()), x
    a = np.ascontiguousarray(x, dtype=dtype)
    return a.ctypes.data_as(ctypes.c_void_p), a


def jet_model_load(path: str, dtype: int = JET_BF16, device: int = 0, max_ctx: int = 0,
                   prefill_token_budget: int = 0, wave_token_budget: int = 0,
                   max_device_bytes: int = 0, hip_stream: int | None = None, flags: int = 0):
    o = jet_load_opts(dtype, device, max_ctx, prefill_token_budget, wave_token_budget,
                      max_device_bytes, hip_stream or None, flags, 0)
    h = ctypes.c_void_p()
    _check(lib().jet_model_load(path.encode(), ctypes.byref(o), ctypes.byref(h)))
    return h


def jet_prefill_prefix(model, prefix_offsets, prefix_tokens):
    po, k1 = _ptr(prefix_offsets, np.int64)
    pt, k2 = _ptr(prefix_tokens, np.int32)
    n_q = len(k1) - 1
    h = ctypes.c_void_p()
    _check(lib().jet_prefill_prefix(model, n_q, po, pt, ctypes.byref(h)))
    return h


def jet_generate_trace(model, prefix, n_q: int, n_steps: int, temperature: float = 0.0, seed: int = 0, out=None):
    """Extends every question of `prefix` by n_steps sampled tokens (in place).
    Returns the tokens as int32 [n_q, n_steps] (host), or writes them into
    `out` (a contiguous int32 tensor or array of n_q * n_steps, host or device)
    and returns it."""
    if out is None:
        out = np.empty((n_q, max(int(n_steps), 0)), np.int32)
    ot, keep = _ptr(out, np.int32)
    if isinstance(out, np.ndarray) and keep is not out:
        raise TypeError("out must be a contiguous int32 array")
    _check(lib().jet_generate_trace(model, prefix, int(n_steps), float(temperature),
                                    ctypes.c_uint64(seed & 0xFFFFFFFFFFFFFFFF), ot))
    return out


def jet_score_candidates(model, prefix, q_cand_offsets, cand_tok_offsets, cand_tokens,
                         out_token_logprob=True, out_cand_sum=None, _entry="jet_score_candidates"):
    """Returns (token log-probs or None, candidate sums). Pass torch tensors as
    outputs to have the library write them in place (host or device)."""
    qo, k1 = _ptr(q_cand_offsets, np.int64)
    co, k2 = _ptr(cand_tok_offsets, np.int64)
    ct, k3 = _ptr(cand_tokens, np.int32)
    n_cand = len(k2) - 1
    n_tok = int(k2[-1])
    if out_cand_sum is None:
        out_cand_sum = np.empty(n_cand, np.float32)
    if out_token_logprob is True:
        out_token_logprob = np.empty(n_tok, np.float32)
    elif out_token_logprob is False:
        out_token_logprob = None
    ot, k4 = _ptr(out_token_logprob, np.float32) if out_token_logprob is not None else (None, None)
    os_, k5 = _ptr(out_cand_sum, np.float32)
    if isinstance(out_cand_sum, np.ndarray) and k5 is not out_cand_sum:
        raise TypeError("out_cand_sum must be a contiguous float32 array")
    if isinstance(out_token_logprob, np.ndarray) and k4 is not out_token_logprob:
        raise TypeError("out_token_logprob must be a contiguous float32 array")
    _check(getattr(lib(), _entry)(model, prefix, qo, co, ct, ot, os_))
    return out_token_logprob, out_cand_sum


def jet_score_candidates_noalloc(model, prefix, q_cand_offsets, cand_tok_offsets, cand_tokens,
                                 out_token_logprob=True, out_cand_sum=None):
    """jet_score_candidates with every work buffer in the library's fixed
    per-device scratch (no device allocation); same arguments and results."""
    return jet_score_candidates(model, prefix, q_cand_offsets, cand_tok_offsets, cand_tokens,
                                out_token_logprob, out_cand_sum, _entry="jet_score_candidates_noalloc")


def jet_decide(mode: int, q_cand_offsets, cand_sum):
    qo, k1 = _ptr(q_cand_offsets, np.int64)
    cs, k2 = _ptr(cand_sum, np.float32)
    n_q = len(k1) - 1
    q = np.empty(len(k2), np.float64)
    choice = np.empty(n_q, np.int32)
    value = np.full(n_q, np.nan)
    _check(lib().jet_decide(mode, n_q, qo, cs, q.ctypes.data_as(ctypes.c_void_p),
                            choice.ctypes.data_as(ctypes.c_void_p), value.ctypes.data_as(ctypes.c_void_p)))
    return q, choice, value


def jet_answer_classes(q_cand_offsets, cand_tok_offsets, cand_tokens):
    """Per candidate, the index within its question of the first candidate
    with the same token sequence (equivalent labels, Section 3.3)."""
    qo, k1 = _ptr(q_cand_offsets, np.int64)
    co, k2 = _ptr(cand_tok_offsets, np.int64)
    ct, k3 = _ptr(cand_tokens, np.int32)
    out = np.empty(len(k2) - 1, np.int32)
    _check(lib().jet_answer_classes(len(k1) - 1, qo, co, ct, out.ctypes.data_as(ctypes.c_void_p)))
    return out


def jet_evaluate(q_cand_offsets, cand_sum, gold, cand_class=None):
    """(correct[n_q], gold_nll[n_q], accuracy, mean_nll) against reference
    answers, equivalent labels pooled (Section 3.3; Section 5)."""
    qo, k1 = _ptr(q_cand_offsets, np.int64)
    cs, k2 = _ptr(cand_sum, np.float32)
    gd, k3 = _ptr(gold, np.int32)
    cc, k4 = (None, None) if cand_class is None else _ptr(cand_class, np.int32)
    n_q = len(k1) - 1
    correct = np.empty(n_q, np.int32)
    nll = np.empty(n_q, np.float64)
    acc, mnll = ctypes.c_double(), ctypes.c_double()
    _check(lib().jet_evaluate(n_q, qo, cs, cc, gd, correct.ctypes.data_as(ctypes.c_void_p),
                              nll.ctypes.data_as(ctypes.c_void_p), ctypes.byref(acc), ctypes.byref(mnll)))
    return correct, nll, acc.value, mnll.value


def jet_candidate_layout(prefix_offsets, q_cand_offsets, cand_tok_offsets, max_ctx: int = 0):
    po, k1 = _ptr(prefix_offsets, np.int64)
    qo, k2 = _ptr(q_cand_offsets, np.int64)
    co, k3 = _ptr(cand_tok_offsets, np.int64)
    n_q = len(k1) - 1
    n = ctypes.c_int64()
    _check(lib().jet_candidate_layout(n_q, po, qo, co, max_ctx, 0, ctypes.byref(n), None, None, None, None, None))
    R = n.value
    out = {k: np.empty(R, np.int32) for k in ("row_pos", "row_q", "row_c", "row_tok")}
    out["lm_row"] = np.empty(int(k3[-1]), np.int32)
    P = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    _check(lib().jet_candidate_layout(n_q, po, qo, co, max_ctx, R, ctypes.byref(n), P(out["row_pos"]),
                                      P(out["row_q"]), P(out["row_c"]), P(out["row_tok"]), P(out["lm_row"])))
    return out


def jet_stats_get(model) -> dict:
    s = jet_stats()
    _check(lib().jet_stats_get(model, ctypes.byref(s)))
    d = {k: getattr(s, k) for k in ("prefix_tokens", "prefix_evals", "cand_body_tokens", "scored_tokens",
                                     "lm_rows", "prefill_waves", "score_waves")}
    for f in ("kernel_launches", "kernel_ms", "kernel_flops", "kernel_bytes"):
        d[f] = dict(zip(KERNEL_CLASSES, list(getattr(s, f))))
    return d


def jet_stats_reset(model) -> None:
    _check(lib().jet_stats_reset(model))


def jet_model_info(model) -> dict:
    v, nl, mc, ni = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    dt = ctypes.c_int32()
    _check(lib().jet_model_info(model, ctypes.byref(v), ctypes.byref(nl), ctypes.byref(mc), ctypes.byref(dt),
                                ctypes.byref(ni)))
    return dict(vocab=v.value, n_layers=nl.value, max_ctx=mc.value, dtype=dt.value,
                f16_inexact_weights=ni.value)


def jet_routes_get(model, which: int) -> np.ndarray:
    """Experts chosen per (layer, row) by the latest prefill (0) or scoring
    (1) call: int32 [n_layers, rows, top_k], -1 where a layer routed no row."""
    rows, nl, k = ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int32()
    _check(lib().jet_routes_get(model, which, ctypes.byref(rows), ctypes.byref(nl), ctypes.byref(k), None, 0))
    out = np.empty((nl.value, rows.value, k.value), np.int32)
    _check(lib().jet_routes_get(model, which, None, None, None, out.ctypes.data_as(ctypes.c_void_p), out.size))
    return out


def jet_prefix_free(prefix) -> None:
    lib().jet_prefix_free(prefix)


def jet_model_free(model) -> None:
    lib().jet_model_free(model)
