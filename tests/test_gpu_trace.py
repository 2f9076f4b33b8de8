"""GPU: reasoning traces (Section 3.4) through the C ABI against the fp64
oracle.

The sampler's discrete choice is checked the way routing is: at every step
the GPU's token must be one the oracle's keys allow (its key within the
logit tolerance of the oracle's maximum, 2 x per-token tolerance / tau, or
2 x per-token tolerance at tau = 0), and the oracle then continues along the
GPU's trace. The candidates scored on the extended prefix are compared at
the scoring tolerances; the extended prefix also scores like a fresh prefill
of x || trace.
"""
import sys

import numpy as np
import pytest

import jet_synth
import oracle
from oracle import generate as og
from paper_2609_33874_amd import jet as J

from test_gpu_parity import TOL, check_parity

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, file=sys.__stderr__, flush=True)


def extended(wl, trace):
    pre = [np.concatenate([wl.prefix(q), trace[q]]).astype(np.int32) for q in range(wl.n_questions)]
    return jet_synth.from_lists(pre, [wl.candidates(q) for q in range(wl.n_questions)])


def gpu_trace_and_scores(path, wl, dtype, n, tau, seed, steps=None):
    m = J.jet_model_load(path, dtype=dtype)
    try:
        p = J.jet_prefill_prefix(m, wl.prefix_offsets, wl.prefix_tokens)
        try:
            parts = []
            for k in (steps or [n]):
                parts.append(J.jet_generate_trace(m, p, wl.n_questions, k, tau, seed))
            trace = np.concatenate(parts, axis=1)
            tok, sums = J.jet_score_candidates(m, p, wl.q_cand_offsets, wl.cand_tok_offsets, wl.cand_tokens)
        finally:
            J.jet_prefix_free(p)
        ext = extended(wl, trace)
        p2 = J.jet_prefill_prefix(m, ext.prefix_offsets, ext.prefix_tokens)
        try:
            tok2, sums2 = J.jet_score_candidates(m, p2, ext.q_cand_offsets, ext.cand_tok_offsets, ext.cand_tokens)
        finally:
            J.jet_prefix_free(p2)
    finally:
        J.jet_model_free(m)
    return trace, tok, sums, tok2, sums2


def model_path(spec, model_dir):
    if spec == "wide_ffn_bf16":
        # the small dense model with a 2048-wide FFN: the decode steps' down
        # projection (K = 2048, 4 rows) then takes the split-K GEMM path
        import os
        p = os.path.join(model_dir, "wide_ffn_bf16.jetm")
        if not os.path.exists(p):
            s = dict(jet_synth.MODEL_SPECS["small_gqa_bf16"])
            s["ffn"] = 2048
            jet_synth.write_model(p, s)
        return p
    return jet_synth.ensure_model(spec, cache_dir=model_dir)


CASES = [
    ("wide_ffn_bf16", "small", J.JET_F16, 0.8),
    ("small_gqa_bf16", "small", J.JET_FP32, 0.0),
    ("small_gqa_bf16", "small", J.JET_F16, 0.8),
    ("small_hybrid_bf16", "small_hybrid", J.JET_FP32, 0.8),
    ("small_hybrid_bf16", "small_hybrid", J.JET_F16, 0.0),
    ("small_hybrid_bf16", "small_hybrid", J.JET_BF16, 0.8),
    ("small_gqa_bf16", "small", J.JET_BF16, 1.0),
    ("small_moe_bf16", "small_moe", J.JET_FP32, 0.8),
]


@pytest.mark.parametrize("spec,wname,dtype,tau", CASES)
def test_trace_matches_oracle(spec, wname, dtype, tau, model_dir):
    path = model_path(spec, model_dir)
    wl = jet_synth.make_workload(wname, n_questions=4)
    n, seed = 5, 20260921
    log(f"[trace] {spec} dtype={dtype} tau={tau} Q={wl.n_questions} n={n}")
    trace, tok, sums, tok2, sums2 = gpu_trace_and_scores(path, wl, dtype, n, tau, seed)
    t_tol = TOL[dtype][0]
    key_tol = 2 * t_tol / tau if tau > 0 else 2 * t_tol
    model = oracle.Model(path)
    worst = 0.0
    for q in range(wl.n_questions):
        _, st = og.generate_trace(model, wl.prefix(q), q, n, tau, seed, forced=trace[q])
        for t, s in enumerate(st):
            gap = s["max_key"] - s["key"]
            worst = max(worst, gap)
            assert gap <= key_tol, f"question {q} step {t}: GPU token {trace[q][t]} is {gap:.3e} below the maximum"
    log(f"[trace] largest key gap of a GPU token {worst:.3e} (allowed {key_tol:.1e})")
    ext = extended(wl, trace)
    ref_tok, ref_sums = oracle.score_unshared(model, ext)
    dt, ds = check_parity(ext, tok, sums, ref_tok, ref_sums, dtype)
    log(f"[trace] scores on x || trace: max|d tok|={dt:.3e} max|d sum|={ds:.3e}")
    # the extended prefix scores like a fresh prefill of x || trace
    d_fresh = np.abs(tok.astype(np.float64) - tok2).max()
    assert d_fresh <= t_tol, d_fresh
    if dtype == J.JET_FP32:
        assert d_fresh <= 1e-5, d_fresh


@pytest.mark.parametrize("spec,wname", [("small_hybrid_bf16", "small_hybrid"), ("small_gqa_bf16", "small")])
def test_trace_in_parts_equals_one_call_greedy(spec, wname, model_dir):
    """Greedy tokens do not depend on the step counter, so traces of 2 + 4
    steps (the hybrid's convolution ring turns over mid-way) and of 6 steps
    in one call give the same tokens and scores."""
    path = jet_synth.ensure_model(spec, cache_dir=model_dir)
    wl = jet_synth.make_workload(wname, n_questions=3)
    tr1, tok1, s1, _, _ = gpu_trace_and_scores(path, wl, J.JET_FP32, 6, 0.0, 1)
    tr2, tok2, s2, _, _ = gpu_trace_and_scores(path, wl, J.JET_FP32, 6, 0.0, 1, steps=[2, 4])
    np.testing.assert_array_equal(tr1, tr2)
    assert np.abs(tok1.astype(np.float64) - tok2).max() <= 1e-5


def test_trace_zero_steps_and_errors(model_dir):
    path = jet_synth.ensure_model("small_gqa_bf16", cache_dir=model_dir)
    wl = jet_synth.make_workload("small", n_questions=3)
    m = J.jet_model_load(path, dtype=J.JET_F16, max_ctx=400)
    try:
        p = J.jet_prefill_prefix(m, wl.prefix_offsets, wl.prefix_tokens)
        try:
            tok0, _ = J.jet_score_candidates(m, p, wl.q_cand_offsets, wl.cand_tok_offsets, wl.cand_tokens)
            out = J.jet_generate_trace(m, p, wl.n_questions, 0, 0.5, 3)
            assert out.shape == (wl.n_questions, 0)
            tok1, _ = J.jet_score_candidates(m, p, wl.q_cand_offsets, wl.cand_tok_offsets, wl.cand_tokens)
            np.testing.assert_array_equal(tok0, tok1)
            for n, tau in ((-1, 0.0), (2, -0.5), (2, float("nan")), (2, float("inf"))):
                with pytest.raises(J.JetError) as e:
                    J.jet_generate_trace(m, p, wl.n_questions, n, tau, 3)
                assert e.value.code == J.JET_E_INVALID
            P = np.diff(wl.prefix_offsets)
            with pytest.raises(J.JetError) as e:
                J.jet_generate_trace(m, p, wl.n_questions, int(400 - P.max() + 1), 0.0, 3)
            assert e.value.code == J.JET_E_CAPACITY
            # unchanged after the refused calls
            tok2, _ = J.jet_score_candidates(m, p, wl.q_cand_offsets, wl.cand_tok_offsets, wl.cand_tokens)
            np.testing.assert_array_equal(tok0, tok2)
        finally:
            J.jet_prefix_free(p)
    finally:
        J.jet_model_free(m)
