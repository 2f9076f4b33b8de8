"""jet_score_candidates_noalloc (every work buffer in the library's fixed
per-device scratch) against jet_score_candidates through the C ABI: two calls
in a row, the second with a smaller input, on dense, hybrid and
mixture-of-experts models and on the full-size dense 1.5B workload (many
waves of the scratch's size); the scratch-too-small error leaves the next
call unharmed. Tolerances as for the oracle parity (the two entry points run
the same kernels; only the split of the candidates into waves differs)."""
import sys

import numpy as np
import pytest

import jet_synth
from paper_2609_33874_amd import jet as J

pytestmark = pytest.mark.gpu

TOL = {J.JET_FP32: (1e-4, 1e-4), J.JET_F16: (2e-2, 5e-2)}


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def both(m, p, wl):
    ref = J.jet_score_candidates(m, p, wl.q_cand_offsets, wl.cand_tok_offsets, wl.cand_tokens)
    got = J.jet_score_candidates_noalloc(m, p, wl.q_cand_offsets, wl.cand_tok_offsets, wl.cand_tokens)
    return ref, got


def check(tag, wl, ref, got, dtype):
    t_tol, s_tol = TOL[dtype]
    dt = np.abs(got[0].astype(np.float64) - ref[0])
    ds = np.abs(got[1].astype(np.float64) - ref[1])
    log(f"[noalloc] {tag}: max|d tok|={dt.max():.3e} max|d sum|={ds.max():.3e} "
        f"bitwise={np.array_equal(got[0], ref[0]) and np.array_equal(got[1], ref[1])}")
    assert np.all(np.isfinite(got[0])) and np.all(np.isfinite(got[1]))
    assert dt.max() <= t_tol
    m = np.diff(wl.cand_tok_offsets)
    assert np.all(ds <= (m * t_tol if dtype == J.JET_FP32 else s_tol))


@pytest.mark.parametrize("spec,wname,dtype", [
    ("small_gqa_bf16", "small", J.JET_F16),
    ("small_gqa_fp32", "small", J.JET_FP32),
    ("small_hybrid_bf16", "small_hybrid", J.JET_F16),
    ("small_moe_bf16", "small_moe", J.JET_F16),
])
def test_noalloc_matches_scoring(spec, wname, dtype, model_dir):
    path = jet_synth.ensure_model(spec, cache_dir=model_dir)
    wl = jet_synth.make_workload(wname)
    small = wl.subset(list(range(3)))
    m = J.jet_model_load(path, dtype=dtype)
    try:
        for tag, w in (("call 1", wl), ("call 2 (smaller)", small)):
            p = J.jet_prefill_prefix(m, w.prefix_offsets, w.prefix_tokens)
            try:
                ref, got = both(m, p, w)
            finally:
                J.jet_prefix_free(p)
            check(f"{spec} {tag}", w, ref, got, dtype)
    finally:
        J.jet_model_free(m)


def test_noalloc_full_size_in_waves():
    """All 256 questions of the dense 1.5B choice workload: ~12k candidate
    rows, several waves of the scratch; then a smaller call."""
    path = jet_synth.ensure_model("dense_1p5b")
    wl = jet_synth.make_workload("dense_1p5b_k4")
    m = J.jet_model_load(path, dtype=J.JET_F16)
    try:
        for tag, w in (("full", wl), ("smaller", wl.subset(list(range(40))))):
            p = J.jet_prefill_prefix(m, w.prefix_offsets, w.prefix_tokens)
            try:
                waves0 = J.jet_stats_get(m)["score_waves"]
                ref = J.jet_score_candidates(m, p, w.q_cand_offsets, w.cand_tok_offsets, w.cand_tokens)
                waves1 = J.jet_stats_get(m)["score_waves"]
                got = J.jet_score_candidates_noalloc(m, p, w.q_cand_offsets, w.cand_tok_offsets, w.cand_tokens)
                waves2 = J.jet_stats_get(m)["score_waves"]
            finally:
                J.jet_prefix_free(p)
            log(f"[noalloc] dense_1p5b_k4 {tag}: waves {waves1 - waves0} (workspace) vs {waves2 - waves1} (scratch)")
            if tag == "full":
                assert waves2 - waves1 > 1
            check(f"dense_1p5b_k4 {tag}", w, ref, got, J.JET_F16)
    finally:
        J.jet_model_free(m)


def test_noalloc_capacity_error_then_next_call(model_dir):
    """A candidate whose rows cannot fit the scratch is refused with
    JET_E_CAPACITY, outputs untouched; the next call is unaffected."""
    path = jet_synth.ensure_model("small_gqa_bf16", cache_dir=model_dir)
    rng = np.random.default_rng(5)
    long = jet_synth.from_lists([rng.integers(0, 3000, 40).astype(np.int32)],
                                [[rng.integers(0, 3000, 8000).astype(np.int32)]])
    wl = jet_synth.make_workload("small", n_questions=4)
    m = J.jet_model_load(path, dtype=J.JET_F16)
    try:
        p = J.jet_prefill_prefix(m, long.prefix_offsets, long.prefix_tokens)
        try:
            out = np.full(1, 7.0, np.float32)
            with pytest.raises(J.JetError) as e:
                J.jet_score_candidates_noalloc(m, p, long.q_cand_offsets, long.cand_tok_offsets, long.cand_tokens,
                                               None, out)
            assert e.value.code == J.JET_E_CAPACITY
            assert out[0] == 7.0
        finally:
            J.jet_prefix_free(p)
        p = J.jet_prefill_prefix(m, wl.prefix_offsets, wl.prefix_tokens)
        try:
            ref, got = both(m, p, wl)
        finally:
            J.jet_prefix_free(p)
        check("after a refused call", wl, ref, got, J.JET_F16)
    finally:
        J.jet_model_free(m)
