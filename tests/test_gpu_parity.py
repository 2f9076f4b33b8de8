"""GPU parity: the HIP scoring path, called through the C ABI, against the
fp64 oracle on the same seeded inputs.

Tolerances: per-token |d ell| <= 1e-4 and per-candidate |d s| <= m * 1e-4 in
the fp32 mode; per-token <= 2e-2 and per-candidate <= 5e-2 in the bf16 modes
(the single-bf16 mode only on 2-layer models: its rounding grows with depth,
and a 4-layer mixture-of-experts hybrid measured 0.26 per token); identical
argmax wherever the oracle's margin exceeds 0.1 nats; integer layout bit-exact.
"""
import os
import sys

import numpy as np
import pytest

import jet_synth
import oracle
from paper_2609_33874_amd import jet as J

pytestmark = pytest.mark.gpu

TOL = {J.JET_FP32: (1e-4, 1e-4), J.JET_BF16: (2e-2, 5e-2), J.JET_BF16_SINGLE: (2e-2, 5e-2),
       J.JET_F16: (2e-2, 5e-2), J.JET_F16P: (2e-2, 5e-2)}


def log(msg):
    print(msg, file=sys.__stderr__, flush=True)


def check_parity(wl, tok, sums, ref_tok, ref_sums, dtype):
    t_tol, s_tol = TOL[dtype]
    m = np.diff(wl.cand_tok_offsets)
    dt = np.abs(tok.astype(np.float64) - ref_tok)
    ds = np.abs(sums.astype(np.float64) - ref_sums)
    s_lim = m * t_tol if dtype == J.JET_FP32 else np.full(len(m), s_tol)
    assert dt.max() <= t_tol, f"per-token max |d| = {dt.max():.3e} at {dt.argmax()}"
    assert np.all(ds <= s_lim), f"per-candidate max |d| = {ds.max():.3e}"
    # decisions agree wherever the oracle margin exceeds 0.1 nats
    for q in range(wl.n_questions):
        a, b = wl.q_cand_offsets[q], wl.q_cand_offsets[q + 1]
        if b - a < 2:
            continue
        r = np.sort(ref_sums[a:b])
        if r[-1] - r[-2] > 0.1:
            assert np.argmax(sums[a:b]) == np.argmax(ref_sums[a:b])
    return dt.max(), ds.max()


def check_evaluation(wl, sums, ref_sums, max_ds):
    """Accuracy / gold NLL through the C ABI on the GPU's scores against the
    oracle's evaluation of its own scores, seeded gold labels. Each
    log-sum-exp moves by at most max|d s|, so the NLL by at most twice that."""
    rng = np.random.default_rng(11)
    K = np.diff(wl.q_cand_offsets)
    gold = np.array([rng.integers(0, k) for k in K], np.int32)
    cls = J.jet_answer_classes(wl.q_cand_offsets, wl.cand_tok_offsets, wl.cand_tokens)
    np.testing.assert_array_equal(cls, oracle.answer_classes(wl.q_cand_offsets, wl.cand_tok_offsets,
                                                             wl.cand_tokens))
    c, nll, _, _ = J.jet_evaluate(wl.q_cand_offsets, sums, gold, cls)
    oc, onll, _, _ = oracle.evaluate(wl.q_cand_offsets, ref_sums, gold, cls)
    assert np.abs(nll - onll).max() <= 2 * max_ds + 1e-12
    for q in range(wl.n_questions):
        a, b = wl.q_cand_offsets[q], wl.q_cand_offsets[q + 1]
        r = np.sort(ref_sums[a:b])
        if b - a < 2 or r[-1] - r[-2] > 0.1:
            assert c[q] == oc[q], q


def run_gpu(path, wl, dtype, **kw):
    m = J.jet_model_load(path, dtype=dtype, **kw)
    try:
        p = J.jet_prefill_prefix(m, wl.prefix_offsets, wl.prefix_tokens)
        try:
            tok, sums = J.jet_score_candidates(m, p, wl.q_cand_offsets, wl.cand_tok_offsets, wl.cand_tokens)
            stats = J.jet_stats_get(m)
        finally:
            J.jet_prefix_free(p)
    finally:
        J.jet_model_free(m)
    return tok, sums, stats


_ORACLE_CACHE = {}


def oracle_scores(path, name, wl):
    key = (path, name)
    if key not in _ORACLE_CACHE:
        _ORACLE_CACHE[key] = oracle.score_unshared(path, wl)
    return _ORACLE_CACHE[key]


CASES = [
    # (model spec, workload, dtype)
    ("tiny_dense_fp32", "tiny", J.JET_FP32),
    ("tiny_dense_bf16", "tiny", J.JET_BF16),
    ("small_gqa_bf16", "small", J.JET_BF16),
    ("small_gqa_bf16", "small", J.JET_FP32),
    ("small_gqa_bf16", "small", J.JET_BF16_SINGLE),
    ("tiny_dense_bf16", "tiny", J.JET_BF16_SINGLE),
    ("small_hybrid_fp32", "small_hybrid", J.JET_FP32),
    ("small_hybrid_bf16", "small_hybrid", J.JET_BF16),
    ("small_hybrid_bf16", "small_hybrid", J.JET_FP32),
    ("tiny_dense_bf16", "tiny", J.JET_F16),
    ("small_gqa_bf16", "small", J.JET_F16),
    ("small_hybrid_bf16", "small_hybrid", J.JET_F16),
    ("small_gqa_bf16", "small", J.JET_F16P),
    ("small_hybrid_bf16", "small_hybrid", J.JET_F16P),
    # mixture-of-experts FFN (no pair-bf16 mode for it)
    ("small_moe_fp32", "small_moe", J.JET_FP32),
    ("small_moe_bf16", "small_moe", J.JET_FP32),
    ("small_moe_bf16", "small_moe", J.JET_F16),
    ("small_moe_bf16", "small_moe", J.JET_F16P),
    ("tiny_moe_bf16", "tiny_moe", J.JET_BF16_SINGLE),
    ("tiny_moe_bf16", "tiny_moe", J.JET_F16),
    ("tiny_moe_bf16", "tiny_moe_long", J.JET_F16),   # 256-row expert tiles in the prefill
    # block-quantized weights: dequantized at load (fp32), int8 in the GEMMs (fp16)
    ("small_gqa_q8", "small_q8", J.JET_FP32),
    ("small_gqa_q8", "small_q8", J.JET_F16),
    ("small_gqa_q4", "small_q4", J.JET_FP32),
    ("small_gqa_q4", "small_q4", J.JET_F16),
]


@pytest.mark.parametrize("spec,wname,dtype", CASES)
def test_scores_match_oracle(spec, wname, dtype, model_dir):
    path = jet_synth.ensure_model(spec, cache_dir=model_dir)
    wl = jet_synth.make_workload(wname)
    log(f"[parity] {spec} {wname} dtype={dtype} Q={wl.n_questions} N={wl.n_candidates}")
    ref_tok, ref_sums = oracle_scores(path, wname, wl)
    tok, sums, stats = run_gpu(path, wl, dtype)
    dt, ds = check_parity(wl, tok, sums, ref_tok, ref_sums, dtype)
    log(f"[parity] max|d tok|={dt:.3e} max|d sum|={ds:.3e}")
    from conftest import record_parity
    record_parity(f"{spec}/{wname}/dtype{dtype}", max_tok=dt, max_sum=ds)
    check_evaluation(wl, sums, ref_sums, ds)
    # work counters follow the closed forms of shared-prefix evaluation (Section 4.1)
    P = np.diff(wl.prefix_offsets)
    m = np.diff(wl.cand_tok_offsets)
    assert stats["prefix_tokens"] == P.sum()
    assert stats["prefix_evals"] == wl.n_questions
    assert stats["cand_body_tokens"] == (m - 1).sum()
    # one LM-head row per scored token: the first token's logits are taken
    # again per candidate so that its target logit comes from the same tile
    # as its log-sum-exp
    assert stats["lm_rows"] == m.sum()


@pytest.mark.parametrize("spec,wname", [("small_gqa_bf16", "small"), ("small_hybrid_bf16", "small_hybrid")])
def test_prefix_sharing_matches_unshared_on_gpu(spec, wname, model_dir):
    """Unshared evaluation (each candidate with its own copy of the prefix,
    K P prefix tokens) gives the same scores as shared evaluation (P tokens)."""
    path = jet_synth.ensure_model(spec, cache_dir=model_dir)
    wl = jet_synth.make_workload(wname, n_questions=6)
    tok_s, sum_s, st_s = run_gpu(path, wl, J.JET_FP32)
    pre, cands = [], []
    for q in range(wl.n_questions):
        for y in wl.candidates(q):
            pre.append(wl.prefix(q)); cands.append([y])
    un = jet_synth.from_lists(pre, cands)
    tok_u, sum_u, st_u = run_gpu(path, un, J.JET_FP32)
    np.testing.assert_allclose(tok_u, tok_s, atol=2e-5, rtol=0)
    K = np.diff(wl.q_cand_offsets)
    P = np.diff(wl.prefix_offsets)
    assert st_s["prefix_tokens"] == P.sum()
    assert st_u["prefix_tokens"] == (K * P).sum()


def test_waves_and_budgets_do_not_change_scores(model_dir):
    path = jet_synth.ensure_model("small_gqa_bf16", cache_dir=model_dir)
    wl = jet_synth.make_workload("small", n_questions=8)
    a_tok, a_sum, _ = run_gpu(path, wl, J.JET_FP32)
    b_tok, b_sum, st = run_gpu(path, wl, J.JET_FP32, prefill_token_budget=300, wave_token_budget=20)
    assert st["prefill_waves"] > 1 and st["score_waves"] > 1
    np.testing.assert_allclose(b_tok, a_tok, atol=1e-5, rtol=0)


@pytest.mark.parametrize("dtype", [J.JET_BF16, J.JET_F16, J.JET_F16P])
def test_duplicates_permutation_and_determinism(dtype, model_dir):
    path = jet_synth.ensure_model("small_gqa_bf16", cache_dir=model_dir)
    base = jet_synth.make_workload("small", n_questions=4)
    pre, cands, perm_idx = [], [], []
    rng = np.random.default_rng(3)
    for q in range(base.n_questions):
        cs = base.candidates(q)
        cs = cs + [cs[0].copy()]                  # a duplicate of the first candidate
        perm = rng.permutation(len(cs))
        pre.append(base.prefix(q)); cands.append([cs[i] for i in perm])
        perm_idx.append(perm)
    wl = jet_synth.from_lists(pre, cands)
    t1, s1, _ = run_gpu(path, wl, dtype)
    t2, s2, _ = run_gpu(path, wl, dtype)
    np.testing.assert_array_equal(t1, t2)        # run to run: bitwise
    np.testing.assert_array_equal(s1, s2)
    _, s0, _ = run_gpu(path, base, dtype)
    for q in range(base.n_questions):
        a = wl.q_cand_offsets[q]
        perm = perm_idx[q]
        got = s1[a:a + len(perm)]
        orig = np.concatenate([s0[base.q_cand_offsets[q]:base.q_cand_offsets[q + 1]],
                               s0[base.q_cand_offsets[q]:base.q_cand_offsets[q] + 1]])
        np.testing.assert_allclose(got, orig[perm], atol=5e-2, rtol=0)
        # the two copies of the duplicated candidate score identically
        dup = [i for i, p in enumerate(perm) if p in (0, len(perm) - 1)]
        assert got[dup[0]] == got[dup[1]]


@pytest.mark.parametrize("dtype", [J.JET_F16, J.JET_F16P])
@pytest.mark.parametrize("spec,wname", [("small_gqa_bf16", "small"), ("small_hybrid_bf16", "small_hybrid"),
                                        ("small_moe_bf16", "small_moe")])
def test_reused_prefix_buffers(spec, wname, dtype, model_dir):
    """A prefix's device buffers go back to the model's pool when it is freed
    and the next prefill takes them with their old contents: scores must not
    depend on that (every buffer is written before it is read)."""
    path = jet_synth.ensure_model(spec, cache_dir=model_dir)
    a = jet_synth.make_workload(wname, n_questions=6)
    b = jet_synth.make_workload(wname, n_questions=6, seed=7)
    m = J.jet_model_load(path, dtype=dtype)
    try:
        def run(wl):
            p = J.jet_prefill_prefix(m, wl.prefix_offsets, wl.prefix_tokens)
            try:
                return J.jet_score_candidates(m, p, wl.q_cand_offsets, wl.cand_tok_offsets, wl.cand_tokens)
            finally:
                J.jet_prefix_free(p)
        ta, sa = run(a)        # fresh buffers
        run(b)                 # same sizes class, other contents
        ta2, sa2 = run(a)      # buffers reused from the pool
        np.testing.assert_array_equal(ta, ta2)
        np.testing.assert_array_equal(sa, sa2)
        # a second live prefix while the first is held: distinct buffers
        p1 = J.jet_prefill_prefix(m, a.prefix_offsets, a.prefix_tokens)
        p2 = J.jet_prefill_prefix(m, b.prefix_offsets, b.prefix_tokens)
        try:
            t1, _ = J.jet_score_candidates(m, p1, a.q_cand_offsets, a.cand_tok_offsets, a.cand_tokens)
            np.testing.assert_array_equal(t1, ta)
        finally:
            J.jet_prefix_free(p2)
            J.jet_prefix_free(p1)
    finally:
        J.jet_model_free(m)


@pytest.mark.parametrize("dtype", [J.JET_BF16, J.JET_F16])
def test_device_resident_inputs_and_outputs(dtype, model_dir):
    import torch
    path = jet_synth.ensure_model("small_gqa_bf16", cache_dir=model_dir)
    wl = jet_synth.make_workload("small", n_questions=5)
    h_tok, h_sum, _ = run_gpu(path, wl, dtype)
    dev = torch.device("cuda:0")
    m = J.jet_model_load(path, dtype=dtype)
    try:
        pt = torch.from_numpy(wl.prefix_tokens).to(dev)
        ct = torch.from_numpy(wl.cand_tokens).to(dev)
        p = J.jet_prefill_prefix(m, wl.prefix_offsets, pt)
        o_tok = torch.empty(len(wl.cand_tokens), dtype=torch.float32, device=dev)
        o_sum = torch.empty(wl.n_candidates, dtype=torch.float32, device=dev)
        J.jet_score_candidates(m, p, wl.q_cand_offsets, wl.cand_tok_offsets, ct, o_tok, o_sum)
        np.testing.assert_array_equal(o_tok.cpu().numpy(), h_tok)
        np.testing.assert_array_equal(o_sum.cpu().numpy(), h_sum)
        bad = ct.clone()
        bad[3] = 10 ** 6
        before = o_sum.clone()
        with pytest.raises(J.JetError) as e:
            J.jet_score_candidates(m, p, wl.q_cand_offsets, wl.cand_tok_offsets, bad, o_tok, o_sum)
        assert e.value.code == J.JET_E_INVALID
        assert torch.equal(before, o_sum)  # outputs untouched on error
        J.jet_prefix_free(p)
    finally:
        J.jet_model_free(m)


def test_error_paths_on_gpu(model_dir):
    path = jet_synth.ensure_model("tiny_dense_fp32", cache_dir=model_dir)
    for dt in (J.JET_BF16, J.JET_F16):
        with pytest.raises(J.JetError) as e:
            J.jet_model_load(path, dtype=dt)  # f32 weights are not bf16 values
        assert e.value.code == J.JET_E_INVALID
    m = J.jet_model_load(path, dtype=J.JET_FP32, max_ctx=40)
    try:
        with pytest.raises(J.JetError) as e:
            J.jet_prefill_prefix(m, [0, 3], np.array([1, 2, 5000], np.int32))
        assert e.value.code == J.JET_E_INVALID
        with pytest.raises(J.JetError) as e:
            J.jet_prefill_prefix(m, [0, 41], np.zeros(41, np.int32))
        assert e.value.code == J.JET_E_CAPACITY
        p = J.jet_prefill_prefix(m, [0, 38], np.zeros(38, np.int32))
        out = np.full(1, 7.0, np.float32)
        with pytest.raises(J.JetError) as e:  # 38 + 4 - 1 > 40
            J.jet_score_candidates(m, p, [0, 1], [0, 4], np.ones(4, np.int32), None, out)
        assert e.value.code == J.JET_E_CAPACITY
        assert out[0] == 7.0
        J.jet_score_candidates(m, p, [0, 1], [0, 3], np.ones(3, np.int32), None, out)
        J.jet_prefix_free(p)
    finally:
        J.jet_model_free(m)


def test_moe_rejects_pair_mode(model_dir):
    path = jet_synth.ensure_model("small_moe_bf16", cache_dir=model_dir)
    with pytest.raises(J.JetError) as e:
        J.jet_model_load(path, dtype=J.JET_BF16)
    assert e.value.code == J.JET_E_INVALID


def test_device_budget_oom(model_dir):
    path = jet_synth.ensure_model("small_gqa_bf16", cache_dir=model_dir)
    with pytest.raises(J.JetError) as e:
        J.jet_model_load(path, dtype=J.JET_BF16, max_device_bytes=1 << 16)
    assert e.value.code == J.JET_E_OOM


@pytest.mark.parametrize("spec,wname,dtype",
                         [(s, w, d) for s, w in (("small_hybrid_bf16", "small_hybrid"), ("small_gqa_bf16", "small"))
                          for d in (J.JET_BF16, J.JET_F16, J.JET_F16P)] +
                         [("small_moe_bf16", "small_moe", d) for d in (J.JET_F16, J.JET_BF16_SINGLE)])
def test_candidate_isolation_on_gpu(spec, wname, dtype, model_dir):
    """A candidate scored together with its siblings equals the same candidate
    scored alone against the same prefix, bitwise: the forked recurrent state
    and the own-suffix attention never see a sibling (Section 4.1, 5.6)."""
    path = jet_synth.ensure_model(spec, cache_dir=model_dir)
    wl = jet_synth.make_workload(wname, n_questions=3)
    m = J.jet_model_load(path, dtype=dtype)
    try:
        p = J.jet_prefill_prefix(m, wl.prefix_offsets, wl.prefix_tokens)
        tok, sums = J.jet_score_candidates(m, p, wl.q_cand_offsets, wl.cand_tok_offsets, wl.cand_tokens)
        for q in range(wl.n_questions):
            for j, y in enumerate(wl.candidates(q)):
                c = wl.q_cand_offsets[q] + j
                qco = np.zeros(wl.n_questions + 1, np.int64)
                qco[q + 1:] = 1
                t1, s1 = J.jet_score_candidates(m, p, qco, [0, len(y)], y)
                np.testing.assert_array_equal(t1, tok[wl.cand_tok_offsets[c]:wl.cand_tok_offsets[c + 1]])
                assert s1[0] == sums[c]
        J.jet_prefix_free(p)
    finally:
        J.jet_model_free(m)


@pytest.mark.parametrize("dtype", [J.JET_FP32, J.JET_F16])
def test_moe_routes_recorded_and_valid(dtype, model_dir):
    """The experts the GPU kept (JET_FLAG_RECORD_ROUTES) are a top-k of the
    oracle's logits up to rounding, and the oracle run on exactly those sets
    matches the GPU's scores at the mode's tolerance; recording does not
    change the scores."""
    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    from _routes import candidate_routes
    spec = "small_moe_fp32" if dtype == J.JET_FP32 else "small_moe_bf16"
    path = jet_synth.ensure_model(spec, cache_dir=model_dir)
    wl = jet_synth.make_workload("small_moe")
    m = J.jet_model_load(path, dtype=dtype, flags=J.JET_FLAG_RECORD_ROUTES)
    try:
        p = J.jet_prefill_prefix(m, wl.prefix_offsets, wl.prefix_tokens)
        try:
            tok, sums = J.jet_score_candidates(m, p, wl.q_cand_offsets, wl.cand_tok_offsets, wl.cand_tokens)
            pre, cand = J.jet_routes_get(m, 0), J.jet_routes_get(m, 1)
        finally:
            J.jet_prefix_free(p)
    finally:
        J.jet_model_free(m)
    h = jet_synth.read_header(path)
    L, k, T = h["n_layers"], h["top_k"], int(wl.prefix_offsets[-1])
    assert pre.shape == (L, T, k) and cand.shape == (L, int(np.sum(np.diff(wl.cand_tok_offsets) - 1)), k)
    # every body row routed by every layer; prefix rows by every layer but
    # the last (an attention layer: it runs only each question's last row)
    last = wl.prefix_offsets[1:] - 1
    assert h["layer_types"][-1] == "attn"
    assert np.all(pre[:-1] >= 0) and np.all(cand >= 0) and np.all(pre[-1, last] >= 0)
    assert np.count_nonzero(pre[-1, :, 0] >= 0) == wl.n_questions and np.all(pre[-1][pre[-1, :, 0] < 0] == -1)
    assert np.all(pre < h["n_experts"]) and np.all(cand < h["n_experts"])
    srt = np.sort(np.concatenate([pre[:-1].reshape(-1, k), cand.reshape(-1, k)]), axis=1)
    assert np.all(srt[:, 1:] != srt[:, :-1])  # distinct experts per row
    ref = run_gpu(path, wl, dtype)
    np.testing.assert_array_equal(tok, ref[0])
    qs = list(range(wl.n_questions))
    gaps = []
    ref_tok, ref_sum = oracle.score_unshared(path, wl.subset(qs), routes=candidate_routes(wl, pre, cand, qs),
                                             route_gaps=gaps)
    g = np.concatenate(gaps)
    log(f"[routes] {spec} dtype {dtype}: {len(g)} rows, {int(np.sum(g < 0))} not the oracle's top-k, "
        f"smallest margin {g.min():.3e}")
    assert g.min() >= -(1e-3 if dtype == J.JET_FP32 else 2e-2)
    check_parity(wl, tok, sums, ref_tok, ref_sum, dtype)


@pytest.mark.parametrize("spec", ["small_gqa_q8", "small_gqa_q4"])
def test_block_quantized_modes_and_gemm_tiles(spec, model_dir):
    """Block-quantized model (int8 or int4 blocks): the modes without a
    quantized GEMM path are refused; a prefill long enough for 256x256
    quantized tiles matches the oracle in fp16."""
    path = jet_synth.ensure_model(spec, cache_dir=model_dir)
    for dt in (J.JET_BF16, J.JET_F16P, J.JET_BF16_SINGLE):
        with pytest.raises(J.JetError) as e:
            J.jet_model_load(path, dtype=dt)
        assert e.value.code == J.JET_E_INVALID
    # 3 questions of ~7.9k prefix tokens: the gate/up GEMM (23.7k x 1536) has
    # 93 x 6 tiles of 256x256 (>= 512: the 256-row quantized tiles), the
    # others run 128x128 tiles with a ragged last row tile
    rng = np.random.default_rng(3)
    pre = [rng.integers(0, 3000, n).astype(np.int32) for n in (7950, 7900, 7861)]
    cands = [[rng.integers(0, 3000, m).astype(np.int32) for m in (1, 5, 17)], [rng.integers(0, 3000, 9).astype(np.int32)],
             [rng.integers(0, 3000, 3).astype(np.int32)]]
    wl = jet_synth.from_lists(pre, cands)
    tok, sums, _ = run_gpu(path, wl, J.JET_F16)
    ref_tok, ref_sum = oracle.score_unshared(path, wl)
    dt, ds = check_parity(wl, tok, sums, ref_tok, ref_sum, J.JET_F16)
    log(f"[{spec}] long prefill: max|d tok|={dt:.3e} max|d sum|={ds:.3e}")
