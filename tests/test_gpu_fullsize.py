"""Full-size GPU parity: the real workload shapes in the launch configuration
that bench.py times (every question on the GPU, in the fp16 mode bench.py
times and in the pair-bf16 mode), checked against the fp64 oracle on sampled
questions and through properties that hold at any size.
"""
import contextlib
import os
import sys

import numpy as np
import pytest

import jet_synth
import oracle
from paper_2609_33874_amd import jet as J

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def dense_1p5b_path():
    return jet_synth.ensure_model("dense_1p5b")


# the fp16 mode (what bench.py times) and the pair-bf16 mode
DTYPES = [pytest.param(J.JET_F16, id="f16"), pytest.param(J.JET_BF16, id="bf16pair")]
# the 64-layer model: fp16 with attention-side pairs (what bench.py times
# there), and the pair-bf16 mode
DTYPES_DEEP = [pytest.param(J.JET_F16P, id="f16p"), pytest.param(J.JET_BF16, id="bf16pair")]


@pytest.fixture(scope="module")
def dense_1p5b_models(dense_1p5b_path):
    models = {}

    def get(dtype):
        if dtype not in models:
            for m in models.values():  # one copy of the weights at a time
                J.jet_model_free(m)
            models.clear()
            models[dtype] = J.jet_model_load(dense_1p5b_path, dtype=dtype)
        return models[dtype]
    yield get
    for m in models.values():
        J.jet_model_free(m)


@contextlib.contextmanager
def large_model(spec):
    """Path of a large model file; a file this test wrote is deleted afterwards
    (the largest files do not all fit on the disk at once)."""
    path = os.path.join(jet_synth.model_cache_dir(), f"{spec}_s{jet_synth.MASTER_SEED}.jetm")
    existed = os.path.exists(path)
    path = jet_synth.ensure_model(spec)
    try:
        yield path
    finally:
        if not existed and os.path.exists(path):
            os.remove(path)


def run(model, wl):
    p = J.jet_prefill_prefix(model, wl.prefix_offsets, wl.prefix_tokens)
    try:
        return J.jet_score_candidates(model, p, wl.q_cand_offsets, wl.cand_tok_offsets, wl.cand_tokens)
    finally:
        J.jet_prefix_free(p)


_ORACLE = {}


def oracle_subset(path, name, wl, qs):
    """Oracle scores of questions qs of workload `name` (cached across modes)."""
    key = (path, name, tuple(qs))
    if key not in _ORACLE:
        _ORACLE[key] = oracle.score_unshared(path, wl.subset(qs))
    return _ORACLE[key]


def sampled_parity(path, name, wl, tok, sums, qs, dtype):
    ref_tok, ref_sum = oracle_subset(path, name, wl, qs)
    got_tok = np.concatenate([tok[wl.cand_tok_offsets[wl.q_cand_offsets[q]]:
                                  wl.cand_tok_offsets[wl.q_cand_offsets[q + 1]]] for q in qs])
    got_sum = np.concatenate([sums[wl.q_cand_offsets[q]:wl.q_cand_offsets[q + 1]] for q in qs])
    dt = np.abs(got_tok - ref_tok).max()
    ds = np.abs(got_sum - ref_sum).max()
    log(f"[fullsize] {name} dtype {dtype} questions {qs}: max|d tok|={dt:.3e} max|d sum|={ds:.3e}")
    from conftest import record_parity
    record_parity(f"fullsize/{name}/dtype{dtype}/q{qs}", max_tok=dt, max_sum=ds)
    assert dt <= 2e-2 and ds <= 5e-2
    return ref_sum, got_sum


def properties(wl, tok, sums):
    assert np.all(np.isfinite(tok)) and np.all(tok <= 1e-4)
    # sums are the per-candidate sums of the token log-probs (Eq. 3)
    s = np.add.reduceat(tok.astype(np.float64), wl.cand_tok_offsets[:-1]) if len(tok) else tok
    np.testing.assert_allclose(sums, s, atol=1e-3, rtol=1e-5)


@pytest.mark.parametrize("dtype", DTYPES)
def test_dense_1p5b_k4_full(dtype, dense_1p5b_path, dense_1p5b_models):
    wl = jet_synth.make_workload("dense_1p5b_k4")
    log(f"[fullsize] dense_1p5b_k4 dtype {dtype}: {wl.n_questions} questions, "
        f"{int(wl.prefix_offsets[-1])} prefix tokens")
    model = dense_1p5b_models(dtype)
    tok, sums = run(model, wl)
    properties(wl, tok, sums)
    sampled_parity(dense_1p5b_path, "dense_1p5b_k4", wl, tok, sums, [0, 97, 255], dtype)
    st = J.jet_stats_get(model)
    assert st["prefix_tokens"] >= int(wl.prefix_offsets[-1])


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("name", ["dense_1p5b_binary", "dense_1p5b_ordinal"])
def test_dense_1p5b_decisions_full(name, dtype, dense_1p5b_path, dense_1p5b_models):
    wl = jet_synth.make_workload(name)
    log(f"[fullsize] {name} dtype {dtype}: {wl.n_questions} questions, {int(wl.prefix_offsets[-1])} prefix tokens")
    tok, sums = run(dense_1p5b_models(dtype), wl)
    properties(wl, tok, sums)
    ref_sum, got_sum = sampled_parity(dense_1p5b_path, name, wl, tok, sums, [0, wl.n_questions - 1], dtype)
    mode = J.JET_BINARY if name.endswith("binary") else J.JET_ORDINAL
    K = 2 if mode == J.JET_BINARY else 5
    qo = np.arange(0, len(ref_sum) + 1, K, dtype=np.int64)
    _, _, v_gpu = J.jet_decide(mode, qo, got_sum.astype(np.float32))
    qs_o, _, v_ref = oracle.decide("binary" if mode == J.JET_BINARY else "ordinal", qo, ref_sum)
    # sums within 5e-2 move q(true) / the expected level by at most ~K * 5e-2
    np.testing.assert_allclose(v_gpu, np.array(v_ref, dtype=np.float64), atol=0.05 * K)
    _, _, v_all = J.jet_decide(mode, wl.q_cand_offsets, sums)
    assert np.all(np.isfinite(v_all))
    if mode == J.JET_BINARY:
        assert np.all((v_all >= 0) & (v_all <= 1))
    else:
        assert np.all((v_all >= 0) & (v_all <= K - 1))


@pytest.mark.parametrize("dtype", DTYPES)
def test_hybrid_4b_k4_full(dtype):
    """4B-shape hybrid (24 delta-rule + 8 attention layers): all 128 questions
    on the GPU, the shortest-prefix question checked against the oracle."""
    path = jet_synth.ensure_model("hybrid_4b")
    wl = jet_synth.make_workload("hybrid_4b_k4")
    log(f"[fullsize] hybrid_4b_k4 dtype {dtype}: {wl.n_questions} questions, "
        f"{int(wl.prefix_offsets[-1])} prefix tokens")
    m = J.jet_model_load(path, dtype=dtype)
    try:
        tok, sums = run(m, wl)
    finally:
        J.jet_model_free(m)
    properties(wl, tok, sums)
    q = int(np.argmin(np.diff(wl.prefix_offsets)))
    sampled_parity(path, "hybrid_4b_k4", wl, tok, sums, [q], dtype)


# The fp64 oracle of a 35B-shape question reads every expert of every layer
# (minutes on the host).
@pytest.mark.timeout(900)
def test_moe_35b_a3b_k4_full():
    """35B-A3B-shape mixture-of-experts hybrid (30 delta-rule + 10 attention
    layers, 256 experts, top 8, shared expert): all 128 questions on the GPU
    in the fp16 mode (properties, bitwise the same on a second run), and the
    shortest-prefix question in the fp32 mode against the oracle.

    Routing is a discrete choice among router logits that lie close together
    (about 0.05 apart between the 8th and 9th of 256 at this initialisation):
    a rounding difference that reorders two of them swaps an expert, which
    moves the row's output by a finite step. At 40 layers x ~200 rows per
    sequence the fp16 mode's activation rounding does this many times per
    sequence, so its error against the fp64 oracle is logged, not bounded;
    the fp32 mode does it rarely, and is held to the 16-bit tolerance. The
    same head grouping and expert count are held to the fp32 tolerance at
    small size (test_gpu_edges.py)."""
    with large_model("moe_35b_a3b") as path:
        _moe_35b_a3b_k4_full(path)


def _moe_35b_a3b_k4_full(path):
    wl = jet_synth.make_workload("moe_35b_a3b_k4")
    log(f"[fullsize] moe_35b_a3b_k4: {wl.n_questions} questions, {int(wl.prefix_offsets[-1])} prefix tokens")
    m = J.jet_model_load(path, dtype=J.JET_F16)
    try:
        tok, sums = run(m, wl)
        tok2, sums2 = run(m, wl)
    finally:
        J.jet_model_free(m)
    np.testing.assert_array_equal(tok, tok2)
    np.testing.assert_array_equal(sums, sums2)
    properties(wl, tok, sums)
    q = int(np.argmin(np.diff(wl.prefix_offsets)))
    ref_tok, ref_sum = oracle_subset(path, "moe_35b_a3b_k4", wl, [q])
    sub = wl.subset([q])
    a, b = wl.cand_tok_offsets[wl.q_cand_offsets[q]], wl.cand_tok_offsets[wl.q_cand_offsets[q + 1]]
    log(f"[fullsize] moe f16 question {q}: max|d tok|={np.abs(tok[a:b] - ref_tok).max():.3e}")
    m = J.jet_model_load(path, dtype=J.JET_FP32)
    try:
        tok32, sums32 = run(m, sub)
    finally:
        J.jet_model_free(m)
    dt = np.abs(tok32 - ref_tok).max()
    ds = np.abs(sums32 - ref_sum).max()
    log(f"[fullsize] moe fp32 question {q}: max|d tok|={dt:.3e} max|d sum|={ds:.3e}")
    from conftest import record_parity
    record_parity(f"fullsize/moe_35b_a3b_k4/dtype{J.JET_FP32}/q{[q]}", max_tok=dt, max_sum=ds)
    assert dt <= 2e-2 and ds <= 5e-2


@pytest.fixture(scope="module")
def dense_27b_path():
    with large_model("dense_27b") as path:
        yield path


# The fp64 oracle of one 27B-shape candidate sequence runs for minutes on the
# host, longer than a per-test limit meant for GPU calls.
@pytest.mark.timeout(900)
@pytest.mark.parametrize("dtype", DTYPES_DEEP)
def test_dense_27b_k10_full(dtype, dense_27b_path):
    """27B-shape dense decoder (64 layers, d=5120): all 64 questions on the
    GPU; one whole candidate sequence (the shortest question's shortest
    candidate, ~1.1k positions) checked against the oracle, plus properties."""
    path = dense_27b_path
    wl = jet_synth.make_workload("dense_27b_k10")
    log(f"[fullsize] dense_27b_k10 dtype {dtype}: {wl.n_questions} questions, "
        f"{int(wl.prefix_offsets[-1])} prefix tokens")
    m = J.jet_model_load(path, dtype=dtype)
    try:
        tok, sums = run(m, wl)
    finally:
        J.jet_model_free(m)
    properties(wl, tok, sums)
    q = int(np.argmin(np.diff(wl.prefix_offsets)))
    cands = wl.candidates(q)
    j = int(np.argmin([len(y) for y in cands]))
    c = wl.q_cand_offsets[q] + j
    key = (path, "dense_27b_k10", q, j)
    if key not in _ORACLE:
        _ORACLE[key] = oracle.score_unshared(path, jet_synth.from_lists([wl.prefix(q)], [[cands[j]]]))
    ref_tok, ref_sum = _ORACLE[key]
    got = tok[wl.cand_tok_offsets[c]:wl.cand_tok_offsets[c + 1]]
    dt = np.abs(got - ref_tok).max()
    ds = abs(float(sums[c]) - float(ref_sum[0]))
    log(f"[fullsize] 27b dtype {dtype} question {q} candidate {j}: max|d tok|={dt:.3e} |d sum|={ds:.3e}")
    from conftest import record_parity
    record_parity(f"fullsize/dense_27b_k10/dtype{dtype}/q{q}c{j}", max_tok=dt, max_sum=ds)
    assert dt <= 2e-2 and ds <= 5e-2
