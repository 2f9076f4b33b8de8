"""GPU parity at the edges of the kernels' tiling and of the request shapes,
against the fp64 oracle (same tolerances as test_gpu_parity.py):

* prefix lengths on both sides of the 64-key attention tiles (1, 63, 64, 65,
  127, 128, 129, 200) and candidate lengths 1, 2, 15, 16, 17, with a question
  that has no candidates;
* hybrid models: prefixes and candidates of 1..5 tokens, where the width-4
  convolution's history runs into the zero start of a prefix and from a
  candidate into its question's prefix tail;
* a call with no candidates at all.
"""
import sys

import numpy as np
import pytest

import jet_synth
import oracle
from paper_2609_33874_amd import jet as J

pytestmark = pytest.mark.gpu

TOL = {J.JET_FP32: 1e-4, J.JET_BF16: 2e-2, J.JET_F16: 2e-2, J.JET_F16P: 2e-2}


def log(msg):
    print(msg, file=sys.__stderr__, flush=True)


def edge_workload(vocab, prefix_lens, cand_lens, seed, empty_question=True):
    rng = np.random.default_rng(seed)
    prefixes, cands = [], []
    for i, p in enumerate(prefix_lens):
        prefixes.append(rng.integers(0, vocab, p).astype(np.int32))
        # rotate the candidate lengths so every prefix meets several of them
        ls = [cand_lens[(i + j) % len(cand_lens)] for j in range(3)]
        cands.append([rng.integers(0, vocab, m).astype(np.int32) for m in ls])
    if empty_question:
        prefixes.append(rng.integers(0, vocab, 7).astype(np.int32))
        cands.append([])
    return jet_synth.from_lists(prefixes, cands)


def score(path, wl, dtype):
    m = J.jet_model_load(path, dtype=dtype)
    try:
        p = J.jet_prefill_prefix(m, wl.prefix_offsets, wl.prefix_tokens)
        try:
            return J.jet_score_candidates(m, p, wl.q_cand_offsets, wl.cand_tok_offsets, wl.cand_tokens)
        finally:
            J.jet_prefix_free(p)
    finally:
        J.jet_model_free(m)


def compare(path, wl, dtype, name):
    tok, sums = score(path, wl, dtype)
    ref_tok, ref_sum = oracle.score_unshared(path, wl)
    t = TOL[dtype]
    m = np.diff(wl.cand_tok_offsets)
    dt = np.abs(tok.astype(np.float64) - ref_tok)
    ds = np.abs(sums.astype(np.float64) - ref_sum)
    log(f"[edges] {name} dtype {dtype}: {len(m)} candidates, max|d tok|={dt.max():.3e} max|d sum|={ds.max():.3e}")
    assert dt.max() <= t
    assert np.all(ds <= (m * t if dtype == J.JET_FP32 else 5e-2))


@pytest.mark.parametrize("dtype", [J.JET_BF16, J.JET_FP32, J.JET_F16, J.JET_F16P])
def test_attention_tile_boundaries(dtype, model_dir):
    path = jet_synth.ensure_model("small_gqa_bf16", cache_dir=model_dir)
    wl = edge_workload(3000, [1, 63, 64, 65, 127, 128, 129, 200], [1, 2, 15, 16, 17], seed=11)
    compare(path, wl, dtype, "tile boundaries")


@pytest.mark.parametrize("dtype", [J.JET_BF16, J.JET_FP32, J.JET_F16])
def test_hybrid_short_sequences(dtype, model_dir):
    path = jet_synth.ensure_model("small_hybrid_bf16", cache_dir=model_dir)
    vocab = jet_synth.read_header(path)["vocab"]
    wl = edge_workload(vocab, [1, 2, 3, 4, 5, 33], [1, 2, 3, 4, 5], seed=12)
    compare(path, wl, dtype, "hybrid short")


@pytest.mark.parametrize("a_log", [2.0, 6.0])
@pytest.mark.parametrize("dtype", [J.JET_FP32, J.JET_F16, J.JET_BF16])
def test_hybrid_strong_decay(dtype, a_log, model_dir):
    """Delta-rule layers with strong decay: alpha = exp(-e^A_log softplus(a +
    dt_bias)) with softplus of order 1 lies around e^-3..e^-8 for A_log = 2
    (the chunk's decay products span e^-100 and below) and below e^-150 for
    A_log = 6 (0 in fp32: the state is forgotten at every step), over
    prefixes that span several chunks of the chunked recurrence (fp16 and
    bf16-pair modes) with ragged tails."""
    import os
    path = os.path.join(model_dir, f"edge_hybrid_decay{int(a_log)}.jetm")
    if not os.path.exists(path):
        spec = dict(jet_synth.MODEL_SPECS["small_hybrid_bf16"])
        spec["gdn_a_log"] = a_log
        jet_synth.write_model(path, spec)
    vocab = jet_synth.read_header(path)["vocab"]
    wl = edge_workload(vocab, [1, 31, 32, 33, 95, 200], [1, 2, 7, 17], seed=14)
    compare(path, wl, dtype, f"hybrid decay A_log={a_log}")


def test_no_candidates(model_dir):
    path = jet_synth.ensure_model("small_gqa_bf16", cache_dir=model_dir)
    m = J.jet_model_load(path, dtype=J.JET_BF16)
    try:
        p = J.jet_prefill_prefix(m, [0, 5, 9], np.arange(1, 10, dtype=np.int32))
        tok, sums = J.jet_score_candidates(m, p, [0, 0, 0], [0], np.zeros(0, np.int32))
        assert len(tok) == 0 and len(sums) == 0
        J.jet_prefix_free(p)
    finally:
        J.jet_model_free(m)


WIDE = {
    # 8 query heads per KV head (the 35B-A3B shape's grouping)
    "wide_gqa": dict(arch="dense", dtype="bf16", d_model=256, n_layers=2, n_heads=16, n_kv_heads=2,
                     head_dim=128, ffn=256, vocab=2048, max_ctx=4096),
    # 256 experts, top 8 (the 35B-A3B shape's routing), small experts
    "many_experts": dict(arch="dense", dtype="bf16", d_model=256, n_layers=2, n_heads=2, n_kv_heads=1,
                         head_dim=128, ffn=64, vocab=2048, n_experts=256, top_k=8, moe_ffn=64,
                         shared_ffn=64, max_ctx=4096),
}


@pytest.mark.parametrize("name", sorted(WIDE))
def test_wide_grouping_and_many_experts(name, model_dir):
    """fp32-mode parity and run-to-run bitwise determinism at the 35B-A3B
    shape's head grouping and expert count."""
    import os
    path = os.path.join(model_dir, f"edge_{name}.jetm")
    if not os.path.exists(path):
        jet_synth.write_model(path, WIDE[name])
    wl = edge_workload(2048, [1, 40, 64, 65, 130, 300], [1, 2, 9, 17], seed=13, empty_question=False)
    compare(path, wl, J.JET_FP32, name)
    a = score(path, wl, J.JET_F16)
    b = score(path, wl, J.JET_F16)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


def test_model_freed_before_its_prefix():
    """Freeing a model first frees its live prefixes' buffers and detaches
    them: scoring against a detached prefix is refused, freeing it works, and
    the device is fine for the next model (jet.h, Ownership)."""
    path = jet_synth.ensure_model("small_gqa_bf16")
    wl = jet_synth.make_workload("small", n_questions=3)
    m = J.jet_model_load(path, dtype=J.JET_F16)
    p1 = J.jet_prefill_prefix(m, wl.prefix_offsets, wl.prefix_tokens)
    p2 = J.jet_prefill_prefix(m, wl.prefix_offsets, wl.prefix_tokens)
    J.jet_prefix_free(p2)          # one freed in order, one left alive
    ref_tok, ref_sum = J.jet_score_candidates(m, p1, wl.q_cand_offsets, wl.cand_tok_offsets, wl.cand_tokens)
    J.jet_model_free(m)
    m2 = J.jet_model_load(path, dtype=J.JET_F16)
    try:
        with pytest.raises(J.JetError) as e:
            J.jet_score_candidates(m2, p1, wl.q_cand_offsets, wl.cand_tok_offsets, wl.cand_tokens)
        assert e.value.code == J.JET_E_INVALID
        J.jet_prefix_free(p1)
        p3 = J.jet_prefill_prefix(m2, wl.prefix_offsets, wl.prefix_tokens)
        try:
            tok, sums = J.jet_score_candidates(m2, p3, wl.q_cand_offsets, wl.cand_tok_offsets, wl.cand_tokens)
        finally:
            J.jet_prefix_free(p3)
    finally:
        J.jet_model_free(m2)
    np.testing.assert_array_equal(tok, ref_tok)
    np.testing.assert_array_equal(sums, ref_sum)


def _inexact_f16(vals_bf16_bits, k):
    """How many bf16 values (bits) times 2^k numpy's fp16 rounding changes."""
    v = (vals_bf16_bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64) * 2.0 ** k
    return int(np.count_nonzero(v.astype(np.float16).astype(np.float64) != v))


def test_fp16_load_counts_inexact_weights(tmp_path):
    """The fp16 modes scale each matrix by 2^k (largest magnitude into
    [2^14, 2^15)) and convert; values far below the largest round. The loader
    reports how many: planted tiny values in one matrix change the count by
    exactly numpy's count of fp16 roundings of that matrix."""
    import shutil
    src = jet_synth.ensure_model("small_gqa_bf16")
    path = str(tmp_path / "planted.jetm")
    shutil.copy(src, path)
    m = J.jet_model_load(src, dtype=J.JET_F16)
    try:
        n0 = J.jet_model_info(m)["f16_inexact_weights"]
    finally:
        J.jet_model_free(m)
    h = jet_synth.read_header(path)
    t = next(t for t in h["tensors"] if t["name"] == "blk.0.wo")   # loaded as one matrix
    w = np.memmap(path, dtype=np.uint16, mode="r+", offset=t["offset"], shape=(t["nbytes"] // 2,))
    mag = ((w.astype(np.uint32) & 0x7FFF) << 16).view(np.float32)
    k = 14 - int(np.floor(np.log2(float(mag.max()))))
    before = _inexact_f16(np.array(w), k)
    # 2^-45 * (1 + 2^-7), -2^-40 * 1.5, 2^-50: far below fp16's step after scaling
    planted = np.array([2.0 ** -45 * (1 + 2.0 ** -7), -(2.0 ** -40) * 1.5, 2.0 ** -50], np.float32)
    w[[3, 1000, 5000]] = (planted.view(np.uint32) >> 16).astype(np.uint16)
    w.flush()
    after = _inexact_f16(np.array(w), k)
    del w
    assert after - before >= 2
    m = J.jet_model_load(path, dtype=J.JET_F16)
    try:
        n1 = J.jet_model_info(m)["f16_inexact_weights"]
    finally:
        J.jet_model_free(m)
    log(f"[edges] inexact fp16 weights: {n0} -> {n1} (numpy: {before} -> {after} in blk.0.wo)")
    assert n1 - n0 == after - before
