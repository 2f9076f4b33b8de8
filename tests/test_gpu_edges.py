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
    print(msg, flush=True)
    sys.stdout.flush()


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
