"""Pins of the fp64 oracle against values fixed by the paper and by mathematics.

Each check is independent of the oracle's own formulas: the paper's worked
example, closed forms, invariants, brute force, and independent library
implementations of the same network blocks (transformers' Qwen2 decoder and
Qwen3-Next gated delta-rule layer, evaluated on the same weights).
"""
import copy
import json
import math
import os

import numpy as np
import pytest
import scipy.special

import jet_synth
import oracle
from oracle import model as om

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _spec(name, **over):
    s = dict(jet_synth.MODEL_SPECS[name])
    s.update(over)
    return s


@pytest.fixture(scope="module")
def tiny_path(model_dir):
    return jet_synth.ensure_model("tiny_dense_fp32", cache_dir=model_dir)


@pytest.fixture(scope="module")
def micro_hybrid_path(model_dir):
    return jet_synth.ensure_model("micro_hybrid_fp32", cache_dir=model_dir)


@pytest.fixture(scope="module")
def pin_dense_path(model_dir):
    # larger init so every term of every block moves the result visibly
    p = os.path.join(model_dir, "pin_dense.jetm")
    if not os.path.exists(p):
        jet_synth.write_model(p, _spec("tiny_dense_fp32", n_heads=4, n_kv_heads=2,
                                       init_std=0.08, vocab=300))
    return p


@pytest.fixture(scope="module")
def pin_hybrid_path(model_dir):
    p = os.path.join(model_dir, "pin_hybrid.jetm")
    if not os.path.exists(p):
        jet_synth.write_model(p, _spec("micro_hybrid_fp32", init_std=0.15))
    return p


@pytest.fixture(scope="module")
def pin_moe_path(model_dir):
    p = os.path.join(model_dir, "pin_moe.jetm")
    if not os.path.exists(p):
        jet_synth.write_model(p, _spec("micro_moe_fp32", init_std=0.15))
    return p


# --------------------------------------------------------------------------
# Section 3.1-3.3: log-probabilities, sums, normalisation, decisions
# --------------------------------------------------------------------------

def test_worked_example_normalisation():
    g = json.load(open(os.path.join(GOLDEN, "worked_example.json")))
    s = np.log(np.array(g["likelihoods"]))
    q = oracle.normalize(s)
    np.testing.assert_allclose(q, g["normalized"], rtol=0, atol=1e-15)
    assert oracle.decide_choice(s) == 0


def test_log_softmax_brute_force_sums_to_one():
    rng = np.random.default_rng(1)
    z = rng.normal(0, 3.0, size=(6, 1024))
    V = z.shape[1]
    for r in range(z.shape[0]):
        ell = oracle.log_softmax_rows(np.repeat(z[r:r + 1], V, axis=0), np.arange(V))
        assert abs(np.sum(np.exp(ell)) - 1.0) < 1e-12
        # the unshifted textbook form agrees for moderate logits
        naive = z[r] - np.log(np.sum(np.exp(z[r])))
        np.testing.assert_allclose(ell, naive, atol=1e-13, rtol=0)
        np.testing.assert_allclose(ell, z[r] - scipy.special.logsumexp(z[r]), atol=1e-13, rtol=0)


def test_log_softmax_large_logits_stay_finite():
    z = np.array([[1000.0, 999.0, -1000.0]])
    ell = oracle.log_softmax_rows(np.repeat(z, 3, 0), np.arange(3))
    assert np.all(np.isfinite(ell[:2]))
    np.testing.assert_allclose(ell[:2], [-math.log1p(math.exp(-1.0)), -1.0 - math.log1p(math.exp(-1.0))],
                               atol=1e-12)


def test_decisions_closed_forms():
    s = np.array([-3.2, -1.5])
    assert oracle.decide_binary(s) == pytest.approx(1.0 / (1.0 + math.exp(-(s[1] - s[0]))), abs=1e-15)
    s5 = np.array([-4.0, -2.0, -2.5, -7.0, -3.0])
    q = oracle.normalize(s5)
    # equal scores: lowest index wins; duplicates split the mass
    assert oracle.decide_choice(np.array([-1.0, -0.5, -0.5])) == 1
    np.testing.assert_allclose(oracle.normalize(np.array([-2.0, -2.0])), [0.5, 0.5], atol=1e-16)
    # a constant shift of every score leaves q unchanged (Eq. 4)
    np.testing.assert_allclose(oracle.normalize(s5 + 123.0), q, atol=1e-15)
    with pytest.raises(ValueError):
        oracle.decide_binary(s5)


def _ordinal_pins(decide_ordinal):
    """Hand values of the expected zero-based level (Section 3.3, Eq. 5's
    ordinal rule with levels 0..K-1 in supplied order)."""
    g = json.load(open(os.path.join(GOLDEN, "worked_example.json")))
    # worked example as a two-level scale: q = (0.75, 0.25) -> E = 0 * 0.75 + 1 * 0.25
    assert decide_ordinal(np.log(np.array(g["likelihoods"]))) == pytest.approx(0.25, abs=1e-15)
    # K equal scores: q uniform, E = (K - 1) / 2
    for K in (2, 3, 5, 10):
        assert decide_ordinal(np.full(K, -3.7)) == pytest.approx((K - 1) / 2, abs=1e-13)
    # one level 60 nats ahead: E is its (zero-based) index to exp(-60)*K^2
    for K, j in ((5, 0), (5, 3), (7, 6)):
        s = np.full(K, -80.0)
        s[j] = -20.0
        assert decide_ordinal(s) == pytest.approx(j, abs=1e-20 + 1e-24 * K)
    # two levels: E equals q(level 1), i.e. the binary rule sigma(s1 - s0)
    for s in ([-3.2, -1.5], [0.0, -9.0], [2.0, 2.0]):
        assert decide_ordinal(np.array(s)) == pytest.approx(1.0 / (1.0 + math.exp(s[0] - s[1])), abs=1e-15)
    # three levels with q = (1/2, 1/3, 1/6): E = 1/3 + 2/6 = 2/3
    assert decide_ordinal(np.log([3.0, 2.0, 1.0])) == pytest.approx(2.0 / 3.0, abs=1e-15)


def test_decide_ordinal_hand_values():
    _ordinal_pins(oracle.decide_ordinal)


@pytest.mark.parametrize("mistake", ["one_based", "reversed_levels", "unnormalised"])
def test_decide_ordinal_pin_detects_planted_mistakes(mistake):
    def planted(s):
        q = oracle.normalize(s) if mistake != "unnormalised" else np.exp(np.asarray(s) - np.max(s))
        K = len(q)
        lev = {"one_based": np.arange(1, K + 1), "reversed_levels": np.arange(K)[::-1],
               "unnormalised": np.arange(K)}[mistake]
        return float(np.sum(lev * q))
    with pytest.raises(AssertionError):
        _ordinal_pins(planted)


def test_evaluation_closed_forms():
    """Accuracy and gold NLL (Section 5) with pooled equivalent labels
    (Section 3.3), against values fixed by the paper and by closed forms."""
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "worked_example.json")))
    s = np.log(np.array(g["likelihoods"]))
    # worked example: q = (0.75, 0.25); gold = first label -> -ln 0.75, correct
    c, nll, acc, mnll = oracle.evaluate([0, 2], s, [0])
    assert c[0] == 1 and nll[0] == pytest.approx(-math.log(g["normalized"][0]), abs=1e-15)
    c, nll, _, _ = oracle.evaluate([0, 2], s, [1])
    assert c[0] == 0 and nll[0] == pytest.approx(-math.log(g["normalized"][1]), abs=1e-15)
    # equal scores over K labels, r of them with the gold text: NLL = ln(K / r)
    K = 6
    cls = np.array([0, 1, 0, 3, 0, 5], np.int32)  # labels 0, 2, 4 share a text
    for gold, r in ((2, 3), (1, 1), (5, 1)):
        c, nll, _, _ = oracle.evaluate([0, K], np.full(K, -2.5), [gold], cls)
        assert nll[0] == pytest.approx(math.log(K / r), abs=1e-15)
        # ties go to label 0, whose text is accepted only for the first group
        assert c[0] == int(cls[gold] == 0)
    # any label with the gold text is accepted: predicted label 2, gold label 0
    c, nll, _, _ = oracle.evaluate([0, 3], np.array([-3.0, -9.0, -1.0]), [0], np.array([0, 1, 0]))
    assert c[0] == 1
    z = math.exp(-3.0) + math.exp(-9.0) + math.exp(-1.0)
    assert nll[0] == pytest.approx(-math.log((math.exp(-3.0) + math.exp(-1.0)) / z), abs=1e-14)
    # binary: gold true -> softplus(s0 - s1); correct iff q(true) > 1/2
    rng = np.random.default_rng(3)
    for _ in range(50):
        sb = rng.normal(-5, 2, size=2)
        if rng.random() < 0.2:
            sb[1] = sb[0]
        c, nll, _, _ = oracle.evaluate([0, 2], sb, [1])
        assert nll[0] == pytest.approx(math.log1p(math.exp(sb[0] - sb[1])), abs=1e-13)
        assert c[0] == int(oracle.decide_binary(sb) > 0.5)
    # a question with one candidate: certain, correct
    c, nll, _, _ = oracle.evaluate([0, 1], np.array([-40.0]), [0])
    assert c[0] == 1 and nll[0] == 0.0
    # means over questions
    qco = [0, 2, 5, 6]
    sm = np.array([-1.0, -2.0, -3.0, -3.0, -3.0, -7.0])
    c, nll, acc, mnll = oracle.evaluate(qco, sm, [1, 2, 0])
    assert list(c) == [0, 0, 1]
    assert acc == pytest.approx(1 / 3, abs=1e-16)
    assert mnll == pytest.approx((math.log1p(math.exp(1.0)) + math.log(3.0) + 0.0) / 3, abs=1e-14)


def test_answer_classes_by_token_sequence():
    """Equivalent labels are those with identical token sequences within one
    question (hand-computed classes; Section 3.3)."""
    seqs = [[5, 6], [7], [5, 6], [5], [7], [5, 6, 1],  # question 0
            [7], [7]]                                  # question 1: same tokens again
    qco = np.array([0, 6, 8], np.int64)
    cto = np.concatenate([[0], np.cumsum([len(x) for x in seqs])]).astype(np.int64)
    toks = np.concatenate(seqs).astype(np.int32)
    np.testing.assert_array_equal(oracle.answer_classes(qco, cto, toks), [0, 1, 0, 3, 1, 5, 0, 0])


def test_zero_weights_give_uniform_vocabulary(model_dir):
    g = json.load(open(os.path.join(GOLDEN, "zero_model_logprob.json")))["per_token"]
    for spec, wname in (("tiny_dense_fp32", "tiny"), ("micro_hybrid_fp32", "micro_hybrid")):
        p = jet_synth.ensure_model(spec, zero=True, cache_dir=model_dir)
        V = jet_synth.read_header(p)["vocab"]
        wl = jet_synth.make_workload(wname)
        tok, sums = oracle.score_unshared(p, wl)
        assert np.all(tok == g[str(V)]), (spec, np.unique(tok))
        m = np.diff(wl.cand_tok_offsets)
        np.testing.assert_allclose(sums, m * g[str(V)], rtol=1e-15, atol=0)


# --------------------------------------------------------------------------
# network blocks: closed forms and special cases
# --------------------------------------------------------------------------

def test_q8_weights_against_the_bf16_twin(model_dir):
    """Block-quantized storage: the oracle's dequantized weights of a q8 model
    lie within half a quantization step (plus bf16 rounding) of the bf16
    model drawn from the same seed, every block's scale is tight (its largest
    |q| is at least 64) and all-zero q8 weights give exactly -ln|V|."""
    pq = jet_synth.ensure_model("micro_q8", cache_dir=model_dir)
    pb = os.path.join(model_dir, "micro_q8_bf16twin.jetm")
    if not os.path.exists(pb):
        jet_synth.write_model(pb, _spec("micro_q8", dtype="bf16"))
    mq, mb = om.Model(pq), om.Model(pb)
    checked = 0
    for t in mq.h["tensors"]:
        if t["dtype"] != "q8":
            continue
        raw = jet_synth.tensor_raw(pq, t["name"], mq.h)
        wq, wb = mq.w(t["name"]), mb.w(t["name"])
        step = np.ldexp(1.0, np.repeat(np.asarray(raw.e, np.int64), 32, axis=-1))
        assert np.all(np.abs(wq - wb) <= 0.5 * step + np.abs(wb) * 2.0 ** -8), t["name"]
        qmax = np.abs(np.asarray(raw.q, np.int32)).reshape(-1, 32).max(axis=1)
        assert np.all(qmax >= 64) and np.all(qmax <= 127)
        checked += 1
    assert checked >= 5
    pz = os.path.join(model_dir, "micro_q8_zero.jetm")
    if not os.path.exists(pz):
        jet_synth.write_model(pz, _spec("micro_q8"), zero=True)
    wl = jet_synth.make_workload("micro_hybrid", vocab=512, Q=2, P=(3, 9), K=3, m=(1, 4))
    tok, sums = oracle.score_unshared(pz, wl)
    np.testing.assert_allclose(tok, -math.log(512), rtol=0, atol=1e-12)


def test_q4_packing_of_a_hand_built_block():
    """int4 storage read by hand: byte i holds value 2i in its low nibble and
    2i+1 in its high nibble, two's complement; the oracle's weight is
    q * 2^e with the block's own exponent."""
    vals = np.array([-8, 7, -1, 0, 1, -2, 3, -5] * 4, np.int8)
    want = bytes([0x78, 0x0F, 0xE1, 0xB3] * 4)
    packed, e = jet_synth.quantize_q4(vals.astype(np.float32) * np.float32(0.25))
    # max|w| = 2 = 8 * 2^-2 > 7 * 2^-2: the exponent rises to -1 and the
    # values halve (rint rounds halves to even)
    assert int(e[0]) == -1
    assert np.array_equal(jet_synth.unpack_q4(packed), np.rint(vals / 2.0).astype(np.int8))
    assert np.array_equal(jet_synth.unpack_q4(np.frombuffer(want, np.uint8)), vals)
    raw = jet_synth.Q4Raw(np.frombuffer(want, np.uint8)[None, :], np.array([[-3]], np.int8))
    assert raw.shape == (1, 32)
    np.testing.assert_array_equal(om.upcast(raw)[0], vals.astype(np.float64) / 8.0)


def test_q4_weights_against_the_bf16_twin(model_dir):
    """int4 blocks: the oracle's dequantized weights of a q4 model lie within
    half a quantization step (plus bf16 rounding) of the bf16 model drawn from
    the same seed, and every block's scale is tight (its largest |q| is 4..7)."""
    pq = jet_synth.ensure_model("micro_q4", cache_dir=model_dir)
    pb = os.path.join(model_dir, "micro_q4_bf16twin.jetm")
    if not os.path.exists(pb):
        jet_synth.write_model(pb, _spec("micro_q4", dtype="bf16"))
    mq, mb = om.Model(pq), om.Model(pb)
    checked = 0
    for t in mq.h["tensors"]:
        if t["dtype"] != "q4":
            continue
        assert t["nbytes"] == int(np.prod(t["shape"])) // 2 + int(np.prod(t["shape"])) // 32
        raw = jet_synth.tensor_raw(pq, t["name"], mq.h)
        wq, wb = mq.w(t["name"]), mb.w(t["name"])
        step = np.ldexp(1.0, np.repeat(np.asarray(raw.e, np.int64), 32, axis=-1))
        assert np.all(np.abs(wq - wb) <= 0.5 * step + np.abs(wb) * 2.0 ** -8), t["name"]
        qmax = np.abs(np.asarray(raw.q, np.int32)).reshape(-1, 32).max(axis=1)
        assert np.all(qmax >= 4) and np.all(qmax <= 7)
        checked += 1
    assert checked >= 5


def test_rope_identity_and_relative_position():
    rng = np.random.default_rng(2)
    x = rng.normal(size=(1, 3, 32))
    np.testing.assert_array_equal(om.rope(x, np.array([0]), 1e6), x)
    q = rng.normal(size=(1, 1, 32)); k = rng.normal(size=(1, 1, 32))
    for th in (1e4, 1e6):
        d1 = np.sum(om.rope(q, np.array([7]), th) * om.rope(k, np.array([3]), th))
        d2 = np.sum(om.rope(q, np.array([4007]), th) * om.rope(k, np.array([4003]), th))
        assert abs(d1 - d2) < 1e-9
        # norms are preserved
        assert abs(np.linalg.norm(om.rope(q, np.array([123]), th)) - np.linalg.norm(q)) < 1e-12
    # the pairs are (i, i + hd/2): a vector living only in dim 0 rotates into dim 16
    e0 = np.zeros((1, 1, 32)); e0[0, 0, 0] = 1.0
    r = om.rope(e0, np.array([1]), 1e6)
    assert abs(r[0, 0, 0] - math.cos(1.0)) < 1e-15 and abs(r[0, 0, 16] - math.sin(1.0)) < 1e-15


def test_attention_special_cases():
    rng = np.random.default_rng(3)
    # a single visible key returns its value exactly
    q = rng.normal(size=(1, 4, 16)); k = rng.normal(size=(1, 2, 16)); v = rng.normal(size=(1, 2, 16))
    out = om.attention(q, k, v, np.array([0]), np.array([0]))
    for h in range(4):
        np.testing.assert_allclose(out[0, h], v[0, h // 2], atol=1e-15)
    # zero queries: uniform weights over the visible keys (causal prefix mean)
    n = 5
    q = np.zeros((n, 4, 16)); k = rng.normal(size=(n, 2, 16)); v = rng.normal(size=(n, 2, 16))
    out = om.attention(q, k, v, np.arange(n), np.arange(n))
    for i in range(n):
        for h in range(4):
            np.testing.assert_allclose(out[i, h], v[:i + 1, h // 2].mean(axis=0), atol=1e-14)


def test_gated_delta_rule_closed_forms():
    rng = np.random.default_rng(4)
    H, dk, dv, n = 2, 8, 6, 5
    S0 = rng.normal(size=(H, dv, dk))
    q = rng.normal(size=(n, H, dk)); k = rng.normal(size=(n, H, dk)); v = rng.normal(size=(n, H, dv))
    # alpha = 1, beta = 0: state unchanged, output is S0 q
    o, S = om.gdn_recurrence(q, k, v, np.ones((n, H)), np.zeros((n, H)), S0)
    np.testing.assert_allclose(S, S0, atol=0)
    np.testing.assert_allclose(o, np.einsum("hvk,nhk->nhv", S0, q), atol=1e-13)
    # alpha = 1, beta = 1, unit keys: the state maps k_t to v_t exactly afterwards
    ku = k / np.linalg.norm(k, axis=-1, keepdims=True)
    S = S0
    for t in range(n):
        _, S = om.gdn_recurrence(q[t:t + 1], ku[t:t + 1], v[t:t + 1], np.ones((1, H)), np.ones((1, H)), S)
        np.testing.assert_allclose(np.einsum("hvk,hk->hv", S, ku[t]), v[t], atol=1e-12)
    # alpha = 0 forgets everything before the step
    o0, _ = om.gdn_recurrence(q[:1], k[:1], v[:1], np.zeros((1, H)), np.full((1, H), 0.7), S0)
    o1, _ = om.gdn_recurrence(q[:1], k[:1], v[:1], np.zeros((1, H)), np.full((1, H), 0.7), np.zeros_like(S0))
    np.testing.assert_allclose(o0, o1, atol=1e-15)


def test_causal_conv_matches_direct_sum():
    rng = np.random.default_rng(5)
    x = rng.normal(size=(7, 3)); w = rng.normal(size=(3, 4))
    out, tail = om.causal_conv(x, np.zeros((3, 3)), w)
    for t in range(7):
        ref = sum(w[:, j] * (x[t - 3 + j] if t - 3 + j >= 0 else 0.0) for j in range(4))
        np.testing.assert_allclose(out[t], ref, atol=1e-14)
    np.testing.assert_array_equal(tail, x[-3:])
    # splitting the sequence and carrying the tail gives the same output
    o1, t1 = om.causal_conv(x[:2], np.zeros((3, 3)), w)
    o2, _ = om.causal_conv(x[2:], t1, w)
    np.testing.assert_allclose(np.concatenate([o1, o2]), out, atol=1e-15)


# --------------------------------------------------------------------------
# independent library implementations of the same blocks
# --------------------------------------------------------------------------

def _hf_qwen2(path):
    import torch
    from transformers import Qwen2Config, Qwen2ForCausalLM
    m = oracle.Model(path)
    h = m.h
    cfg = Qwen2Config(vocab_size=h["vocab"], hidden_size=h["d_model"], intermediate_size=h["ffn"],
                      num_hidden_layers=h["n_layers"], num_attention_heads=h["n_heads"],
                      num_key_value_heads=h["n_kv_heads"], head_dim=h["head_dim"],
                      rms_norm_eps=h["rms_eps"], rope_theta=h["rope_theta"],
                      max_position_embeddings=4096, tie_word_embeddings=False,
                      attn_implementation="eager")
    net = Qwen2ForCausalLM(cfg).double().eval()
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a))
    with torch.no_grad():
        net.model.embed_tokens.weight.copy_(T(m.w("tok_embed")))
        for i, layer in enumerate(net.model.layers):
            W = m.layer(i)
            layer.input_layernorm.weight.copy_(T(W["attn_norm"]))
            layer.post_attention_layernorm.weight.copy_(T(W["ffn_norm"]))
            at = layer.self_attn
            at.q_proj.weight.copy_(T(W["wq"])); at.q_proj.bias.zero_()
            at.k_proj.weight.copy_(T(W["wk"])); at.k_proj.bias.zero_()
            at.v_proj.weight.copy_(T(W["wv"])); at.v_proj.bias.zero_()
            at.o_proj.weight.copy_(T(W["wo"]))
            layer.mlp.gate_proj.weight.copy_(T(W["w_gate"]))
            layer.mlp.up_proj.weight.copy_(T(W["w_up"]))
            layer.mlp.down_proj.weight.copy_(T(W["w_down"]))
        net.model.norm.weight.copy_(T(m.w("final_norm")))
        net.lm_head.weight.copy_(T(m.w("lm_head")))
    return net


def test_dense_scores_match_transformers_qwen2(pin_dense_path):
    """End-to-end: logits of an independent decoder implementation on the same
    weights give the same per-token log-probabilities (covers the projection
    orientation, RoPE pairing, GQA head mapping, causal mask, SwiGLU order and
    the one-position shift between a token and the row that predicts it)."""
    import torch
    net = _hf_qwen2(pin_dense_path)
    V = jet_synth.read_header(pin_dense_path)["vocab"]
    wl = jet_synth.make_workload("tiny", n_questions=3, vocab=V, P=(9, 30), m=(1, 6))
    tok, sums = oracle.score_unshared(pin_dense_path, wl)
    ref = np.zeros_like(tok)
    for q in range(wl.n_questions):
        x = wl.prefix(q)
        for j, y in enumerate(wl.candidates(q)):
            c = wl.q_cand_offsets[q] + j
            seq = np.concatenate([x, y]).astype(np.int64)
            with torch.no_grad():
                logits = net(torch.from_numpy(seq)[None]).logits[0].numpy()
            lp = logits - scipy.special.logsumexp(logits, axis=1, keepdims=True)
            P = len(x)
            ref[wl.cand_tok_offsets[c]:wl.cand_tok_offsets[c + 1]] = [lp[P - 1 + t, y[t]] for t in range(len(y))]
    # transformers normalises in float32 internally, so agreement is ~1e-6
    np.testing.assert_allclose(tok, ref, atol=2e-5, rtol=0)
    assert np.std(tok) > 0.05  # the pin model is far from uniform


def test_dense_pin_detects_planted_mistakes(pin_dense_path, monkeypatch):
    """The transformers pin is sensitive: a wrong RoPE pairing or a wrong GQA
    head mapping planted in the oracle moves the scores well past the pin's
    tolerance."""
    V = jet_synth.read_header(pin_dense_path)["vocab"]
    wl = jet_synth.make_workload("tiny", n_questions=2, vocab=V, P=(9, 30), m=(1, 6))
    good, _ = oracle.score_unshared(pin_dense_path, wl)

    def rope_interleaved(x, pos, theta):
        hd = x.shape[-1]
        c, s = om.rope_angles(pos, hd, theta)
        c, s = c[:, None, :], s[:, None, :]
        x1, x2 = x[..., 0::2], x[..., 1::2]
        out = np.empty_like(x)
        out[..., 0::2] = x1 * c - x2 * s
        out[..., 1::2] = x2 * c + x1 * s
        return out

    monkeypatch.setattr(om, "rope", rope_interleaved)
    bad, _ = oracle.score_unshared(pin_dense_path, wl)
    assert np.max(np.abs(bad - good)) > 1e-3
    monkeypatch.undo()

    real_attention = om.attention

    def attention_wrong_group(q, k, v, qp, kp):
        return real_attention(q, k[:, ::-1], v[:, ::-1], qp, kp)

    monkeypatch.setattr(om, "attention", attention_wrong_group)
    bad, _ = oracle.score_unshared(pin_dense_path, wl)
    assert np.max(np.abs(bad - good)) > 1e-3


def _hf_gdn(m, layer):
    import torch
    from transformers.models.qwen3_next.configuration_qwen3_next import Qwen3NextConfig
    from transformers.models.qwen3_next.modeling_qwen3_next import Qwen3NextGatedDeltaNet
    h = m.h
    H, dk, dv = h["gdn_heads"], h["gdn_dk"], h["gdn_dv"]
    cfg = Qwen3NextConfig(hidden_size=h["d_model"], linear_num_value_heads=H, linear_num_key_heads=H,
                          linear_key_head_dim=dk, linear_value_head_dim=dv,
                          linear_conv_kernel_dim=h["conv_kernel"], hidden_act="silu",
                          rms_norm_eps=h["rms_eps"], num_hidden_layers=4,
                          layer_types=["linear_attention"] * 4)
    net = Qwen3NextGatedDeltaNet(cfg, layer).double().eval()
    W = m.layer(layer)
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a))
    qkvz = []
    for hh in range(H):
        qkvz += [W["gdn_wq"][hh * dk:(hh + 1) * dk], W["gdn_wk"][hh * dk:(hh + 1) * dk],
                 W["gdn_wv"][hh * dv:(hh + 1) * dv], W["gdn_wz"][hh * dv:(hh + 1) * dv]]
    ba = []
    for hh in range(H):
        ba += [W["gdn_wb"][hh:hh + 1], W["gdn_wa"][hh:hh + 1]]
    with torch.no_grad():
        net.in_proj_qkvz.weight.copy_(T(np.concatenate(qkvz)))
        net.in_proj_ba.weight.copy_(T(np.concatenate(ba)))
        net.conv1d.weight.copy_(T(W["gdn_conv"][:, None, :]))
        net.A_log.copy_(T(W["gdn_A_log"]))
        net.dt_bias.copy_(T(W["gdn_dt_bias"]))
        net.norm.weight.copy_(T(W["gdn_norm"]))
        net.out_proj.weight.copy_(T(W["gdn_wo"]))
    return net, W


def test_gdn_layer_matches_transformers_qwen3next(pin_hybrid_path):
    """The gated delta-rule layer (projections, causal conv + SiLU, l2 norms,
    beta / decay gates, recurrence, gated output norm, output projection)
    against transformers' Qwen3-Next implementation (its chunked form)."""
    import torch
    m = oracle.Model(pin_hybrid_path)
    rng = np.random.default_rng(6)
    n = 23
    a = rng.normal(size=(n, m.d))
    for layer in (0, 2):
        net, W = _hf_gdn(m, layer)
        with torch.no_grad():
            ref = net(torch.from_numpy(a)[None]).numpy()[0]
        got, _ = om._gdn_layer(m.h, W, a, [slice(0, n)], [None], layer, False, m.eps)
        # transformers runs the recurrence in float32
        np.testing.assert_allclose(got, ref, atol=2e-5 * np.abs(ref).max(), rtol=0)
        assert np.abs(ref).max() > 1e-2


def test_gdn_recurrence_matches_transformers_recurrent_form():
    import torch
    from transformers.models.qwen3_next.modeling_qwen3_next import torch_recurrent_gated_delta_rule
    rng = np.random.default_rng(7)
    n, H, dk, dv = 9, 3, 8, 5
    q = rng.normal(size=(n, H, dk)); k = rng.normal(size=(n, H, dk)); v = rng.normal(size=(n, H, dv))
    g = -np.abs(rng.normal(size=(n, H))); beta = 1 / (1 + np.exp(-rng.normal(size=(n, H))))
    S0 = rng.normal(size=(H, dv, dk))
    qn = om.l2norm(q); kn = om.l2norm(k)
    o, S = om.gdn_recurrence(qn / np.sqrt(dk), kn, v, np.exp(g), beta, S0)
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a))[None]
    ref_o, ref_S = torch_recurrent_gated_delta_rule(T(q), T(k), T(v), T(g), T(beta),
                                                    initial_state=T(np.transpose(S0, (0, 2, 1)))[0][None],
                                                    output_final_state=True, use_qk_l2norm_in_kernel=True)
    np.testing.assert_allclose(o, ref_o[0].double().numpy(), atol=1e-5)
    # transformers keeps the state as [dk, dv]
    np.testing.assert_allclose(S, np.transpose(ref_S[0].double().numpy(), (0, 2, 1)), atol=1e-5)


# --------------------------------------------------------------------------
# invariants of the scoring method (Section 4.1, Section 5.6)
# --------------------------------------------------------------------------

def _hf_moe_block(m, li):
    """transformers' Qwen2-MoE sparse block (router, experts, gated shared
    expert) in float64 holding block li's weights of the oracle's model."""
    import torch
    from transformers.models.qwen2_moe.configuration_qwen2_moe import Qwen2MoeConfig
    from transformers.models.qwen2_moe.modeling_qwen2_moe import Qwen2MoeSparseMoeBlock
    h = m.h
    cfg = Qwen2MoeConfig(hidden_size=h["d_model"], num_experts=h["n_experts"],
                         num_experts_per_tok=h["top_k"], norm_topk_prob=True,
                         moe_intermediate_size=h["moe_ffn"], shared_expert_intermediate_size=h["shared_ffn"],
                         hidden_act="silu")
    blk = Qwen2MoeSparseMoeBlock(cfg).double()
    W = m.layer(li)
    T = lambda x: torch.from_numpy(np.ascontiguousarray(x))
    with torch.no_grad():
        blk.gate.weight.copy_(T(W["moe_router"]))
        for e in range(h["n_experts"]):
            blk.experts.gate_up_proj[e].copy_(T(np.concatenate([m.expert(li, "moe_gate", e),
                                                                m.expert(li, "moe_up", e)])))
            blk.experts.down_proj[e].copy_(T(m.expert(li, "moe_down", e)))
        blk.shared_expert.gate_proj.weight.copy_(T(W["shared_gate"]))
        blk.shared_expert.up_proj.weight.copy_(T(W["shared_up"]))
        blk.shared_expert.down_proj.weight.copy_(T(W["shared_down"]))
        blk.shared_expert_gate.weight.copy_(T(W["shared_router"]))
    return blk, W


def test_moe_block_matches_transformers_qwen2moe(pin_moe_path):
    """The oracle's mixture-of-experts FFN against transformers' Qwen2-MoE
    sparse block on the same weights and inputs (its router softmax runs in
    float32, hence the tolerance)."""
    import torch
    m = om.Model(pin_moe_path)
    a = np.random.default_rng(5).normal(size=(40, m.d))
    for li in range(len(m.layer_types)):
        blk, W = _hf_moe_block(m, li)
        with torch.no_grad():
            ref = blk(torch.from_numpy(a)[None])
        ref = (ref[0] if isinstance(ref, tuple) else ref)[0].numpy()
        got = om.moe_ffn(m, li, W, a)
        assert np.abs(ref).max() > 1e-2
        np.testing.assert_allclose(got, ref, rtol=0, atol=2e-6 * np.abs(ref).max())


def test_moe_routing_special_cases(pin_moe_path):
    """Equal router logits keep the lowest-index experts with equal weights;
    keeping every expert gives the full softmax mixture; no shared expert
    and one expert reduce to the dense SwiGLU FFN."""
    m = om.Model(pin_moe_path)
    W = dict(m.layer(0))
    a = np.random.default_rng(6).normal(size=(7, m.d))
    ffn = [om.swiglu_ffn(a, m.expert(0, "moe_gate", e), m.expert(0, "moe_up", e), m.expert(0, "moe_down", e))
           for e in range(m.n_experts)]
    g = 1.0 / (1.0 + np.exp(-(a @ W["shared_router"].T)))
    shared = g * om.swiglu_ffn(a, W["shared_gate"], W["shared_up"], W["shared_down"])
    W0 = dict(W, moe_router=np.zeros_like(W["moe_router"]))
    k = m.top_k
    np.testing.assert_allclose(om.moe_ffn(m, 0, W0, a), sum(ffn[:k]) / k + shared, rtol=0, atol=1e-12)
    sel, w = om.moe_route(np.array([[0.5, 2.0, 2.0, -1.0]]), 2)
    assert list(sel[0]) == [1, 2] and np.allclose(w, 0.5)
    m_all = om.Model(pin_moe_path)
    m_all.top_k = m.n_experts
    z = a @ W["moe_router"].T
    p = np.exp(z - z.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    np.testing.assert_allclose(om.moe_ffn(m_all, 0, W, a), sum(p[:, [e]] * ffn[e] for e in range(m.n_experts)) + shared,
                               rtol=0, atol=1e-12)
    m_one = om.Model(pin_moe_path)
    m_one.top_k = 1
    Wn = {k_: v for k_, v in W.items() if not k_.startswith("shared_")}
    best = np.argmax(z, axis=1)
    np.testing.assert_allclose(om.moe_ffn(m_one, 0, Wn, a), np.stack([ffn[best[i]][i] for i in range(len(a))]),
                               rtol=0, atol=1e-12)


def test_moe_forced_routing_pins(pin_moe_path):
    """Forced routing (checking a routing decided elsewhere) against the
    unforced rule: forcing the rule's own choice changes nothing, -1 rows are
    routed by the rule, a forced set S equals the unforced mixture of a model
    that holds only the experts S (all kept), the order inside S does not
    matter, and the reported gap is the logit margin of the set."""
    m = om.Model(pin_moe_path)
    W = dict(m.layer(0))
    k, E = m.top_k, m.n_experts
    a = np.random.default_rng(11).normal(size=(9, m.d))
    z = a @ W["moe_router"].T
    own, _ = om.moe_route(z, k)
    base = om.moe_ffn(m, 0, W, a)
    gaps = []
    np.testing.assert_array_equal(om.moe_ffn(m, 0, W, a, own, gaps), base)
    srt = np.sort(z, axis=1)[:, ::-1]
    np.testing.assert_allclose(gaps[0], srt[:, k - 1] - srt[:, k], rtol=0, atol=1e-14)
    assert np.all(gaps[0] >= 0)
    np.testing.assert_array_equal(om.moe_ffn(m, 0, W, a, np.full((len(a), k), -1)), base)
    # one forced set for every row, against a model holding only those experts
    S = np.array([E - 1, 0][:k] + list(range(1, k - 1)))
    sub = om.Model(pin_moe_path)
    sub.n_experts = sub.top_k = k
    sub.expert = lambda li, name, e: m.expert(li, name, int(S[e]))
    Wsub = dict(W, moe_router=W["moe_router"][S])
    ref = om.moe_ffn(sub, 0, Wsub, a)
    forced = np.tile(S, (len(a), 1))
    g2 = []
    np.testing.assert_allclose(om.moe_ffn(m, 0, W, a, forced, g2), ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(om.moe_ffn(m, 0, W, a, forced[:, ::-1].copy()), ref, rtol=0, atol=1e-12)
    out = np.ones((len(a), E), bool)
    out[:, S] = False
    np.testing.assert_allclose(g2[0], z[:, S].min(axis=1) - np.where(out, z, -np.inf).max(axis=1), atol=1e-14)
    # the k-th expert swapped for the (k+1)-th: gap is minus the k-th margin
    order = np.argsort(-z, axis=1, kind="stable")
    swap = order[:, :k].copy()
    swap[:, k - 1] = order[:, k]
    g3 = []
    om.moe_ffn(m, 0, W, a, swap, g3)
    np.testing.assert_allclose(g3[0], -(srt[:, k - 1] - srt[:, k]), rtol=0, atol=1e-14)


def test_moe_forced_routes_follow_their_sequence(pin_moe_path):
    """forward(routes=...) aligns each sequence's forced rows with that
    sequence: two sequences stacked, one forced and one left to the rule,
    each equal to its own forward alone."""
    m = om.Model(pin_moe_path)
    rng = np.random.default_rng(12)
    V, L, k = m.V, len(m.layer_types), m.top_k
    s0 = rng.integers(0, V, 11)
    s1 = rng.integers(0, V, 7)
    r0 = np.stack([np.stack([rng.permutation(m.n_experts)[:k] for _ in range(len(s0))]) for _ in range(L)])
    r1 = np.full((L, len(s1), k), -1)
    both, _ = om.forward(m, [s0, s1], routes=[r0, r1])
    alone0, _ = om.forward(m, [s0], routes=[r0])
    alone1, _ = om.forward(m, [s1])
    np.testing.assert_allclose(both[0], alone0[0], rtol=0, atol=1e-12)
    np.testing.assert_allclose(both[1], alone1[0], rtol=0, atol=1e-12)
    plain0, _ = om.forward(m, [s0])
    assert np.abs(plain0[0] - alone0[0]).max() > 1e-6   # the forced experts did change sequence 0


@pytest.mark.parametrize("which", ["dense", "hybrid", "moe"])
def test_prefix_sharing_equals_unshared(which, pin_dense_path, pin_hybrid_path, pin_moe_path):
    path = {"dense": pin_dense_path, "hybrid": pin_hybrid_path, "moe": pin_moe_path}[which]
    V = jet_synth.read_header(path)["vocab"]
    wl = jet_synth.make_workload("micro_hybrid", vocab=V, Q=3, P=(4, 17), K=4, m=(1, 6))
    a, sa = oracle.score_unshared(path, wl)
    b, sb = oracle.score_incremental(path, wl)
    np.testing.assert_allclose(a, b, atol=1e-10, rtol=0)
    np.testing.assert_allclose(sa, sb, atol=1e-10, rtol=0)


@pytest.mark.parametrize("which", ["dense", "hybrid", "moe"])
def test_isolation_and_planted_leak(which, pin_dense_path, pin_hybrid_path, pin_moe_path):
    """Scoring a candidate after its siblings equals scoring it alone; the
    planted leak (state not restored between candidates) is detected."""
    path = {"dense": pin_dense_path, "hybrid": pin_hybrid_path, "moe": pin_moe_path}[which]
    V = jet_synth.read_header(path)["vocab"]
    wl = jet_synth.make_workload("micro_hybrid", vocab=V, Q=2, P=(6, 12), K=4, m=(2, 6))
    full, _ = oracle.score_incremental(path, wl)
    for q in range(wl.n_questions):
        x = wl.prefix(q)
        for j, y in enumerate(wl.candidates(q)):
            alone = jet_synth.from_lists([x], [[y]])
            t, _ = oracle.score_incremental(path, alone)
            c = wl.q_cand_offsets[q] + j
            np.testing.assert_array_equal(t, full[wl.cand_tok_offsets[c]:wl.cand_tok_offsets[c + 1]])
    leaky, _ = oracle.score_incremental(path, wl, leak=True)
    assert np.max(np.abs(leaky - full)) > 1e-3


def test_candidate_permutation_invariance(pin_dense_path):
    V = jet_synth.read_header(pin_dense_path)["vocab"]
    wl = jet_synth.make_workload("tiny", n_questions=3, vocab=V, P=(5, 20), m=(1, 5))
    _, s = oracle.score_unshared(pin_dense_path, wl)
    rng = np.random.default_rng(8)
    pre, cands, perm_all = [], [], []
    for q in range(wl.n_questions):
        cs = wl.candidates(q)
        perm = rng.permutation(len(cs))
        pre.append(wl.prefix(q)); cands.append([cs[i] for i in perm])
        perm_all += [wl.q_cand_offsets[q] + i for i in perm]
    _, s2 = oracle.score_unshared(pin_dense_path, jet_synth.from_lists(pre, cands))
    np.testing.assert_allclose(s2, s[perm_all], atol=1e-12, rtol=0)


def test_duplicates_and_causality(pin_dense_path):
    """Equal answer text gives equal likelihood (Section 3.3), and a token's
    log-probability depends only on the tokens before it (Eq. 3 chain rule)."""
    V = jet_synth.read_header(pin_dense_path)["vocab"]
    x = np.array([5, 9, 2, 77, 31, 8], np.int32)
    y = np.array([10, 20, 30, 40], np.int32)
    y2 = y.copy(); y2[-1] = 41
    wl = jet_synth.from_lists([x], [[y, y.copy(), y2, y[:2]]])
    tok, s = oracle.score_unshared(pin_dense_path, wl)
    assert abs(s[0] - s[1]) < 1e-12
    assert oracle.decide_choice(np.array([s[0], s[1]])) == 0
    np.testing.assert_allclose(tok[8:11], tok[0:3], atol=1e-12)   # y2 shares its first 3 tokens
    assert abs(tok[11] - tok[3]) > 1e-6
    np.testing.assert_allclose(tok[12:14], tok[0:2], atol=1e-12)  # the 2-token prefix of y


# --------------------------------------------------------------------------
# Section 3.4: reasoning traces (Gumbel-max sampling, the reading used here)
# --------------------------------------------------------------------------

from oracle import generate as og  # noqa: E402


def test_splitmix64_reference_outputs():
    """The first outputs of SplitMix64 seeded with 0 are the generator's
    published reference values."""
    got = [int(x) for x in og.splitmix64_at(0, np.arange(3))]
    assert got == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_counter_uniforms_are_uniform_and_keyed():
    u = og.uniform_at(7, 3, 2, np.arange(200_000))
    assert 0.0 < u.min() and u.max() < 1.0
    assert abs(u.mean() - 0.5) < 4 * math.sqrt(1 / 12 / len(u))
    assert abs(u.var() - 1 / 12) < 2e-3
    # every coordinate of the counter changes the draw
    base = og.uniform_at(7, 3, 2, 5)
    for other in (og.uniform_at(8, 3, 2, 5), og.uniform_at(7, 4, 2, 5), og.uniform_at(7, 3, 3, 5),
                  og.uniform_at(7, 3, 2, 6)):
        assert other != base


def test_gumbel_max_draws_from_tempered_softmax():
    """argmax(z / tau + G) over fresh counters has the frequencies of
    softmax(z / tau) (the Gumbel-max property), within 5 standard errors."""
    z = np.array([0.3, 1.2, -0.5, 0.9, 0.0])
    tau, n = 0.7, 40_000
    counts = np.zeros(len(z))
    for t in range(n):
        counts[og.first_argmax(og.sample_keys(z, tau, 99, 1, t))] += 1
    p = scipy.special.softmax(z / tau)
    se = np.sqrt(p * (1 - p) / n)
    assert np.all(np.abs(counts / n - p) < 5 * se), (counts / n, p)


def test_greedy_keys_and_ties():
    z = np.array([1.0, 3.0, 3.0, -2.0])
    np.testing.assert_array_equal(og.sample_keys(z, 0.0, 5, 0, 0), z)
    assert og.first_argmax(og.sample_keys(z, 0.0, 5, 0, 0)) == 1      # lowest index among equal maxima


def test_greedy_trace_is_the_scorer_argmax(pin_hybrid_path):
    """Each greedy trace token is the most likely next token by the pinned
    scorer: scoring every vocabulary entry as a one-token candidate after the
    trace so far (Eq. 2) puts its maximum on the generated token."""
    model = oracle.Model(pin_hybrid_path)
    V = model.h["vocab"]
    x = np.array([3, 17, 250, 9, 400, 44], np.int32)
    toks, steps = og.generate_trace(model, x, 0, 3, 0.0, 1)
    seq = list(x)
    for t in range(3):
        wl = jet_synth.from_lists([np.asarray(seq, np.int32)], [[np.array([v], np.int32) for v in range(V)]])
        _, s = oracle.score_unshared(model, wl)
        assert int(np.argmax(s)) == int(toks[t])
        assert steps[t]["choice"] == int(toks[t]) and steps[t]["key"] == steps[t]["max_key"]
        seq.append(int(toks[t]))


def test_forced_trace_reports_the_gap(pin_dense_path):
    model = oracle.Model(pin_dense_path)
    x = np.array([5, 9, 2, 77], np.int32)
    toks, _ = og.generate_trace(model, x, 2, 4, 0.9, 7)
    again, st = og.generate_trace(model, x, 2, 4, 0.9, 7, forced=toks)
    np.testing.assert_array_equal(again, toks)
    assert all(s["key"] == s["max_key"] for s in st)
    other = toks.copy()
    other[1] = (toks[1] + 1) % model.h["vocab"]
    _, st2 = og.generate_trace(model, x, 2, 4, 0.9, 7, forced=other)
    assert st2[1]["key"] < st2[1]["max_key"]
