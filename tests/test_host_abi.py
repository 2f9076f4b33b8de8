"""C ABI checks that need no GPU: exports, decisions (Eq. 4-5), the integer
row layout (bit-exact) and request validation."""
import json
import math
import os
import re

import numpy as np
import pytest

import jet_synth
import oracle
from paper_2609_33874_amd import jet as J

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_symbol():
    hdr = open(os.path.join(ROOT, "include", "jet.h")).read()
    declared = set(re.findall(r"^(?:int|void|const char \*)\s*(jet_[a-z_]+)\s*\(", hdr, re.M))
    assert declared == set(J.EXPORTS)
    L = J.lib()
    for name in declared:
        assert hasattr(L, name), name


def test_decide_worked_example():
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "worked_example.json")))
    s = np.log(np.array(g["likelihoods"], np.float32))
    q, choice, _ = J.jet_decide(J.JET_CHOICE, [0, 2], s)
    # float32 inputs: ln 0.06 and ln 0.02 are rounded once to float32
    np.testing.assert_allclose(q, g["normalized"], atol=1e-7)
    assert choice[0] == 0


def test_decide_matches_oracle_rules():
    rng = np.random.default_rng(0)
    qco = np.array([0, 2, 4, 9, 12], np.int64)
    s = rng.normal(-10, 3, size=12).astype(np.float32)
    s[10] = s[11] = s[9] + 1.0  # tie in the last question: lowest index wins
    q, ch, _ = J.jet_decide(J.JET_CHOICE, qco, s)
    oq, och, _ = oracle.decide("choice", qco, s.astype(np.float64))
    np.testing.assert_allclose(q, oq, rtol=0, atol=1e-15)
    np.testing.assert_array_equal(ch, och)
    assert ch[3] == 1
    qb = np.array([0, 2, 4], np.int64)
    _, _, v = J.jet_decide(J.JET_BINARY, qb, s[:4])
    for i in range(2):
        a, b = float(s[2 * i]), float(s[2 * i + 1])
        assert v[i] == pytest.approx(1 / (1 + math.exp(a - b)), abs=1e-15)
    qo = np.array([0, 5, 12], np.int64)
    _, _, v = J.jet_decide(J.JET_ORDINAL, qo, s)
    for i in range(2):
        assert v[i] == pytest.approx(oracle.decide_ordinal(s[qo[i]:qo[i + 1]].astype(np.float64)), abs=1e-13)


def test_decide_ordinal_hand_values():
    """jet_decide's ordinal rule against hand values (Section 3.3: zero-based
    levels in supplied order), independent of the oracle."""
    # K equal scores: (K - 1) / 2 ; one level 60 nats ahead: its index
    cases = [(np.full(5, -3.5), 2.0), (np.full(10, 0.0), 4.5), (np.full(2, -1.0), 0.5)]
    for K, j in ((5, 0), (5, 3), (7, 6)):
        s = np.full(K, -80.0)
        s[j] = -20.0
        cases.append((s, float(j)))
    # q = (1/2, 1/3, 1/6) -> 2/3 ; the worked example as two levels -> 0.25
    cases.append((np.log([3.0, 2.0, 1.0]), 2.0 / 3.0))
    cases.append((np.log([0.06, 0.02]), 0.25))
    qo = np.concatenate([[0], np.cumsum([len(c[0]) for c in cases])]).astype(np.int64)
    s = np.concatenate([c[0] for c in cases]).astype(np.float32)
    _, _, v = J.jet_decide(J.JET_ORDINAL, qo, s)
    # float32 inputs move q by ~1e-7 relative
    np.testing.assert_allclose(v, [c[1] for c in cases], rtol=0, atol=1e-6)
    # two levels: exactly the binary probability of the second
    _, _, vb = J.jet_decide(J.JET_BINARY, np.array([0, 2, 4], np.int64), np.concatenate([[-3.2, -1.5], [0.0, -9.0]]).astype(np.float32))
    _, _, vo = J.jet_decide(J.JET_ORDINAL, np.array([0, 2, 4], np.int64),
                            np.concatenate([[-3.2, -1.5], [0.0, -9.0]]).astype(np.float32))
    np.testing.assert_allclose(vo, vb, rtol=0, atol=1e-15)


def test_decide_rejects_bad_requests():
    with pytest.raises(J.JetError) as e:
        J.jet_decide(J.JET_BINARY, [0, 3], np.zeros(3, np.float32))
    assert e.value.code == J.JET_E_INVALID
    with pytest.raises(J.JetError):
        J.jet_decide(J.JET_ORDINAL, [0, 1], np.zeros(1, np.float32))
    with pytest.raises(J.JetError):
        J.jet_decide(J.JET_CHOICE, [0, 2, 1], np.zeros(2, np.float32))
    with pytest.raises(J.JetError):
        J.jet_decide(J.JET_CHOICE, [0, 0], np.zeros(0, np.float32))
    with pytest.raises(J.JetError):
        J.jet_decide(J.JET_CHOICE, [0, 2], np.array([0.0, np.nan], np.float32))
    with pytest.raises(J.JetError):
        J.jet_decide(7, [0, 2], np.zeros(2, np.float32))


def _eval_case(seed, n_q=200, kmax=8):
    """Seeded questions with 1..kmax candidates of 1..3 tokens from a small
    alphabet (so labels with identical text occur), scores with ties."""
    rng = np.random.default_rng(seed)
    ks = rng.integers(1, kmax + 1, size=n_q)
    qco = np.concatenate([[0], np.cumsum(ks)]).astype(np.int64)
    N = int(qco[-1])
    lens = rng.integers(1, 4, size=N)
    cto = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    toks = rng.integers(0, 3, size=int(cto[-1])).astype(np.int32)
    sums = rng.normal(-12.0, 4.0, size=N).astype(np.float32)
    tie = rng.random(N) < 0.15
    sums[1:][tie[1:]] = sums[:-1][tie[1:]]
    gold = np.array([rng.integers(0, k) for k in ks], np.int32)
    return qco, cto, toks, sums, gold


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_evaluate_matches_oracle(seed):
    qco, cto, toks, sums, gold = _eval_case(seed)
    cls = J.jet_answer_classes(qco, cto, toks)
    np.testing.assert_array_equal(cls, oracle.answer_classes(qco, cto, toks))
    assert (cls != np.arange(len(cls)) - np.repeat(qco[:-1], np.diff(qco))).any()  # duplicates present
    for cc in (cls, None):
        c, nll, acc, mnll = J.jet_evaluate(qco, sums, gold, cc)
        oc, onll, oacc, omnll = oracle.evaluate(qco, sums.astype(np.float64), gold, cc)
        np.testing.assert_array_equal(c, oc)
        np.testing.assert_allclose(nll, onll, rtol=1e-12, atol=1e-13)
        assert acc == oacc and mnll == pytest.approx(omnll, rel=1e-12, abs=1e-13)
        # the prediction is jet_decide's choice
        _, ch, _ = J.jet_decide(J.JET_CHOICE, qco, sums)
        ref = cc if cc is not None else np.arange(len(sums)) - np.repeat(qco[:-1], np.diff(qco))
        np.testing.assert_array_equal(c, ref[qco[:-1] + ch] == ref[qco[:-1] + gold])


def test_evaluate_edge_cases():
    # the gold class far below the rest: NLL stays finite (log form)
    c, nll, acc, mnll = J.jet_evaluate([0, 2], np.array([0.0, -1000.0], np.float32), [1])
    assert c[0] == 0 and nll[0] == pytest.approx(1000.0, abs=1e-9)
    # every label with the gold text: NLL exactly 0 and correct
    c, nll, _, _ = J.jet_evaluate([0, 3], np.array([-1.0, -5.0, -2.0], np.float32), [1], [0, 0, 0])
    assert c[0] == 1 and nll[0] == 0.0
    # one candidate
    c, nll, acc, mnll = J.jet_evaluate([0, 1], np.array([-3.0], np.float32), [0])
    assert (c[0], nll[0], acc, mnll) == (1, 0.0, 1.0, 0.0)
    # binary: correct iff q(true) > 1/2, ties to false
    s = np.array([-2.0, -2.0, -3.0, -1.0], np.float32)
    c, _, _, _ = J.jet_evaluate([0, 2, 4], s, [1, 1])
    _, _, v = J.jet_decide(J.JET_BINARY, [0, 2, 4], s)
    np.testing.assert_array_equal(c, (v > 0.5).astype(np.int32))


def test_evaluate_rejects_bad_requests():
    z = np.zeros(3, np.float32)
    for args in (([0, 3], z, [3]), ([0, 3], z, [-1]), ([0, 3, 3], z, [0, 0]),
                 ([0, 3], np.array([0, np.inf, 0], np.float32), [0])):
        with pytest.raises(J.JetError) as e:
            J.jet_evaluate(*args)
        assert e.value.code == J.JET_E_INVALID
    with pytest.raises(J.JetError):
        J.jet_answer_classes([0, 2], [0, 1, 1], np.zeros(1, np.int32))  # empty candidate
    with pytest.raises(J.JetError):
        J.jet_answer_classes([0, 0], [0], np.zeros(0, np.int32))        # question without candidates


def _expected_layout(wl):
    """Definition: y_{c,t} sits at position P + t - 1 and is predicted by the
    row holding y_{c,t-1}; y_{c,1} by the last prefix position."""
    pos, qq, cc, tok, lm = [], [], [], [], np.zeros(len(wl.cand_tokens), np.int32)
    for q in range(wl.n_questions):
        P = wl.prefix_offsets[q + 1] - wl.prefix_offsets[q]
        for c in range(wl.q_cand_offsets[q], wl.q_cand_offsets[q + 1]):
            t0, t1 = wl.cand_tok_offsets[c], wl.cand_tok_offsets[c + 1]
            lm[t0] = -(q + 1)
            for t in range(1, t1 - t0):
                lm[t0 + t] = len(pos)
                pos.append(P + t - 1); qq.append(q); cc.append(c); tok.append(t0 + t - 1)
    return dict(row_pos=pos, row_q=qq, row_c=cc, row_tok=tok, lm_row=lm)


@pytest.mark.parametrize("name", ["tiny", "small", "dense_1p5b_k4", "dense_1p5b_binary", "dense_27b_k10"])
def test_candidate_layout_bit_exact(name):
    wl = jet_synth.make_workload(name, n_questions=min(40, jet_synth.WORKLOADS[name]["Q"]))
    got = J.jet_candidate_layout(wl.prefix_offsets, wl.q_cand_offsets, wl.cand_tok_offsets)
    exp = _expected_layout(wl)
    for k, v in exp.items():
        np.testing.assert_array_equal(got[k], np.asarray(v, np.int32), err_msg=k)


def test_layout_edge_cases():
    # questions without candidates, single-token candidates only, one long candidate
    wl = jet_synth.from_lists([[1, 2, 3], [4], [5, 6]], [[], [[7], [8]], [[9, 10, 11, 12]]])
    got = J.jet_candidate_layout(wl.prefix_offsets, wl.q_cand_offsets, wl.cand_tok_offsets)
    np.testing.assert_array_equal(got["row_pos"], [2, 3, 4])
    np.testing.assert_array_equal(got["lm_row"], [-2, -2, -3, 0, 1, 2])


def test_layout_validation_errors():
    po = np.array([0, 3], np.int64)
    with pytest.raises(J.JetError) as e:  # empty candidate
        J.jet_candidate_layout(po, [0, 2], [0, 2, 2])
    assert e.value.code == J.JET_E_INVALID
    with pytest.raises(J.JetError):  # empty prefix
        J.jet_candidate_layout([0, 0], [0, 1], [0, 2])
    with pytest.raises(J.JetError):  # decreasing offsets
        J.jet_candidate_layout(po, [0, 2], [0, 3, 1])
    with pytest.raises(J.JetError):  # first offset not zero
        J.jet_candidate_layout(po, [1, 2], [0, 1, 2])
    with pytest.raises(J.JetError) as e:  # P + m - 1 beyond capacity: rejected, never truncated
        J.jet_candidate_layout(po, [0, 1], [0, 5], max_ctx=6)
    assert e.value.code == J.JET_E_CAPACITY
    J.jet_candidate_layout(po, [0, 1], [0, 4], max_ctx=6)  # exactly at capacity is fine


def test_model_load_reports_io_errors(tmp_path):
    with pytest.raises(J.JetError) as e:
        J.jet_model_load(str(tmp_path / "missing.jetm"))
    assert e.value.code in (J.JET_E_IO, J.JET_E_DEVICE)
    bad = tmp_path / "bad.jetm"
    bad.write_bytes(b"NOTAMODEL" * 10)
    with pytest.raises(J.JetError) as e:
        J.jet_model_load(str(bad))
    assert e.value.code in (J.JET_E_IO, J.JET_E_DEVICE)


def test_moe_model_shapes():
    """The 35B-A3B-shape mixture-of-experts model: 33.7B parameters, 2.5B of
    them used per token (8 of 256 experts), every FFN a router, 256 experts
    and a gated shared expert; the small MoE models round-trip their header."""
    s = jet_synth.full_spec("moe_35b_a3b")
    total = jet_synth.n_params("moe_35b_a3b")
    E, k, Fe, d, L = s["n_experts"], s["top_k"], s["moe_ffn"], s["d_model"], s["n_layers"]
    active = total - L * (E - k) * 3 * Fe * d
    assert round(total / 1e9, 1) == 33.7 and round(active / 1e9, 1) == 2.5
    names = {t[0]: t[2] for t in jet_synth.tensor_list("moe_35b_a3b")}
    assert names["blk.0.moe_gate"] == (256, 512, 2048) and names["blk.0.moe_down"] == (256, 2048, 512)
    assert names["blk.39.shared_router"] == (1, 2048) and "blk.0.w_gate" not in names
    assert s["layer_types"] == ["gdn", "gdn", "gdn", "attn"] * 10


def test_model_cache_eviction(tmp_path, monkeypatch):
    """Writing a model file into a full cache deletes the largest other cached
    model files of over the size threshold until the new file fits, and no
    more; small files and the file's own path are never deleted."""
    import collections
    import shutil
    files = {"big1.jetm": 900, "big2.jetm": 700, "big3.jetm": 650, "small.jetm": 100, "other.bin": 5000}
    for name, size in files.items():
        with open(tmp_path / name, "wb") as f:
            f.truncate(size)
    need = sum(jet_synth.tensor_nbytes(dt, shape) for _, dt, shape, _ in jet_synth.tensor_list("tiny_dense_fp32"))
    Usage = collections.namedtuple("Usage", "total used free")
    base_free = need + (2 << 30) - 1500   # room once 1500 more bytes are freed

    def fake_usage(d):
        freed = sum(s for n, s in files.items() if not (tmp_path / n).exists())
        return Usage(0, 0, base_free + freed)

    monkeypatch.setattr(shutil, "disk_usage", fake_usage)
    target = tmp_path / "tiny.jetm"
    jet_synth.make_room(str(target), "tiny_dense_fp32", min_evict=500)
    left = sorted(p.name for p in tmp_path.iterdir())
    # big1 (900) and big2 (700) free 1600 >= 1500; big3, the small file and non-model files stay
    assert left == ["big3.jetm", "other.bin", "small.jetm"]
