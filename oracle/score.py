"""Scoring and decisions of the oracle (test infrastructure only).

* ``log_softmax_rows``: Eq. 2 of Section 3.1, the max-shifted log-probability
  of one supplied token over the full vocabulary (no temperature, no top-k or
  top-p).
* ``score_unshared``: Eq. 3 of Section 3.2 with every candidate run as its own
  full forward over ``x || y_c[1..m_c-1]``; the token ``y_{c,t}`` sits at
  position ``P + t - 1`` and is predicted by the hidden state one position
  earlier, so ``y_{c,1}`` is predicted by the last prefix position
  (Section 4.1).
* ``score_incremental``: the same numbers through a prefix run once whose
  retained state is copied for each candidate (Section 4.1). Self-check only;
  ``leak=True`` plants the isolation bug described in Section 5.6.
* ``normalize`` / ``decide_*``: Eq. 4 and Eq. 5 with the rules of
  Section 3.3; ties go to the lowest candidate index, binary sets are ordered
  (false, true), ordinal levels are zero-based.
* ``answer_classes`` / ``evaluate``: equivalent labels (Section 3.3: labels
  with the same answer text share one likelihood and are pooled in
  evaluation) and the accuracy / gold negative log-likelihood of the
  evaluation protocol (Section 5), straight from those definitions.
"""
from __future__ import annotations

import copy

import numpy as np

from .model import Model, forward, final_logprobs


def log_softmax_rows(z: np.ndarray, targets: np.ndarray) -> np.ndarray:
    """ell = z_y - a - log sum_v exp(z_v - a), a = max_v z_v, per row (Eq. 2)."""
    a = z.max(axis=1, keepdims=True)
    lse = np.log(np.sum(np.exp(z - a), axis=1))
    zy = z[np.arange(z.shape[0]), targets]
    return zy - a[:, 0] - lse


def _groups(wl, max_rows: int):
    """Split questions into groups of at most ~max_rows sequence rows."""
    group, rows = [], 0
    for q in range(wl.n_questions):
        P = wl.prefix_offsets[q + 1] - wl.prefix_offsets[q]
        r = sum(int(P + len(y) - 1) for y in wl.candidates(q))
        if group and rows + r > max_rows:
            yield group
            group, rows = [], 0
        group.append(q)
        rows += r
    if group:
        yield group


def score_unshared(model: Model | str, wl, max_rows: int = 16384, routes: dict | None = None,
                   route_gaps: list | None = None):
    """Per-token log-probs [sum m] (input token order) and sums [N] (Eq. 3).

    Each candidate is an independent full forward with no prefix sharing.
    Mixture-of-experts models: ``routes`` (optional) maps a candidate index
    to the experts to keep along its sequence x || y_c[1..m-1], an int array
    [n_layers, P + m - 1, top_k] (see ``forward``).
    """
    model = Model(model) if isinstance(model, str) else model
    W_lm = model.w("lm_head")
    out_tok = np.zeros(len(wl.cand_tokens))
    for group in _groups(wl, max_rows):
        seqs, meta, rts = [], [], []
        for q in group:
            x = wl.prefix(q)
            for j, y in enumerate(wl.candidates(q)):
                c = int(wl.q_cand_offsets[q]) + j
                seqs.append(np.concatenate([x, y[:-1]]).astype(np.int64))
                meta.append((c, len(x), y))
                if routes is not None:
                    rts.append(routes[c])
        hid, _ = forward(model, seqs, routes=rts if routes is not None else None, route_gaps=route_gaps)
        rows, tgts, dst = [], [], []
        for (c, P, y), hs in zip(meta, hid):
            m = len(y)
            rows.append(hs[P - 1:P - 1 + m])
            tgts.append(y)
            dst.append(np.arange(wl.cand_tok_offsets[c], wl.cand_tok_offsets[c] + m))
        ell = final_logprobs(model, np.concatenate(rows), np.concatenate(tgts), W_lm)
        out_tok[np.concatenate(dst)] = ell
    sums = candidate_sums(out_tok, wl.cand_tok_offsets)
    return out_tok, sums


def candidate_sums(tok: np.ndarray, cand_tok_offsets: np.ndarray) -> np.ndarray:
    """s_c = sum_t ell_{c,t} (Eq. 3), t ascending."""
    n = len(cand_tok_offsets) - 1
    s = np.zeros(n)
    for c in range(n):
        for i in range(cand_tok_offsets[c], cand_tok_offsets[c + 1]):
            s[c] += tok[i]
    return s


def score_incremental(model: Model | str, wl, leak: bool = False):
    """Prefix run once, its retained state copied per candidate (Section 4.1).

    With ``leak=True`` the working state is *not* restored between candidates:
    each candidate continues from the state its predecessor left behind. That
    is the planted mistake the isolation tests must detect.
    """
    model = Model(model) if isinstance(model, str) else model
    W_lm = model.w("lm_head")
    out_tok = np.zeros(len(wl.cand_tokens))
    for q in range(wl.n_questions):
        x = wl.prefix(q)
        P = len(x)
        hid, st = forward(model, [x.astype(np.int64)], want_state=True)
        last = hid[0][P - 1:P]
        prefix_state = st[0]
        working = copy.deepcopy(prefix_state)
        for j, y in enumerate(wl.candidates(q)):
            c = int(wl.q_cand_offsets[q]) + j
            if not leak:
                working = copy.deepcopy(prefix_state)
            rows = [last]
            if len(y) > 1:
                h2, st2 = forward(model, [y[:-1].astype(np.int64)], starts=[P],
                                  states=[working], want_state=True)
                rows.append(h2[0])
                working = st2[0]
            ell = final_logprobs(model, np.concatenate(rows), y, W_lm)
            out_tok[wl.cand_tok_offsets[c]:wl.cand_tok_offsets[c + 1]] = ell
    return out_tok, candidate_sums(out_tok, wl.cand_tok_offsets)


# --------------------------------------------------------------------------
# decisions (Section 3.2 Eq. 4, Section 3.3 Eq. 5)
# --------------------------------------------------------------------------

def normalize(s: np.ndarray) -> np.ndarray:
    """q(c) = exp(s_c - M) / sum_d exp(s_d - M), M = max_d s_d (Eq. 4)."""
    s = np.asarray(s, np.float64)
    e = np.exp(s - s.max())
    return e / e.sum()


def decide_choice(s: np.ndarray) -> int:
    """argmax_c s_c; ties resolved by the fixed supplied order (lowest index)."""
    s = np.asarray(s, np.float64)
    best = 0
    for c in range(1, len(s)):
        if s[c] > s[best]:
            best = c
    return best


def decide_binary(s: np.ndarray) -> float:
    """Candidate set ordered (false, true); returns q(true)."""
    if len(s) != 2:
        raise ValueError("binary decisions need exactly two candidates")
    return float(normalize(s)[1])


def decide_ordinal(s: np.ndarray) -> float:
    """Expected zero-based level sum_i i q(i) over K ordered levels."""
    if len(s) < 2:
        raise ValueError("ordinal decisions need at least two levels")
    q = normalize(s)
    return float(sum(i * q[i] for i in range(len(q))))


def decide(mode: str, q_cand_offsets: np.ndarray, sums: np.ndarray):
    """Per question: (q over its candidates, choice, value) for mode in
    {"choice", "binary", "ordinal"}; value is None for "choice"."""
    qs, choice, value = np.zeros(len(sums)), [], []
    for q in range(len(q_cand_offsets) - 1):
        a, b = int(q_cand_offsets[q]), int(q_cand_offsets[q + 1])
        s = sums[a:b]
        qs[a:b] = normalize(s)
        choice.append(decide_choice(s))
        if mode == "binary":
            value.append(decide_binary(s))
        elif mode == "ordinal":
            value.append(decide_ordinal(s))
        else:
            value.append(None)
    return qs, np.asarray(choice, np.int32), value


# --------------------------------------------------------------------------
# evaluation against reference answers (Section 3.3, Section 5)
# --------------------------------------------------------------------------

def answer_classes(q_cand_offsets, cand_tok_offsets, cand_tokens) -> np.ndarray:
    """Per candidate: the index, within its question, of the first candidate
    whose token sequence is identical (identical text under one tokenizer)."""
    out = np.zeros(int(q_cand_offsets[-1]), np.int32)
    for q in range(len(q_cand_offsets) - 1):
        a, b = int(q_cand_offsets[q]), int(q_cand_offsets[q + 1])
        seqs = [tuple(int(t) for t in cand_tokens[cand_tok_offsets[c]:cand_tok_offsets[c + 1]])
                for c in range(a, b)]
        for j in range(b - a):
            out[a + j] = seqs.index(seqs[j])
    return out


def evaluate(q_cand_offsets, sums, gold, classes=None):
    """Per question: correct (the predicted label, Eq. 5's argmax, has the
    gold answer's text) and gold NLL = -ln of the summed q (Eq. 4) over the
    labels with the gold answer's text; plus their means over questions."""
    correct, nll = [], []
    for q in range(len(q_cand_offsets) - 1):
        a, b = int(q_cand_offsets[q]), int(q_cand_offsets[q + 1])
        cls = list(range(b - a)) if classes is None else [int(x) for x in classes[a:b]]
        p = normalize(sums[a:b])
        g = cls[int(gold[q])]
        correct.append(int(cls[decide_choice(sums[a:b])] == g))
        nll.append(-np.log(sum(p[j] for j in range(b - a) if cls[j] == g)))
    correct = np.asarray(correct, np.int32)
    nll = np.asarray(nll, np.float64)
    return correct, nll, float(np.mean(correct)), float(np.mean(nll))
