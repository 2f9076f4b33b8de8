"""fp64 forward pass of the synthetic decoders (test infrastructure only).

The paper scores pretrained Qwen-family models and does not define their
layers. The blocks below are this implementation's reading of such a decoder;
each one is written as its textbook definition:

* ``rmsnorm``: x / sqrt(mean(x^2) + eps) * g.
* ``rope``: rotate-half pairing (i, i + hd/2), angle pos * theta^(-2i/hd),
  tabulated in fp64.
* ``attention``: softmax(q k^T / sqrt(hd)) v per query head, key/value head
  ``h // (Hq/Hkv)``, key j visible to query i iff pos_j <= pos_i.
* FFN: down(silu(gate(a)) * up(a)).
* ``moe_ffn`` (models with experts): the router scores every expert with one
  linear map; each row keeps its top_k experts by router logit (lowest expert
  index first among equal logits) and mixes their FFN outputs with weights
  softmax over the kept logits (the full softmax renormalised over the kept
  experts); a shared expert's FFN output is added scaled by
  sigmoid(shared_router . a).
* ``gdn_*``: gated delta rule (per head, state S of shape [dv, dk]):
  S <- alpha S;  S <- S + beta (v - S k) k^T;  o = S q, with
  q, k l2-normalised (eps 1e-6), q scaled by 1/sqrt(dk), beta = sigmoid(b),
  alpha = exp(-exp(A_log) * softplus(a + dt_bias)), a causal depthwise
  convolution (kernel 4) + SiLU in front of q, k, v, and an output
  RMSNorm(o) * silu(z) per head.

Pins (tests): transformers' Qwen2 decoder, Qwen3-Next gated delta-rule
layer and Qwen2-MoE sparse block on the same weights, all-zero weights, RoPE and attention special
cases, gated delta-rule closed forms.
"""
from __future__ import annotations

import numpy as np

import jet_synth


def upcast(raw) -> np.ndarray:
    """Exact conversion of stored weights to float64: bf16 bits, f32, or
    block-quantized int8 / int4 values q with one exponent e per block of
    consecutive values along the last dimension (weight = q * 2^e)."""
    if isinstance(raw, (jet_synth.Q8Raw, jet_synth.Q4Raw)):
        q = np.asarray(raw.q, np.float64)
        e = np.repeat(np.asarray(raw.e, np.int64), q.shape[-1] // raw.e.shape[-1], axis=-1)
        return np.ldexp(q, e)
    raw = np.asarray(raw)
    if raw.dtype == np.uint16:
        return (raw.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return raw.astype(np.float64)


class Model:
    """A model file opened for the oracle; weights are upcast on demand."""

    def __init__(self, path: str):
        self.path = path
        self.h = jet_synth.read_header(path)
        self._index = {t["name"]: t for t in self.h["tensors"]}
        self.d = self.h["d_model"]
        self.V = self.h["vocab"]
        self.eps = float(self.h["rms_eps"])
        self.layer_types = self.h["layer_types"]
        self.n_experts = int(self.h.get("n_experts", 0))
        self.top_k = int(self.h.get("top_k", 0))

    def w(self, name: str) -> np.ndarray:
        return upcast(jet_synth.tensor_raw(self.path, name, self.h))

    def layer(self, i: int) -> dict:
        """Weights of block i; the per-expert matrices are read by ``expert``."""
        p = f"blk.{i}."
        return {k[len(p):]: self.w(k) for k in self._index
                if k.startswith(p) and k[len(p):] not in ("moe_gate", "moe_up", "moe_down")}

    def expert(self, i: int, name: str, e: int) -> np.ndarray:
        """Matrix e of the [E, rows, cols] expert tensor ``name`` of block i."""
        return upcast(jet_synth.tensor_raw(self.path, f"blk.{i}.{name}", self.h)[e])


# --------------------------------------------------------------------------
# blocks
# --------------------------------------------------------------------------

def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def rope_angles(pos: np.ndarray, hd: int, theta: float) -> tuple[np.ndarray, np.ndarray]:
    i = np.arange(hd // 2, dtype=np.float64)
    inv = theta ** (-(2.0 * i) / hd)
    ang = np.asarray(pos, np.float64)[:, None] * inv[None, :]
    return np.cos(ang), np.sin(ang)


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """x: [n, H, hd]; rotate the pairs (i, i + hd/2) by pos * theta^(-2i/hd)."""
    hd = x.shape[-1]
    c, s = rope_angles(pos, hd, theta)
    c, s = c[:, None, :], s[:, None, :]
    x1, x2 = x[..., : hd // 2], x[..., hd // 2:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
              q_pos: np.ndarray, k_pos: np.ndarray) -> np.ndarray:
    """Causal grouped-query softmax attention.

    q: [n, Hq, hd]; k, v: [nk, Hkv, hd]; key j is visible to query i iff
    k_pos[j] <= q_pos[i].
    """
    n, hq, hd = q.shape
    hkv = k.shape[1]
    group = hq // hkv
    visible = np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None]
    out = np.empty((n, hq, v.shape[2]))
    for h in range(hq):
        kh = h // group
        s = q[:, h, :] @ k[:, kh, :].T / np.sqrt(hd)
        s = np.where(visible, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v[:, kh, :]
    return out


def swiglu_ffn(a: np.ndarray, Wg: np.ndarray, Wu: np.ndarray, Wd: np.ndarray) -> np.ndarray:
    return (silu(a @ Wg.T) * (a @ Wu.T)) @ Wd.T


def moe_route(logits: np.ndarray, top_k: int) -> tuple[np.ndarray, np.ndarray]:
    """Per row: the top_k expert indices by logit (lowest index first among
    equal logits) and their weights, softmax over the kept logits."""
    sel = np.argsort(-logits, axis=1, kind="stable")[:, :top_k]
    z = np.take_along_axis(logits, sel, axis=1)
    w = np.exp(z - z.max(axis=1, keepdims=True))
    return sel, w / w.sum(axis=1, keepdims=True)


def moe_ffn(model: "Model", li: int, W: dict, a: np.ndarray, forced: np.ndarray | None = None,
            gaps: list | None = None) -> np.ndarray:
    """Mixture-of-experts FFN of block li on rows a [n, d].

    ``forced`` [n, top_k] (optional) names the experts to keep per row, for
    checking a routing decided elsewhere: a row whose first entry is -1 is
    routed here; any other row keeps exactly the named experts, mixed with
    weights softmax over *these* logits at those experts (the same rule as
    unforced routing, applied to the given set). For every forced row,
    ``gaps`` (if a list) receives min(logit of a kept expert) - max(logit of
    an expert not kept): >= 0 when the set is a top-k of these logits,
    negative by how far it is from one.
    """
    logits = a @ W["moe_router"].T
    sel, wts = moe_route(logits, model.top_k)
    if forced is not None:
        rows = np.nonzero(forced[:, 0] >= 0)[0]
        if len(rows):
            fs = forced[rows].astype(np.int64)
            z = np.take_along_axis(logits[rows], fs, axis=1)
            w = np.exp(z - z.max(axis=1, keepdims=True))
            sel = sel.copy()
            wts = wts.copy()
            sel[rows] = fs
            wts[rows] = w / w.sum(axis=1, keepdims=True)
            if gaps is not None:
                out_mask = np.ones((len(rows), logits.shape[1]), bool)
                np.put_along_axis(out_mask, fs, False, axis=1)
                rest = np.where(out_mask, logits[rows], -np.inf).max(axis=1)
                gaps.append(z.min(axis=1) - rest)
    out = np.zeros_like(a)
    for e in np.unique(sel):
        rows, slot = np.nonzero(sel == e)
        y = swiglu_ffn(a[rows], model.expert(li, "moe_gate", e), model.expert(li, "moe_up", e),
                       model.expert(li, "moe_down", e))
        out[rows] += wts[rows, slot][:, None] * y
    if "shared_gate" in W:
        g = 1.0 / (1.0 + np.exp(-(a @ W["shared_router"].T)))
        out += g * swiglu_ffn(a, W["shared_gate"], W["shared_up"], W["shared_down"])
    return out


def l2norm(x: np.ndarray, eps: float = 1e-6) -> np.ndarray:
    return x / np.sqrt(np.sum(x * x, axis=-1, keepdims=True) + eps)


def softplus(x: np.ndarray) -> np.ndarray:
    return np.logaddexp(0.0, x)


def causal_conv(x: np.ndarray, tail: np.ndarray, w: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """Depthwise causal convolution over time.

    x: [n, C] new inputs; tail: [kc-1, C] the inputs just before them (zeros
    at the start of a sequence); w: [C, kc], w[:, kc-1] multiplies the
    current row. Returns (output [n, C], new tail).
    """
    kc = w.shape[1]
    full = np.concatenate([tail, x], axis=0)
    n = x.shape[0]
    out = np.zeros_like(x)
    for j in range(kc):
        out += full[j:j + n] * w[:, j][None, :]
    return out, full[full.shape[0] - (kc - 1):].copy()


def gdn_recurrence(q: np.ndarray, k: np.ndarray, v: np.ndarray, alpha: np.ndarray,
                   beta: np.ndarray, S: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """Gated delta rule, stepwise.

    q, k: [n, H, dk]; v: [n, H, dv]; alpha, beta: [n, H]; S: [H, dv, dk]
    (initial state, not modified). Returns (o [n, H, dv], final state).
    """
    S = S.copy()
    n = q.shape[0]
    o = np.empty(v.shape)
    for t in range(n):
        S *= alpha[t][:, None, None]
        pred = np.matmul(S, k[t][:, :, None])[:, :, 0]          # S k
        S += (beta[t][:, None] * (v[t] - pred))[:, :, None] * k[t][:, None, :]
        o[t] = np.matmul(S, q[t][:, :, None])[:, :, 0]          # S q
    return o, S


# --------------------------------------------------------------------------
# forward over a batch of independent sequences
# --------------------------------------------------------------------------

def _attn_layer(h, W, a_rows, seq_slices, starts, states, li, want_state):
    H_q, H_kv, hd, theta = h["n_heads"], h["n_kv_heads"], h["head_dim"], float(h["rope_theta"])
    q_all = a_rows @ W["wq"].T
    k_all = a_rows @ W["wk"].T
    v_all = a_rows @ W["wv"].T
    out = np.empty((a_rows.shape[0], H_q * hd))
    new_states = []
    for i, sl in enumerate(seq_slices):
        n = sl.stop - sl.start
        pos = starts[i] + np.arange(n)
        q = rope(q_all[sl].reshape(n, H_q, hd), pos, theta)
        k = rope(k_all[sl].reshape(n, H_kv, hd), pos, theta)
        v = v_all[sl].reshape(n, H_kv, hd)
        st = states[i][li] if states[i] is not None else None
        if st is not None:
            k_full = np.concatenate([st[0], k]); v_full = np.concatenate([st[1], v])
            kpos = np.concatenate([st[2], pos])
        else:
            k_full, v_full, kpos = k, v, pos
        out[sl] = attention(q, k_full, v_full, pos, kpos).reshape(n, H_q * hd)
        new_states.append((k_full, v_full, kpos) if want_state else None)
    return out @ W["wo"].T, new_states


def _gdn_layer(h, W, a_rows, seq_slices, states, li, want_state, eps):
    H, dk, dv = h["gdn_heads"], h["gdn_dk"], h["gdn_dv"]
    kc = h["conv_kernel"]
    x_all = np.concatenate([a_rows @ W["gdn_wq"].T, a_rows @ W["gdn_wk"].T,
                            a_rows @ W["gdn_wv"].T], axis=1)
    z_all = a_rows @ W["gdn_wz"].T
    b_all = a_rows @ W["gdn_wb"].T
    a_in = a_rows @ W["gdn_wa"].T
    beta_all = 1.0 / (1.0 + np.exp(-b_all))
    alpha_all = np.exp(-np.exp(W["gdn_A_log"])[None, :] * softplus(a_in + W["gdn_dt_bias"][None, :]))
    out = np.empty((a_rows.shape[0], H * dv))
    new_states = []
    for i, sl in enumerate(seq_slices):
        n = sl.stop - sl.start
        st = states[i][li] if states[i] is not None else None
        S0 = st[0] if st is not None else np.zeros((H, dv, dk))
        tail = st[1] if st is not None else np.zeros((kc - 1, x_all.shape[1]))
        xc, new_tail = causal_conv(x_all[sl], tail, W["gdn_conv"])
        xc = silu(xc)
        q = l2norm(xc[:, :H * dk].reshape(n, H, dk)) / np.sqrt(dk)
        k = l2norm(xc[:, H * dk:2 * H * dk].reshape(n, H, dk))
        v = xc[:, 2 * H * dk:].reshape(n, H, dv)
        o, S1 = gdn_recurrence(q, k, v, alpha_all[sl], beta_all[sl], S0)
        y = rmsnorm(o, W["gdn_norm"], eps) * silu(z_all[sl].reshape(n, H, dv))
        out[sl] = y.reshape(n, H * dv)
        new_states.append((S1, new_tail) if want_state else None)
    return out @ W["gdn_wo"].T, new_states


def forward(model: Model, seqs: list, starts: list | None = None,
            states: list | None = None, want_state: bool = False,
            row_chunk: int = 8192, routes: list | None = None, route_gaps: list | None = None):
    """Run every layer over a batch of independent token sequences.

    seqs[i] holds new token ids whose first position is starts[i]; states[i]
    is None (fresh sequence) or the per-layer state returned by an earlier
    call for the tokens before them. Independent sequences are stacked as
    rows of the same matrix products; attention and the recurrence are run
    per sequence. Mixture-of-experts models only: routes[i] (optional) is an
    int array [n_layers, n_i, top_k] of experts to keep per layer and row
    (-1 rows routed here, see ``moe_ffn``); route_gaps collects the forced
    rows' top-k gaps of every layer. Returns (list of hidden states [n_i, d]
    before the final norm, list of per-layer states or None).
    """
    h = model.h
    starts = starts or [0] * len(seqs)
    states = states or [None] * len(seqs)
    lens = [len(s) for s in seqs]
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(int)
    slices = [slice(offs[i], offs[i + 1]) for i in range(len(seqs))]
    ids = np.concatenate([np.asarray(s, np.int64) for s in seqs])
    E = jet_synth.tensor_raw(model.path, "tok_embed", h)
    x = upcast(E[ids])
    out_states = [[None] * len(model.layer_types) for _ in seqs] if want_state else None
    forced_all = None
    if routes is not None:
        forced_all = np.concatenate([np.asarray(r, np.int64) for r in routes], axis=1)  # [L, rows, k]
    for li, lt in enumerate(model.layer_types):
        W = model.layer(li)
        a = rmsnorm(x, W["attn_norm"], model.eps)
        if lt == "attn":
            delta, st = _attn_layer(h, W, a, slices, starts, states, li, want_state)
        else:
            delta, st = _gdn_layer(h, W, a, slices, states, li, want_state, model.eps)
        x = x + delta
        if want_state:
            for i in range(len(seqs)):
                out_states[i][li] = st[i]
        for r0 in range(0, x.shape[0], row_chunk):
            r = slice(r0, min(r0 + row_chunk, x.shape[0]))
            a = rmsnorm(x[r], W["ffn_norm"], model.eps)
            if model.n_experts:
                fr = None if forced_all is None else forced_all[li, r]
                x[r] = x[r] + moe_ffn(model, li, W, a, fr, route_gaps)
            else:
                x[r] = x[r] + swiglu_ffn(a, W["w_gate"], W["w_up"], W["w_down"])
        del W
    return [x[sl] for sl in slices], out_states


def final_logprobs(model: Model, rows: np.ndarray, targets: np.ndarray,
                   W_lm: np.ndarray | None = None) -> np.ndarray:
    """Final RMSNorm, full-vocabulary logits, then Eq. 2 for each row's target."""
    from .score import log_softmax_rows
    g = model.w("final_norm")
    f = rmsnorm(rows, g, model.eps)
    W = model.w("lm_head") if W_lm is None else W_lm
    z = f @ W.T
    return log_softmax_rows(z, np.asarray(targets, np.int64))
