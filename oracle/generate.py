"""Reasoning traces of the oracle (test infrastructure only).

Section 3.4 (optional reasoning) generates a trace once per question and
freezes it into the context that every candidate is then scored against; the
paper names no sampler. The reading followed here (and by the GPU path) is
Gumbel-max sampling at a temperature tau: token t of question q is

    argmax_v  z_v / tau + G(seed, q, t, v)        (tau > 0)
    argmax_v  z_v                                 (tau = 0)

over the full vocabulary, z the next-token logits after x_q || trace_q[:t],
lowest token id among equal keys. By the Gumbel-max property the first form
draws from softmax(z / tau). G = -log(-log U), where U comes from a
counter-based generator so that every (q, t, v) has its own draw without any
state: SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom
number generators", OOPSLA 2014), output number 1 + (q << 38 | t << 18 | v)
of the stream seeded with `seed`, its top 53 bits mapped to (0, 1) as
(bits + 1/2) / 2^53.

Every step here is a full fp64 forward over the whole sequence so far (no
cache): slow and plainly the definition.
"""
from __future__ import annotations

import numpy as np

from .model import Model, forward, rmsnorm

_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def splitmix64_at(seed: int, index) -> np.ndarray:
    """Output number index + 1 of the SplitMix64 stream seeded with `seed`:
    the state after index + 1 steps of adding the golden gamma, mixed."""
    idx = np.asarray(index, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(seed & 0xFFFFFFFFFFFFFFFF) + (idx + np.uint64(1)) * _GAMMA
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        return z ^ (z >> np.uint64(31))


def uniform_at(seed: int, q: int, t: int, v) -> np.ndarray:
    """U in (0, 1) of (question q, step t, token v)."""
    v = np.asarray(v, dtype=np.uint64)
    index = (np.uint64(q) << np.uint64(38)) | (np.uint64(t) << np.uint64(18)) | v
    bits = splitmix64_at(seed, index) >> np.uint64(11)
    return (bits.astype(np.float64) + 0.5) * 2.0 ** -53


def gumbel_at(seed: int, q: int, t: int, v) -> np.ndarray:
    return -np.log(-np.log(uniform_at(seed, q, t, v)))


def sample_keys(z: np.ndarray, tau: float, seed: int, q: int, t: int) -> np.ndarray:
    """The keys whose argmax is the sampled token (see the module text)."""
    z = np.asarray(z, dtype=np.float64)
    if tau == 0:
        return z.copy()
    return z / tau + gumbel_at(seed, q, t, np.arange(len(z)))


def first_argmax(keys: np.ndarray) -> int:
    """The lowest index among the maxima (numpy's argmax already does this)."""
    return int(np.argmax(keys))


def next_logits(model: Model, seq) -> np.ndarray:
    """Logits of the token after `seq`: final norm of the last hidden row
    times the untied LM head, over the full vocabulary."""
    hid, _ = forward(model, [np.asarray(seq, np.int64)])
    f = rmsnorm(hid[0][-1:], model.w("final_norm"), model.eps)
    return (f @ model.w("lm_head").T)[0]


def generate_trace(model: Model | str, prefix, q: int, n_steps: int, tau: float, seed: int,
                   forced=None):
    """Trace of question q (its index among the call's questions) after
    `prefix`. Returns (tokens, steps): steps[t] holds the step's keys' maximum,
    the key of the token taken and the oracle's own choice. With `forced`,
    token t is forced[t] (the sequence continues with it) and the record shows
    how far it is from the oracle's choice."""
    model = Model(model) if isinstance(model, str) else model
    seq = [int(x) for x in prefix]
    tokens, steps = [], []
    for t in range(n_steps):
        keys = sample_keys(next_logits(model, seq), tau, seed, q, t)
        own = first_argmax(keys)
        y = own if forced is None else int(forced[t])
        steps.append({"max_key": float(keys[own]), "key": float(keys[y]), "choice": own})
        tokens.append(y)
        seq.append(y)
    return np.asarray(tokens, np.int32), steps
