"""fp64 CPU oracle for teacher-forced candidate scoring (JET, arXiv 2609.33874).

TEST INFRASTRUCTURE ONLY. Nothing on the product path may import, call or
execute this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it. It shares no code with the HIP
path; the only common dependency is the seeded input generator ``jet_synth``,
which holds none of the method's arithmetic.

What it computes (plain definitions, no sharing, fp64 throughout):

* every candidate ``c`` of a question ``x`` is run as an independent full
  forward over ``x || y_c[1..m_c-1]`` (no prefix reuse, Section 4.1 names
  independent evaluation as the reference for isolation, Section 5.6);
* the logits of every scored position are materialised over the full
  vocabulary and turned into log-probabilities with the max-shifted form of
  Eq. 2 (Section 3.1);
* candidate scores are the sums of Eq. 3 (Section 3.2), normalised with
  Eq. 4 and turned into a choice / binary probability / ordinal expectation
  with Eq. 5 and the rules of Section 3.3.

The network itself is not defined by the paper (it scores Qwen-family GGUF
models). The decoder used here is a fixed reading: a pre-norm dense decoder
(RMSNorm, rotate-half RoPE, grouped-query attention, SwiGLU, untied head)
and, for hybrid models, gated delta-rule linear-attention layers. Those
blocks are pinned in the tests against independent library implementations
of the same blocks (transformers' Qwen2 and Qwen3-Next modules), against
closed forms and against invariants; see ``oracle.model``.

An *incremental* mode (prefill once, copy the retained state, continue per
candidate; Section 4.1) exists only so that the tests can check that prefix
sharing leaves results unchanged; its ``leak`` switch is the planted mistake
(state carried from one candidate into the next) that the isolation test must
catch.
"""
from .model import Model, forward, final_logprobs, upcast  # noqa: F401
from .score import (score_unshared, score_incremental, log_softmax_rows,  # noqa: F401
                    normalize, decide_choice, decide_binary, decide_ordinal, decide,
                    answer_classes, evaluate)
