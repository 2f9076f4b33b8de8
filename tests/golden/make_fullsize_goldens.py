"""Write the fp64 oracle's scores for sampled questions of the full-size
workloads into ``tests/golden/fullsize_<workload>.json``.

Only ``oracle`` and ``jet_synth`` are used: the expected values never come
from the GPU path. Each file records, next to the scores, the sha256 of every
tensor of the model file and of the sampled sub-workload, so a test that
regenerates the model from its seed can check that it compares against the
same inputs. Every candidate is an independent full forward with no prefix
sharing (Section 5.6 takes independent execution as the reference).

Usage: python tests/golden/make_fullsize_goldens.py [workload ...]
(minutes to hours on a many-core host: the 27B-shape question is ~1.5 PFLOP
of fp64 work; set JET_MODEL_CACHE to a disk with room for the model files).
"""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import jet_synth  # noqa: E402
import oracle  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))


def _longest(wl):
    return int(np.argmax(np.diff(wl.prefix_offsets)))


def _cases(name, wl):
    """(label, question list, candidate index list or None for all)."""
    first = {"dense_1p5b_k4": 8, "dense_1p5b_binary": 8, "dense_1p5b_ordinal": 4,
             "hybrid_4b_k4": 4, "dense_27b_k10": 1}[name]
    qs = list(range(first))
    ql = _longest(wl)
    cases = [("first questions in seed order", qs, None)]
    if name == "dense_27b_k10":
        # the longest-prefix question: its shortest candidate only
        lens = [len(y) for y in wl.candidates(ql)]
        cases.append(("longest-prefix question, shortest candidate", [ql], [int(np.argmin(lens))]))
    elif ql not in qs:
        cases.append(("longest-prefix question", [ql], None))
    return cases


def _sub(wl, qs, cands):
    if cands is None:
        return wl.subset(qs)
    (q,) = qs
    cs = wl.candidates(q)
    return jet_synth.from_lists([wl.prefix(q)], [[cs[j] for j in cands]])


def make(name: str) -> str:
    spec = jet_synth.WORKLOADS[name]["model"]
    t0 = time.time()
    path = jet_synth.ensure_model(spec)
    print(f"[golden] {name}: model {path} ready in {time.time() - t0:.0f}s", flush=True)
    t0 = time.time()
    digests = jet_synth.tensor_digests(path)
    print(f"[golden] {name}: digests in {time.time() - t0:.0f}s", flush=True)
    wl = jet_synth.make_workload(name)
    out = dict(workload=name, model=spec, seed=jet_synth.MASTER_SEED,
               producer="tests/golden/make_fullsize_goldens.py (oracle.score_unshared, fp64)",
               model_sha256=digests, cases=[])
    for label, qs, cands in _cases(name, wl):
        sub = _sub(wl, qs, cands)
        t0 = time.time()
        tok, sums = oracle.score_unshared(path, sub)
        dt = time.time() - t0
        print(f"[golden] {name}: {label} {qs} cands {cands}: {dt:.0f}s", flush=True)
        out["cases"].append(dict(label=label, questions=qs, candidates=cands,
                                 subset_sha256=jet_synth.workload_digest(sub),
                                 oracle_seconds=round(dt, 1),
                                 token_logprob=[float(x) for x in tok],
                                 cand_sum=[float(x) for x in sums]))
    dst = os.path.join(HERE, f"fullsize_{name}.json")
    with open(dst, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    return dst


if __name__ == "__main__":
    names = sys.argv[1:] or ["dense_1p5b_k4", "dense_1p5b_binary", "dense_1p5b_ordinal",
                             "hybrid_4b_k4", "dense_27b_k10"]
    for n in names:
        print("[golden] wrote", make(n), flush=True)
