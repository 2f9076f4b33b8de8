#!/usr/bin/env python3
"""Throughput of teacher-forced candidate scoring on one MI355X.

A step is one pass of the whole hot path over one batch: prefill every
question prefix once (retaining its attention cache), score every candidate
against it (batched candidate bodies, fused LM head + full-vocabulary
log-sum-exp, per-candidate sums), copy the sums to the host and decide.
Inputs (token ids) are resident in HBM before the timed region starts.

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3    # MI355X fp32 (matrix and vector)
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E

MODE_OF = {"dense_1p5b_binary": "binary", "dense_1p5b_ordinal": "ordinal"}
# compute mode per workload: single fp16 activations meet the tolerances on
# every candidate of the 28-layer workloads with room (per candidate 0.026
# against 0.05); on the 64-layer model single fp16 misses them (per token
# 0.042, per candidate 0.21 over the whole workload) and so does f16p (per
# candidate 0.090, 24 of 640 candidates over 0.05); on the 32-layer hybrid
# single fp16 sits at the per-candidate bound (0.047..0.056 depending on the
# rounding order of the delta-rule kernels) and f16p too (0.052). The (hi, lo)
# bf16 pairs stay within 3.4e-4 per token and 1.7e-3 per candidate of the
# oracle on the sampled questions of both
DEFAULT_DTYPE = {"dense_27b_k10": "bf16", "hybrid_4b_k4": "bf16"}

# Sources of each kernel class: a counter summary under profiles/ holds the
# hash of these files as they were when the counters were taken.
KERNEL_SOURCES = {
    "gemm": ["device.h", "gemm_core.h", "k_gemm.hip"],
    "lmhead": ["device.h", "gemm_core.h", "k_gemm.hip"],
    "attn": ["device.h", "k_attn.hip"],
    "gdn": ["device.h", "k_gdn.hip"],
}


def source_hash(cls: str) -> str:
    """Hash of the code (comments and whitespace removed) of a kernel class."""
    import hashlib
    import re
    key = "gemm" if cls.startswith("gemm") else cls.split("_")[0]
    h = hashlib.sha256()
    for f in KERNEL_SOURCES.get(key, []):
        with open(os.path.join(ROOT, "paper_2609_33874_amd", "csrc", f)) as fh:
            code = re.sub(r"/\*.*?\*/", " ", fh.read(), flags=re.S)
        code = re.sub(r"//[^\n]*", " ", code)
        h.update(" ".join(code.split()).encode())
    return h.hexdigest()[:16]


def measured_traffic(cls: str, wname: str, dtype: str):
    """HBM bytes per launch of kernel class `cls` on workload `wname` in mode
    `dtype` from the committed counter summary (FETCH_SIZE and WRITE_SIZE, each
    scaled by what the counter reads for a plain copy of known size), or None
    when there is no summary for that mode or the kernel's sources changed
    since it was taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{cls}_{wname}_{dtype}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_hash") != source_hash(cls) or t.get("dtype") != dtype:
        return None
    return t["hbm_bytes_per_launch"]


def calibrate_copy(nbytes: int = 1 << 30, reps: int = 4) -> int:
    """A plain device-to-device copy of known size, for scaling the HBM byte
    counters (run under rocprofv3 --pmc)."""
    import torch
    x = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda:0").fill_(1.0)
    y = torch.empty_like(x)
    for _ in range(reps):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "reps": reps}), flush=True)
    return 0


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def describe(wname: str) -> dict:
    import jet_synth
    r = jet_synth.WORKLOADS[wname]
    s = jet_synth.full_spec(r["model"])
    return {"workload": wname,
            "model": (f"{s['arch']} {s['n_layers']}L d={s['d_model']} heads {s['n_heads']}/{s['n_kv_heads']} "
                      f"hd={s['head_dim']} "
                      + (f"experts {s['n_experts']} top {s['top_k']} expert ffn={s['moe_ffn']} "
                         f"shared ffn={s['shared_ffn']} " if s["n_experts"] else f"ffn={s['ffn']} ")
                      + f"vocab={s['vocab']} {s['dtype']} random N(0,0.02)"),
            "questions": r["Q"], "prefix_len": list(r["P"]), "prefix_ids": r["ids"],
            "candidates_per_question": r["K"], "candidate_len": list(r["m"])}


def cpu_facts() -> dict:
    """The host CPU the oracle runs on: model, logical CPUs, BLAS threads."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    return {"cpu_model": model, "logical_cpus": os.cpu_count(), "affinity_cpus": len(os.sched_getaffinity(0)),
            "blas_threads": int(threads)}


def cpu_baseline(path: str, wl, min_seconds: float = 10.0, max_questions: int = 16) -> dict:
    """The fp64 oracle (independent full forward per candidate) on the first
    questions of the workload, one at a time, until at least min_seconds of
    CPU work (at most max_questions questions)."""
    import oracle
    facts = cpu_facts()
    threads = facts["blas_threads"]
    done, dt = [], 0.0
    for q in range(min(max_questions, wl.n_questions)):
        sub = wl.subset([q])
        t0 = time.perf_counter()
        oracle.score_unshared(path, sub)
        dt += time.perf_counter() - t0
        done.append(q)
        log(f"oracle question {q} done ({dt:.1f}s)")
        if dt >= min_seconds:
            break
    sub = wl.subset(done)
    P = int(sub.prefix_offsets[-1])
    m = np.diff(sub.cand_tok_offsets)
    return {"value": len(done) / dt, "unit": "questions/s", "cores": int(threads), "kind": "oracle",
            "seconds": dt, **facts,
            "sample": (f"questions 0..{done[-1]} of the workload ({len(done)} questions: {P} prefix tokens, "
                       f"{len(m)} candidates, {int(m.sum())} scored tokens); every candidate an independent "
                       f"fp64 forward")}


def cpu_baseline_layers(path: str, wl, layers=(1, 2)) -> dict:
    """The fp64 oracle where one question is far beyond seconds of CPU work:
    the first candidate of question 0 run through the first layers[0] and
    layers[1] layers of the model (embedding, those layers, final norm, LM
    head over the full vocabulary, Eq. 2-3), timed; the difference is the
    time of one layer at that sequence length, the rest the per-call fixed
    part. Extrapolated to question 0 as the oracle runs it: one call with
    every candidate an independent sequence of P + m - 1 rows through all
    layers (layer time scaled by rows: the projections and FFN, linear in
    rows, are over 90% of a layer's work at these lengths)."""
    import jet_synth
    import oracle
    facts = cpu_facts()
    cands = wl.candidates(0)
    sub = jet_synth.from_lists([wl.prefix(0)], [[cands[0]]])
    model = oracle.Model(path)
    all_layers = list(model.layer_types)
    t = []
    for n in layers:
        model.layer_types = all_layers[:n]
        t0 = time.perf_counter()
        oracle.score_unshared(model, sub)
        t.append(time.perf_counter() - t0)
        log(f"oracle, question 0 candidate 0, first {n} layer(s): {t[-1]:.1f}s")
    per_layer = (t[1] - t[0]) / (layers[1] - layers[0])
    fixed = max(t[0] - layers[0] * per_layer, 0.0)
    P = len(wl.prefix(0))
    rows_sample = P + len(cands[0]) - 1
    rows_q = sum(P + len(y) - 1 for y in cands)
    t_q = fixed + len(all_layers) * per_layer * rows_q / rows_sample
    return {"value": 1.0 / t_q, "unit": "questions/s", "cores": facts["blas_threads"], "kind": "oracle",
            "seconds": sum(t), "extrapolated_seconds_per_question": round(t_q, 1), **facts,
            "sample": (f"question 0, candidate 0 ({rows_sample} positions): the oracle through the first "
                       f"{layers[0]} and {layers[1]} of {len(all_layers)} layers plus the full-vocabulary LM "
                       f"head, timed ({t[0]:.1f}s, {t[1]:.1f}s); per-layer time {per_layer:.2f}s, fixed part "
                       f"{fixed:.2f}s; extrapolated to question 0's {len(cands)} candidates ({rows_q} "
                       f"positions) through all {len(all_layers)} layers")}


REUSE_WORKLOAD = "dense_1p5b_k4"


def unshared_workload(wl):
    """Every candidate as its own question (its prefix prefilled again)."""
    import jet_synth
    pre, cands = [], []
    for q in range(wl.n_questions):
        for y in wl.candidates(q):
            pre.append(wl.prefix(q))
            cands.append([y])
    return jet_synth.from_lists(pre, cands)


class Runner:
    """One model on cuda:0 and the timed step of the hot path."""

    def __init__(self, wname: str, dtype: str, timing: bool, record_routes: bool = False):
        import torch
        import jet_synth
        from paper_2609_33874_amd import jet as J
        self.torch, self.J = torch, J
        self.wname = wname
        spec = jet_synth.WORKLOADS[wname]["model"]
        t = time.perf_counter()
        self.path = jet_synth.ensure_model(spec, evict=True)
        log(f"model file {self.path} ready in {time.perf_counter() - t:.1f}s")
        self.wl = jet_synth.make_workload(wname)
        self.mode = {"binary": J.JET_BINARY, "ordinal": J.JET_ORDINAL}.get(MODE_OF.get(wname, ""), J.JET_CHOICE)
        self.dev = torch.device("cuda:0")
        stream = torch.cuda.current_stream(self.dev)
        flags = (J.JET_FLAG_KERNEL_TIMING if timing else 0) | (J.JET_FLAG_RECORD_ROUTES if record_routes else 0)
        jdt = {"f16": J.JET_F16, "f16p": J.JET_F16P, "bf16": J.JET_BF16, "fp32": J.JET_FP32}[dtype]
        t = time.perf_counter()
        self.model = J.jet_model_load(self.path, dtype=jdt, device=0, hip_stream=stream.cuda_stream, flags=flags)
        self.load_s = time.perf_counter() - t
        log(f"model loaded in {self.load_s:.1f}s")
        self.phase = {"prefill": 0.0, "score": 0.0, "decide": 0.0}

    def inputs(self, w):
        torch = self.torch
        return (torch.from_numpy(w.prefix_tokens).to(self.dev), torch.from_numpy(w.cand_tokens).to(self.dev),
                torch.empty(int(w.cand_tok_offsets[-1]), dtype=torch.float32, device=self.dev),
                torch.empty(w.n_candidates, dtype=torch.float32, device=self.dev))

    def step(self, w, inp):
        J = self.J
        d_pre, d_cand, o_tok, o_sum = inp
        a = time.perf_counter()
        p = J.jet_prefill_prefix(self.model, w.prefix_offsets, d_pre)
        b = time.perf_counter()
        J.jet_score_candidates(self.model, p, w.q_cand_offsets, w.cand_tok_offsets, d_cand, o_tok, o_sum)
        c = time.perf_counter()
        sums = o_sum.cpu().numpy()
        J.jet_decide(self.mode, w.q_cand_offsets, sums)
        d = time.perf_counter()
        J.jet_prefix_free(p)
        self.phase["prefill"] += b - a
        self.phase["score"] += c - b
        self.phase["decide"] += d - c

    def timed(self, w, inp, steps: int, what: str) -> float:
        """Seconds for `steps` steps, bracketed by device synchronisation."""
        self.torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            self.step(w, inp)
            log(f"{what} step {i + 1}/{steps} done")
        self.torch.cuda.synchronize()
        return time.perf_counter() - t0

    def free(self):
        self.J.jet_model_free(self.model)


def tolerance_check(wname: str, dtype: str) -> dict:
    """Every token and candidate of the workload in mode `dtype` against the
    pair-bf16 mode (held by the full-size tests to the oracle's stored scores
    on sampled questions), or, on models with routed experts (no pair mode),
    against the fp32 mode with the share of prefill expert sets the two
    modes choose differently: the largest deviations and how many tokens and
    candidates pass the per-token 2e-2 / per-candidate 5e-2 bounds."""
    import numpy as np
    import jet_synth
    spec = jet_synth.MODEL_SPECS[jet_synth.WORKLOADS[wname]["model"]]
    moe = bool(spec.get("n_experts"))
    ref = "fp32" if moe else "bf16"
    out, routes = {}, {}
    for dt in (dtype, ref):
        r = Runner(wname, dt, timing=False, record_routes=moe)
        try:
            inp = r.inputs(r.wl)
            r.step(r.wl, inp)
            out[dt] = (inp[2].cpu().numpy().astype(np.float64), inp[3].cpu().numpy().astype(np.float64))
            if moe:
                routes[dt] = np.sort(r.J.jet_routes_get(r.model, 0), axis=2)  # [layer, prefix row, top_k]
        finally:
            r.free()
        log(f"tolerance check: {wname} scored in {dt}")
    dtok = np.abs(out[dtype][0] - out[ref][0])
    dsum = np.abs(out[dtype][1] - out[ref][1])
    extra = {}
    if moe:
        # expert sets of the prefill that differ between the two modes
        diff = np.any(routes[dtype] != routes[ref], axis=2)
        extra = {"prefix_rows": int(diff.shape[1]), "route_sets_differing": round(float(diff.mean()), 4),
                 "route_sets_differing_by_layer": [round(float(x), 3) for x in diff.mean(axis=1)],
                 "prefix_rows_with_a_differing_set": round(float(diff.any(axis=0).mean()), 4)}
    return {"workload": wname, "dtype": dtype, "reference": {"bf16": "bf16 (pair operands)", "fp32": "fp32"}[ref],
            **extra, "tokens": int(dtok.size),
            "candidates": int(dsum.size), "max_token_dev": float(dtok.max()), "max_cand_dev": float(dsum.max()),
            "rms_token_dev": float(np.sqrt((dtok ** 2).mean())), "tokens_over_2e-2": int((dtok > 2e-2).sum()),
            "candidates_over_5e-2": int((dsum > 5e-2).sum())}


def prefix_reuse(steps: int, unshared_steps: int) -> dict:
    """Shared vs unshared evaluation of the dense 1.5B choice workload with
    the same kernels (only the prefix sharing switched off)."""
    r = Runner(REUSE_WORKLOAD, "f16", timing=False)
    try:
        inp = r.inputs(r.wl)
        r.step(r.wl, inp)
        ms_sh = 1e3 * r.timed(r.wl, inp, steps, "shared (reuse)") / steps
        del inp
        un = unshared_workload(r.wl)
        uinp = r.inputs(un)
        r.step(un, uinp)  # warm-up (workspace growth)
        ms_un = 1e3 * r.timed(un, uinp, unshared_steps, "unshared (reuse)") / unshared_steps
        del uinp
    finally:
        r.free()
    return {"workload": REUSE_WORKLOAD, "dtype": "f16", "steps": steps, "unshared_steps": unshared_steps,
            "shared_ms_per_step": round(ms_sh, 3), "unshared_ms_per_step": round(ms_un, 3),
            "speedup": round(ms_un / ms_sh, 3)}


def reasoning_trace(steps: int, tau: float = 0.8, seed: int = 7) -> dict:
    """Optional reasoning (Section 3.4) on the dense 1.5B choice workload: a
    trace of `steps` sampled tokens per question (all 256 questions decode
    together, one row each per step) frozen into the retained prefix, then
    one scoring pass on the extended prefix. A decode step reads every
    weight matrix once and every question's cached K/V once; those bytes over
    the step time give its HBM rate."""
    import jet_synth
    import torch
    r = Runner(REUSE_WORKLOAD, "f16", timing=False)
    J, wl = r.J, r.wl
    Q = wl.n_questions
    try:
        inp = r.inputs(wl)
        p = J.jet_prefill_prefix(r.model, wl.prefix_offsets, inp[0])
        toks = torch.empty(Q * steps, dtype=torch.int32, device=r.dev)
        J.jet_generate_trace(r.model, p, Q, 2, tau, seed + 1)  # warm-up (workspace growth)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        J.jet_generate_trace(r.model, p, Q, steps, tau, seed, out=toks)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        log(f"reasoning trace: {steps} steps in {dt:.3f}s")
        # one scoring pass on the extended prefixes
        J.jet_score_candidates(r.model, p, wl.q_cand_offsets, wl.cand_tok_offsets, inp[1], inp[2], inp[3])
        finite = bool(torch.isfinite(inp[3]).all().item())
        J.jet_prefix_free(p)
    finally:
        r.free()
    sp = jet_synth.full_spec(jet_synth.WORKLOADS[REUSE_WORKLOAD]["model"])
    d, L, hd, F, V = sp["d_model"], sp["n_layers"], sp["head_dim"], sp["ffn"], sp["vocab"]
    Hq, Hkv = sp["n_heads"], sp["n_kv_heads"]
    w_bytes = 2.0 * (L * ((Hq + 2 * Hkv) * hd * d + d * Hq * hd + 3 * d * F) + V * d)
    T = float(wl.prefix_offsets[-1]) + 2 * Q  # after the warm-up trace
    kv_bytes = 2.0 * L * 2 * Hkv * hd * (T + Q * (steps + 1) / 2.0)  # mean over the steps
    step_s = dt / steps
    gbs = (w_bytes + kv_bytes) / step_s / 1e9
    return {"workload": REUSE_WORKLOAD, "dtype": "f16", "questions": Q, "steps": steps, "temperature": tau,
            "ms_per_step": round(1e3 * step_s, 3), "tokens_per_s": round(Q * steps / dt, 1),
            "hbm_bytes_per_step": round(w_bytes + kv_bytes), "hbm_gbs": round(gbs, 1),
            "hbm_frac": round(gbs / PEAK_HBM_GBS, 4), "scores_finite_after_trace": finite,
            "note": "per step: the LM head over the last rows, Gumbel-max sampling, one row per question through "
                    "every layer (its K/V appended to the question's cache); includes the one cache relayout"}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="dense_27b_k10",
                    help="default: the 27B-shape dense workload (the largest configuration on one GPU)")
    ap.add_argument("--dtype", choices=["f16", "f16p", "bf16"], default=None,
                    help="f16: bf16 weights held exactly as fp16, fp16 activations (one fp16 product per "
                         "multiply); f16p: f16 with (hi, lo) fp16 pairs on the attention side; bf16: bf16 "
                         "products over (hi, lo) bf16 activation pairs. Default: the fastest mode that meets "
                         "the tolerances on every candidate of the workload (bf16 on dense_27b_k10 and "
                         "hybrid_4b_k4, else f16)")
    ap.add_argument("--unshared-steps", type=int, default=None,
                    help="steps of unshared (per-candidate prefix) evaluation of the timed workload; "
                         "0 = skip; default 2 on dense_1p5b_k4, else 0")
    ap.add_argument("--reuse-steps", type=int, default=3,
                    help="shared steps of the dense 1.5B choice workload for its prefix-reuse speedup "
                         "(with 2 unshared steps), run after the timed workload when that is another "
                         "workload; 0 = skip")
    ap.add_argument("--trace-steps", type=int, default=16,
                    help="reasoning-trace decode steps on the dense 1.5B choice workload after the timed "
                         "workload (0 = skip)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-timing", action="store_true", help="do not time kernels with HIP events")
    ap.add_argument("--tolerance-check", action="store_true",
                    help="only score the whole workload in --dtype and in pair-bf16 and print the deviations")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a 1 GiB device copy (reference for the HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the scoring path has no "
              "multi-GPU mode (questions shard across GPUs with no exchange but the sums; not implemented)", file=sys.stderr)
        return 2
    if args.calibrate_copy:
        return calibrate_copy()
    if args.tolerance_check:
        dt = args.dtype or DEFAULT_DTYPE.get(args.workload, "f16")
        print(json.dumps(tolerance_check(args.workload, dt)), flush=True)
        return 0

    import torch

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        return 1
    wname = args.workload
    if args.dtype is None:
        args.dtype = DEFAULT_DTYPE.get(wname, "f16")
    if args.unshared_steps is None:
        args.unshared_steps = 2 if wname == REUSE_WORKLOAD else 0
    r = Runner(wname, args.dtype, timing=not args.no_timing)
    J, wl = r.J, r.wl
    Q = wl.n_questions
    T_p = int(wl.prefix_offsets[-1])
    T_c = int(wl.cand_tok_offsets[-1])
    inp = r.inputs(wl)
    for i in range(args.warmup):
        r.step(wl, inp)
        log(f"warmup step {i + 1}/{args.warmup} done")
    J.jet_stats_reset(r.model)
    for k in r.phase:
        r.phase[k] = 0.0
    elapsed = r.timed(wl, inp, args.steps, "timed")
    phase = dict(r.phase)
    stats = J.jet_stats_get(r.model)
    ms_step = 1e3 * elapsed / args.steps
    # evaluation utilities on the last step's scores (host; outside the timed
    # steps): equivalent labels and accuracy / gold NLL against seeded
    # synthetic gold labels (random weights: the values themselves mean nothing)
    sums = inp[3].cpu().numpy()
    gold = np.random.default_rng(7).integers(0, np.diff(wl.q_cand_offsets)).astype(np.int32)
    te = time.perf_counter()
    cls = J.jet_answer_classes(wl.q_cand_offsets, wl.cand_tok_offsets, wl.cand_tokens)
    J.jet_evaluate(wl.q_cand_offsets, sums, gold, cls)
    eval_ms = 1e3 * (time.perf_counter() - te)
    qps = Q * args.steps / elapsed

    # per-kernel-class rates from the HIP events around every launch
    kernels = {}
    for cls in J.KERNEL_CLASSES:
        n = stats["kernel_launches"][cls]
        ms = stats["kernel_ms"][cls]
        if n == 0:
            continue
        fl, by = stats["kernel_flops"][cls], stats["kernel_bytes"][cls]
        kernels[cls] = {"launches": n, "ms_total": round(ms, 3), "ms_per_launch": round(ms / n, 4),
                        "tflops": round(fl / (ms * 1e9), 2) if ms > 0 and fl > 0 else None,
                        "gbs": round(by / (ms * 1e6), 1) if ms > 0 and by > 0 else None}
    roofline = None
    if kernels and not args.no_timing:
        dom = max((c for c in kernels if c != "other"), key=lambda c: kernels[c]["ms_total"])
        n = stats["kernel_launches"][dom]
        ms_avg = stats["kernel_ms"][dom] / n
        if dom.startswith("attn"):
            ach = stats["kernel_bytes"][dom] / n / (ms_avg * 1e6)
            roofline = {"kernel": dom, "bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
                        "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": None}
        else:
            ach = stats["kernel_flops"][dom] / n / (ms_avg * 1e9)
            roofline = {"kernel": dom, "bound": "mfma", "achieved": round(ach, 1), "peak": PEAK_BF16_TFLOPS,
                        "unit": "TFLOP/s", "frac": round(ach / PEAK_BF16_TFLOPS, 4), "traffic": None}
        roofline["traffic"] = measured_traffic(dom, wname, args.dtype)
        if not dom.startswith("attn"):
            # (hi, lo) pair operands: two MFMA products per credited multiply
            # (bf16 everywhere; f16p on the attention side's GEMMs)
            pairs = args.dtype == "bf16" or (args.dtype == "f16p" and dom in ("gemm_qkv", "gemm_o"))
            roofline["mfma_products_per_multiply"] = 2 if pairs else 1
            roofline["executed_frac"] = round(roofline["frac"] * (2 if pairs else 1), 4)
        roofline["launches"] = n
        roofline["ms_per_launch"] = round(ms_avg, 4)
        roofline["flops_per_launch"] = stats["kernel_flops"][dom] / n
    gemm_cls = ["gemm_qkv", "gemm_o", "gemm_gateup", "gemm_down", "lmhead"]
    g_ms = sum(stats["kernel_ms"][c] for c in gemm_cls)
    g_fl = sum(stats["kernel_flops"][c] for c in gemm_cls)
    gemm_lm_frac = (g_fl / (g_ms * 1e9)) / PEAK_BF16_TFLOPS if g_ms > 0 else None

    result = {
        "metric": "questions/sec & scored tokens/sec on 1 MI355X; LM-head+GEMM % MFMA peak",
        "value": round(qps, 3), "unit": "questions/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": args.dtype, "data": "synthetic",
        "config": describe(wname),
        "scored_tokens_per_s": round(T_c * args.steps / elapsed, 1),
        "prefix_tokens_per_s": round(T_p * args.steps / phase["prefill"], 1),
        "phase_ms_per_step": {k: round(1e3 * v / args.steps, 2) for k, v in phase.items()},
        "model_load_s": round(r.load_s, 1),
        "gemm_lmhead_mfma_frac": round(gemm_lm_frac, 4) if gemm_lm_frac else None,
        # candidate attention over the shared prefix: bytes of the stored K/V
        # (read once per question and KV head) + Q + O per second, vs HBM peak
        "shared_prefix_attention_hbm_frac": (round(kernels["attn_cand"]["gbs"] / PEAK_HBM_GBS, 4)
                                             if kernels.get("attn_cand", {}).get("gbs") else None),
        "roofline": roofline, "kernels": kernels,
        "evaluate_ms": round(eval_ms, 3),
    }
    import jet_synth
    if jet_synth.MODEL_SPECS[jet_synth.WORKLOADS[wname]["model"]].get("n_experts"):
        # routed experts: scores hold to the oracle only under the same expert
        # choices (near-tie router logits swap experts between any two modes)
        result["parity_bound"] = ("under the GPU's expert choices only (the oracle run on the GPU's routes); "
                                  "unforced, routing near-ties make the error unbounded")

    if args.unshared_steps > 0:
        un = unshared_workload(wl)
        uinp = r.inputs(un)
        r.step(un, uinp)  # warm-up (workspace growth)
        ms_un = 1e3 * r.timed(un, uinp, args.unshared_steps, "unshared") / args.unshared_steps
        result["unshared_ms_per_step"] = round(ms_un, 3)
        result["prefix_reuse_speedup"] = round(ms_un / ms_step, 3)
        del uinp
    del inp
    r.free()
    if wname != REUSE_WORKLOAD and args.reuse_steps > 0:
        result["prefix_reuse"] = prefix_reuse(args.reuse_steps, 2)
    if args.trace_steps > 0:
        result["reasoning_trace"] = reasoning_trace(args.trace_steps)
    if not args.no_cpu_baseline:
        log("timing the fp64 oracle on the CPU")
        P0 = len(wl.prefix(0))
        if P0 * len(wl.candidates(0)) > 8000:   # one question is minutes of fp64 work
            result["cpu_baseline"] = cpu_baseline_layers(r.path, wl)
        else:
            result["cpu_baseline"] = cpu_baseline(r.path, wl)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
