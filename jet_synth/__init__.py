"""Seeded synthetic inputs for candidate scoring: model files and workloads.

This module is the one piece shared by the fp64 oracle and the GPU path. It
holds no arithmetic of the scoring method: it draws random numbers, rounds
them to the storage dtype, writes/reads the model file format, and builds the
CSR arrays that describe questions and candidates.

Model file format (little endian)::

    bytes 0..7    magic  b"JETMDL01"
    bytes 8..15   uint64 length H of the JSON header
    bytes 16..    JSON header (utf-8), then zero padding
    tensors       each at a 4096-byte aligned absolute offset given in the header

Header keys: ``arch`` ("dense" | "hybrid"), ``dtype`` ("bf16" | "f32", the
storage type of every matrix), ``d_model``, ``n_layers``, ``n_heads``,
``n_kv_heads``, ``head_dim``, ``ffn``, ``vocab``, ``rms_eps``, ``rope_theta``,
``layer_types`` (list of "attn" | "gdn"), ``gdn_heads``, ``gdn_dk``, ``gdn_dv``,
``conv_kernel``, ``n_experts`` (0: dense SwiGLU FFN; else every FFN is a
mixture of experts), ``top_k``, ``moe_ffn``, ``shared_ffn`` (0: no shared
expert), ``max_ctx``, ``seed``, ``init_std``, ``zero``, and ``tensors``:
a list of ``{name, dtype, shape, offset, nbytes}``. Matrices use the
``[out_features, in_features]`` convention. Norm gains, ``A_log`` and
``dt_bias`` are stored as f32 whatever the matrix dtype is.

Block-quantized models (``dtype`` "q8"): every matrix whose last dimension
is a multiple of 32 is stored as int8 values q [rows][cols] followed by one
int8 exponent per block of 32 consecutive values of a row, e [rows][cols/32];
the weight is q * 2^e (|q| <= 127). The exponent of a block is the smallest e
with max|w| <= 127 * 2^e over the block's values w, and q = rint(w / 2^e).
Other tensors keep bf16 (matrices) or f32 (norm gains, A_log, dt_bias).
``dtype`` "q4" is the same with 4-bit values: q in -8..7 (two's complement),
two per byte, value 2i of a row in the low nibble of byte i, then the int8
block exponents; the exponent of a block is the smallest e with
max|w| <= 7 * 2^e.

Random numbers: every tensor is split into fixed chunks of ``CHUNK`` elements;
chunk ``j`` of tensor ``name`` is drawn from a Philox-4x64 counter-based
stream keyed on ``(seed, crc32(name) << 32 | j)`` as standard normals in
float32, scaled by ``init_std`` in float32 and rounded to nearest-even into
bfloat16 (or kept as float32). The result therefore does not depend on the
number of threads used to write the file.
"""
from __future__ import annotations

import json
import os
import shutil
import struct
import sys
import time
import zlib
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np

MAGIC = b"JETMDL01"
QBLOCK = 32  # values per quantization block of a "q8" / "q4" matrix
ALIGN = 4096
CHUNK = 1 << 22
# Sampling seed of the paper's experimental protocol (Appendix A); reused here
# as the master seed of every synthetic input.
MASTER_SEED = 20260921

# --------------------------------------------------------------------------
# model shapes
# --------------------------------------------------------------------------

MODEL_SPECS: dict[str, dict] = {
    # 2 layers, d=128, 4 heads of 32 (MHA), SwiGLU 512, vocab 1024, fp32.
    "tiny_dense_fp32": dict(arch="dense", dtype="f32", d_model=128, n_layers=2,
                            n_heads=4, n_kv_heads=4, head_dim=32, ffn=512,
                            vocab=1024, max_ctx=4096),
    # Same shape stored in bf16 (used for bf16-path parity at tiny size).
    "tiny_dense_bf16": dict(arch="dense", dtype="bf16", d_model=128, n_layers=2,
                            n_heads=4, n_kv_heads=4, head_dim=32, ffn=512,
                            vocab=1024, max_ctx=4096),
    # Small GQA model with the production head size (hd=128), bf16.
    "small_gqa_bf16": dict(arch="dense", dtype="bf16", d_model=256, n_layers=2,
                           n_heads=6, n_kv_heads=2, head_dim=128, ffn=768,
                           vocab=3000, max_ctx=8192),
    "small_gqa_fp32": dict(arch="dense", dtype="f32", d_model=256, n_layers=2,
                           n_heads=6, n_kv_heads=2, head_dim=128, ffn=768,
                           vocab=3000, max_ctx=8192),
    # 1.5B-shape dense decoder: 28 layers, d=1536, GQA 12/2 (hd 128), FFN 8960.
    "dense_1p5b": dict(arch="dense", dtype="bf16", d_model=1536, n_layers=28,
                       n_heads=12, n_kv_heads=2, head_dim=128, ffn=8960,
                       vocab=151936, max_ctx=8192),
    # 27B-shape dense decoder: 64 layers, d=5120, GQA 40/8 (hd 128), FFN 17408.
    "dense_27b": dict(arch="dense", dtype="bf16", d_model=5120, n_layers=64,
                      n_heads=40, n_kv_heads=8, head_dim=128, ffn=17408,
                      vocab=151936, max_ctx=8192),
    # 4B-shape hybrid: 8 x [3 gated delta-rule layers + 1 GQA attention layer].
    "hybrid_4b": dict(arch="hybrid", dtype="bf16", d_model=2560, n_layers=32,
                      n_heads=16, n_kv_heads=4, head_dim=128, ffn=9728,
                      vocab=151936, gdn_heads=16, gdn_dk=128, gdn_dv=128,
                      conv_kernel=4, max_ctx=8192),
    # Small hybrid with production head sizes (for GPU parity at small size).
    "small_hybrid_bf16": dict(arch="hybrid", dtype="bf16", d_model=256, n_layers=4,
                              n_heads=2, n_kv_heads=1, head_dim=128, ffn=512,
                              vocab=2048, gdn_heads=2, gdn_dk=128, gdn_dv=128,
                              conv_kernel=4, max_ctx=8192),
    "small_hybrid_fp32": dict(arch="hybrid", dtype="f32", d_model=256, n_layers=4,
                              n_heads=2, n_kv_heads=1, head_dim=128, ffn=512,
                              vocab=2048, gdn_heads=2, gdn_dk=128, gdn_dv=128,
                              conv_kernel=4, max_ctx=8192),
    # Small mixture-of-experts hybrid (3 delta-rule + 1 attention layer, every
    # FFN 8 routed experts of 128, top 2, plus a gated shared expert of 128).
    "small_moe_bf16": dict(arch="hybrid", dtype="bf16", d_model=256, n_layers=4,
                           n_heads=2, n_kv_heads=1, head_dim=128, ffn=128,
                           vocab=2048, gdn_heads=2, gdn_dk=128, gdn_dv=128,
                           conv_kernel=4, n_experts=8, top_k=2, moe_ffn=128,
                           shared_ffn=128, max_ctx=8192),
    "small_moe_fp32": dict(arch="hybrid", dtype="f32", d_model=256, n_layers=4,
                           n_heads=2, n_kv_heads=1, head_dim=128, ffn=128,
                           vocab=2048, gdn_heads=2, gdn_dk=128, gdn_dv=128,
                           conv_kernel=4, n_experts=8, top_k=2, moe_ffn=128,
                           shared_ffn=128, max_ctx=8192),
    # Two-layer dense decoder with mixture-of-experts FFNs (for the
    # single-bf16 mode, whose rounding grows with depth).
    "tiny_moe_bf16": dict(arch="dense", dtype="bf16", d_model=256, n_layers=2,
                          n_heads=2, n_kv_heads=1, head_dim=128, ffn=128,
                          vocab=2048, n_experts=8, top_k=2, moe_ffn=128,
                          shared_ffn=128, max_ctx=8192),
    # 35B-A3B-shape mixture-of-experts hybrid: 10 x [3 delta-rule + 1 GQA
    # attention layer], d=2048, every FFN 256 routed experts of 512 (top 8)
    # plus a gated shared expert of 512: 33.7B parameters, 2.5B active per token.
    "moe_35b_a3b": dict(arch="hybrid", dtype="bf16", d_model=2048, n_layers=40,
                        n_heads=16, n_kv_heads=2, head_dim=128, ffn=512,
                        vocab=151936, gdn_heads=16, gdn_dk=128, gdn_dv=128,
                        conv_kernel=4, n_experts=256, top_k=8, moe_ffn=512,
                        shared_ffn=512, max_ctx=8192),
    # Micro mixture of experts for oracle self-checks on the CPU.
    "micro_moe_fp32": dict(arch="dense", dtype="f32", d_model=64, n_layers=2,
                           n_heads=4, n_kv_heads=2, head_dim=16, ffn=32,
                           vocab=512, n_experts=4, top_k=2, moe_ffn=32,
                           shared_ffn=32, max_ctx=4096),
    # Block-quantized (int8 blocks of 32 with power-of-two scales) dense
    # decoders: the small GQA shape, the 1.5B and the 27B shapes.
    "small_gqa_q8": dict(arch="dense", dtype="q8", d_model=256, n_layers=2,
                         n_heads=6, n_kv_heads=2, head_dim=128, ffn=768,
                         vocab=3000, max_ctx=8192),
    "small_gqa_q4": dict(arch="dense", dtype="q4", d_model=256, n_layers=2,
                         n_heads=6, n_kv_heads=2, head_dim=128, ffn=768,
                         vocab=3000, max_ctx=8192),
    "dense_1p5b_q8": dict(arch="dense", dtype="q8", d_model=1536, n_layers=28,
                          n_heads=12, n_kv_heads=2, head_dim=128, ffn=8960,
                          vocab=151936, max_ctx=8192),
    "dense_1p5b_q4": dict(arch="dense", dtype="q4", d_model=1536, n_layers=28,
                          n_heads=12, n_kv_heads=2, head_dim=128, ffn=8960,
                          vocab=151936, max_ctx=8192),
    "dense_27b_q8": dict(arch="dense", dtype="q8", d_model=5120, n_layers=64,
                         n_heads=40, n_kv_heads=8, head_dim=128, ffn=17408,
                         vocab=151936, max_ctx=8192),
    # Micro quantized decoder for oracle self-checks on the CPU.
    "micro_q8": dict(arch="dense", dtype="q8", d_model=64, n_layers=2,
                     n_heads=4, n_kv_heads=2, head_dim=16, ffn=128,
                     vocab=512, max_ctx=4096),
    "micro_q4": dict(arch="dense", dtype="q4", d_model=64, n_layers=2,
                     n_heads=4, n_kv_heads=2, head_dim=16, ffn=128,
                     vocab=512, max_ctx=4096),
    # Micro hybrid for oracle self-checks on the CPU: L=4, d=64.
    "micro_hybrid_fp32": dict(arch="hybrid", dtype="f32", d_model=64, n_layers=4,
                              n_heads=4, n_kv_heads=2, head_dim=16, ffn=128,
                              vocab=512, gdn_heads=2, gdn_dk=16, gdn_dv=16,
                              conv_kernel=4, max_ctx=4096),
}

DEFAULTS = dict(rms_eps=1e-6, rope_theta=1.0e6, init_std=0.02, n_experts=0, top_k=0,
                moe_ffn=0, shared_ffn=0)


def full_spec(spec: dict | str) -> dict:
    s = dict(MODEL_SPECS[spec]) if isinstance(spec, str) else dict(spec)
    for k, v in DEFAULTS.items():
        s.setdefault(k, v)
    if s["arch"] == "hybrid":
        s.setdefault("layer_types", ["gdn", "gdn", "gdn", "attn"] * (s["n_layers"] // 4))
    else:
        s.setdefault("layer_types", ["attn"] * s["n_layers"])
    assert len(s["layer_types"]) == s["n_layers"]
    return s


def tensor_list(spec: dict) -> list[tuple[str, str, tuple, str]]:
    """(name, storage dtype, shape, init) for every tensor, in file order.

    init is "normal" (i.i.d. N(0, init_std^2)), "ones", "zeros" or
    "const:<value>".
    """
    s = full_spec(spec)
    d, V, F = s["d_model"], s["vocab"], s["ffn"]
    q8 = s["dtype"] in ("q8", "q4")
    out = []

    def mat(name, shape, init="normal"):
        dt = (s["dtype"] if shape[-1] % QBLOCK == 0 else "bf16") if q8 else s["dtype"]
        out.append((name, dt, tuple(shape), init))

    mt = "bf16" if q8 else s["dtype"]
    mat("tok_embed", (V, d))
    for i, lt in enumerate(s["layer_types"]):
        p = f"blk.{i}."
        out.append((p + "attn_norm", "f32", (d,), "ones"))
        if lt == "attn":
            hq, hkv, hd = s["n_heads"], s["n_kv_heads"], s["head_dim"]
            mat(p + "wq", (hq * hd, d))
            mat(p + "wk", (hkv * hd, d))
            mat(p + "wv", (hkv * hd, d))
            mat(p + "wo", (d, hq * hd))
        else:
            H, dk, dv, kc = s["gdn_heads"], s["gdn_dk"], s["gdn_dv"], s["conv_kernel"]
            mat(p + "gdn_wq", (H * dk, d))
            mat(p + "gdn_wk", (H * dk, d))
            mat(p + "gdn_wv", (H * dv, d))
            mat(p + "gdn_wz", (H * dv, d))
            mat(p + "gdn_wb", (H, d))
            mat(p + "gdn_wa", (H, d))
            out.append((p + "gdn_conv", mt, (2 * H * dk + H * dv, kc), "normal"))
            a_log = float(s.get("gdn_a_log", 0.0))  # optional constant (decay strength)
            out += [(p + "gdn_A_log", "f32", (H,), f"const:{a_log!r}" if a_log else "zeros"),
                    (p + "gdn_dt_bias", "f32", (H,), "zeros"),
                    (p + "gdn_norm", "f32", (dv,), "ones")]
            mat(p + "gdn_wo", (d, H * dv))
        out.append((p + "ffn_norm", "f32", (d,), "ones"))
        if s["n_experts"] == 0:
            mat(p + "w_gate", (F, d))
            mat(p + "w_up", (F, d))
            mat(p + "w_down", (d, F))
        else:
            E, Fe, Fs = s["n_experts"], s["moe_ffn"], s["shared_ffn"]
            mat(p + "moe_router", (E, d))
            mat(p + "moe_gate", (E, Fe, d))
            mat(p + "moe_up", (E, Fe, d))
            mat(p + "moe_down", (E, d, Fe))
            if Fs:
                mat(p + "shared_router", (1, d))
                mat(p + "shared_gate", (Fs, d))
                mat(p + "shared_up", (Fs, d))
                mat(p + "shared_down", (d, Fs))
    out.append(("final_norm", "f32", (d,), "ones"))
    mat("lm_head", (V, d))
    return out


def n_params(spec) -> int:
    return int(sum(np.prod(sh) for _, _, sh, _ in tensor_list(spec)))


# --------------------------------------------------------------------------
# writing / reading model files
# --------------------------------------------------------------------------

def _f32_to_bf16_rne(x: np.ndarray, out: np.ndarray) -> None:
    """Round float32 to bfloat16 bits (round to nearest, ties to even)."""
    u = x.view(np.uint32)
    t = u >> 16
    t &= 1
    t += 0x7FFF
    t += u
    t >>= 16
    out[:] = t


def quantize_q8(val: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """Blocks of QBLOCK float32 values -> (int8 q, int8 exponent per block):
    the smallest e with max|w| <= 127 * 2^e, q = rint(w / 2^e)."""
    blocks = np.asarray(val, np.float32).reshape(-1, QBLOCK)
    amax = np.abs(blocks).max(axis=1).astype(np.float64)
    m, x = np.frexp(amax / 127.0)          # amax / 127 = m 2^x, m in [0.5, 1)
    e = np.where(m == 0.5, x - 1, x)       # ceil(log2(amax / 127))
    e = np.where(amax > 0, e, 0).clip(-126, 126).astype(np.int32)
    scale = np.ldexp(np.float32(1.0), -e).astype(np.float32)[:, None]
    q = np.rint(blocks * scale).clip(-127, 127).astype(np.int8)   # exact power-of-two scaling
    return q.reshape(-1), e.astype(np.int8)


def quantize_q4(val: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """Blocks of QBLOCK float32 values -> (packed int4 bytes, int8 exponent
    per block): the smallest e with max|w| <= 7 * 2^e, q = rint(w / 2^e),
    value 2i in the low nibble of byte i."""
    blocks = np.asarray(val, np.float32).reshape(-1, QBLOCK)
    amax = np.abs(blocks).max(axis=1).astype(np.float64)
    m, x = np.frexp(amax / 7.0)
    e = np.where(m == 0.5, x - 1, x)       # ceil(log2(amax / 7))
    e = np.where(amax > 0, e, 0).clip(-126, 126).astype(np.int32)
    scale = np.ldexp(np.float32(1.0), -e).astype(np.float32)[:, None]
    q = np.rint(blocks * scale).clip(-8, 7).astype(np.int8).reshape(-1)
    u = (q.astype(np.uint8) & np.uint8(0x0F))
    packed = (u[0::2] | (u[1::2] << np.uint8(4))).astype(np.uint8)
    return packed, e.astype(np.int8)


def unpack_q4(packed: np.ndarray) -> np.ndarray:
    """Packed int4 bytes [..., n / 2] -> int8 values [..., n]."""
    b = np.asarray(packed, np.uint8)
    lo = (b & np.uint8(0x0F)).astype(np.int8)
    hi = (b >> np.uint8(4)).astype(np.int8)
    lo = np.where(lo > 7, lo - 16, lo).astype(np.int8)
    hi = np.where(hi > 7, hi - 16, hi).astype(np.int8)
    out = np.empty(b.shape[:-1] + (2 * b.shape[-1],), np.int8)
    out[..., 0::2] = lo
    out[..., 1::2] = hi
    return out


class Q4Raw:
    """Stored packed int4 values and per-block exponents of a "q4" tensor
    (rows indexable like the tensor itself, the last dimension whole)."""

    def __init__(self, p: np.ndarray, e: np.ndarray):
        self.p, self.e = p, e

    @property
    def shape(self):
        return self.p.shape[:-1] + (2 * self.p.shape[-1],)

    @property
    def q(self):
        return unpack_q4(self.p)

    def __getitem__(self, idx):
        return Q4Raw(self.p[idx], self.e[idx])


class Q8Raw:
    """Stored int8 values and per-block exponents of a "q8" tensor (rows
    indexable like the tensor itself, the last dimension whole)."""

    def __init__(self, q: np.ndarray, e: np.ndarray):
        self.q, self.e = q, e

    @property
    def shape(self):
        return self.q.shape

    def __getitem__(self, idx):
        return Q8Raw(self.q[idx], self.e[idx])


def _fill_chunk(seed: int, name: str, j: int, std: float, init: str,
                dst, dtype: str, zero: bool) -> None:
    if dtype == "q8":
        dq, de = dst
        val = np.empty(dq.size, np.float32)
        _fill_chunk(seed, name, j, std, init, val, "f32", zero)
        dq[:], de[:] = quantize_q8(val)
        return
    if dtype == "q4":
        dp, de = dst
        val = np.empty(2 * dp.size, np.float32)
        _fill_chunk(seed, name, j, std, init, val, "f32", zero)
        dp[:], de[:] = quantize_q4(val)
        return
    n = dst.size
    if init == "ones":
        val = np.ones(n, np.float32)
    elif init == "zeros" or zero:
        val = np.zeros(n, np.float32)
    elif init.startswith("const:"):
        val = np.full(n, float(init[6:]), np.float32)
    else:
        key = (zlib.crc32(name.encode()) << 32) | j
        g = np.random.Generator(np.random.Philox(key=[seed, key]))
        val = np.empty(n, np.float32)
        g.standard_normal(out=val, dtype=np.float32)
        val *= np.float32(std)
    if dtype == "bf16":
        _f32_to_bf16_rne(val, dst)
    else:
        dst[:] = val


def _np_storage(dtype: str):
    return np.uint16 if dtype == "bf16" else np.int8 if dtype == "q8" else np.float32


def tensor_nbytes(dtype: str, shape) -> int:
    n = int(np.prod(shape))
    if dtype == "q8":
        return n + n // QBLOCK
    if dtype == "q4":
        return n // 2 + n // QBLOCK
    return n * (2 if dtype == "bf16" else 4)


def write_model(path: str, spec: dict | str, seed: int = MASTER_SEED,
                zero: bool = False, threads: int | None = None) -> dict:
    """Write a seeded synthetic model file; returns its header."""
    s = full_spec(spec)
    tensors = []
    # header is written last; reserve generous room for it
    hdr_room = 1 << 20
    off = ALIGN * ((16 + hdr_room + ALIGN - 1) // ALIGN)
    for name, dt, shape, init in tensor_list(s):
        nbytes = tensor_nbytes(dt, shape)
        tensors.append(dict(name=name, dtype=dt, shape=list(shape), offset=off,
                            nbytes=nbytes, init=init))
        off += ALIGN * ((nbytes + ALIGN - 1) // ALIGN)
    header = dict(format=1, **{k: v for k, v in s.items()}, seed=int(seed), zero=bool(zero),
                  tensors=[{k: t[k] for k in ("name", "dtype", "shape", "offset", "nbytes")}
                           for t in tensors])
    hjson = json.dumps(header).encode()
    assert len(hjson) <= hdr_room
    free = shutil.disk_usage(os.path.dirname(os.path.abspath(path))).free
    if free < off + (1 << 30):
        # a memory-mapped write past the end of the disk would end the process with SIGBUS
        raise OSError(f"{path}: {off / 2**30:.1f} GiB needed, {free / 2**30:.1f} GiB free")
    tmp = path + ".tmp"
    with open(tmp, "wb") as f:
        f.truncate(off)
        f.seek(0)
        f.write(MAGIC + struct.pack("<Q", len(hjson)) + hjson)
    mm = np.memmap(tmp, dtype=np.uint8, mode="r+")
    jobs = []
    for t in tensors:
        if t["dtype"] == "q8":
            n = int(np.prod(t["shape"]))
            q = mm[t["offset"]:t["offset"] + n].view(np.int8)
            e = mm[t["offset"] + n:t["offset"] + t["nbytes"]].view(np.int8)
            for j in range(0, (n + CHUNK - 1) // CHUNK):
                jobs.append((t["name"], j, t["init"], (q[j * CHUNK:(j + 1) * CHUNK],
                                                       e[j * CHUNK // QBLOCK:(j + 1) * CHUNK // QBLOCK]), "q8"))
            continue
        if t["dtype"] == "q4":
            n = int(np.prod(t["shape"]))
            pk = mm[t["offset"]:t["offset"] + n // 2]
            e = mm[t["offset"] + n // 2:t["offset"] + t["nbytes"]].view(np.int8)
            for j in range(0, (n + CHUNK - 1) // CHUNK):
                jobs.append((t["name"], j, t["init"], (pk[j * CHUNK // 2:(j + 1) * CHUNK // 2],
                                                       e[j * CHUNK // QBLOCK:(j + 1) * CHUNK // QBLOCK]), "q4"))
            continue
        n = t["nbytes"] // (2 if t["dtype"] == "bf16" else 4)
        arr = mm[t["offset"]:t["offset"] + t["nbytes"]].view(_np_storage(t["dtype"]))
        for j in range(0, (n + CHUNK - 1) // CHUNK):
            jobs.append((t["name"], j, t["init"], arr[j * CHUNK:(j + 1) * CHUNK], t["dtype"]))
    nthr = threads or max(1, min(32, len(os.sched_getaffinity(0))))
    std = s["init_std"]
    # large files take minutes: report the chunks written about every 20 s on
    # the process's own stderr (a test runner capturing output would hold it)
    total, t_last = len(jobs), time.monotonic()
    with ThreadPoolExecutor(nthr) as ex:
        for i, _ in enumerate(ex.map(lambda a: _fill_chunk(seed, a[0], a[1], std, a[2], a[3], a[4], zero), jobs)):
            if time.monotonic() - t_last > 20:
                t_last = time.monotonic()
                print(f"[jet_synth] {os.path.basename(path)}: {i + 1}/{total} chunks written", file=sys.__stderr__,
                      flush=True)
    mm.flush()
    del mm
    os.replace(tmp, path)
    return header


def read_header(path: str) -> dict:
    with open(path, "rb") as f:
        head = f.read(16)
        if head[:8] != MAGIC:
            raise ValueError(f"{path}: not a model file")
        (n,) = struct.unpack("<Q", head[8:16])
        return json.loads(f.read(n))


def tensor_raw(path: str, name: str, header: dict | None = None):
    """Memory-mapped raw storage of one tensor: uint16 bf16 bits, float32, or
    for "q8" a Q8Raw of the int8 values and int8 block exponents, for "q4" a
    Q4Raw of the packed int4 values and int8 block exponents."""
    h = header or read_header(path)
    for t in h["tensors"]:
        if t["name"] == name:
            shape = tuple(t["shape"])
            if t["dtype"] == "q8":
                n = int(np.prod(shape))
                q = np.memmap(path, dtype=np.int8, mode="r", offset=t["offset"], shape=shape)
                e = np.memmap(path, dtype=np.int8, mode="r", offset=t["offset"] + n,
                              shape=shape[:-1] + (shape[-1] // QBLOCK,))
                return Q8Raw(q, e)
            if t["dtype"] == "q4":
                n = int(np.prod(shape))
                pk = np.memmap(path, dtype=np.uint8, mode="r", offset=t["offset"],
                               shape=shape[:-1] + (shape[-1] // 2,))
                e = np.memmap(path, dtype=np.int8, mode="r", offset=t["offset"] + n // 2,
                              shape=shape[:-1] + (shape[-1] // QBLOCK,))
                return Q4Raw(pk, e)
            return np.memmap(path, dtype=_np_storage(t["dtype"]), mode="r",
                             offset=t["offset"], shape=shape)
    raise KeyError(name)


def model_cache_dir() -> str:
    d = os.environ.get("JET_MODEL_CACHE") or os.path.join("/tmp", "jet_models")
    os.makedirs(d, exist_ok=True)
    return d


def make_room(path: str, spec: dict | str, min_evict: int = 8 << 30) -> None:
    """While the disk lacks room for `spec`'s file at `path`, deletes the
    largest other cached model files (``*.jetm`` of over `min_evict` bytes in
    the same folder; each is written again from its seed when needed)."""
    import shutil
    need = sum(tensor_nbytes(dt, shape) for _, dt, shape, _ in tensor_list(spec)) + (2 << 30)
    d = os.path.dirname(os.path.abspath(path))
    others = sorted((os.path.join(d, f) for f in os.listdir(d) if f.endswith(".jetm")),
                    key=os.path.getsize, reverse=True)
    for f in others:
        if shutil.disk_usage(d).free >= need:
            break
        if os.path.abspath(f) != os.path.abspath(path) and os.path.getsize(f) > min_evict:
            print(f"[jet_synth] removing cached {os.path.basename(f)} to make room for {os.path.basename(path)}",
                  flush=True)
            os.remove(f)


def ensure_model(spec_name: str, seed: int = MASTER_SEED, zero: bool = False,
                 cache_dir: str | None = None, evict: bool = False) -> str:
    """Path of the model file for a named spec, writing it if absent (with
    evict, after deleting other large cached model files if the disk lacks
    room for it)."""
    d = cache_dir or model_cache_dir()
    path = os.path.join(d, f"{spec_name}_s{seed}{'_zero' if zero else ''}.jetm")
    if not os.path.exists(path):
        if evict:
            make_room(path, spec_name)
        write_model(path, spec_name, seed=seed, zero=zero)
    return path


# --------------------------------------------------------------------------
# workloads
# --------------------------------------------------------------------------

@dataclass
class Workload:
    """Questions and candidates as CSR arrays (the layout the C ABI takes)."""
    prefix_offsets: np.ndarray   # int64 [Q+1]
    prefix_tokens: np.ndarray    # int32 [sum P]
    q_cand_offsets: np.ndarray   # int64 [Q+1]
    cand_tok_offsets: np.ndarray  # int64 [N+1]
    cand_tokens: np.ndarray      # int32 [sum m]

    @property
    def n_questions(self) -> int:
        return len(self.prefix_offsets) - 1

    @property
    def n_candidates(self) -> int:
        return len(self.cand_tok_offsets) - 1

    def prefix(self, q: int) -> np.ndarray:
        return self.prefix_tokens[self.prefix_offsets[q]:self.prefix_offsets[q + 1]]

    def candidates(self, q: int) -> list[np.ndarray]:
        return [self.cand_tokens[self.cand_tok_offsets[c]:self.cand_tok_offsets[c + 1]]
                for c in range(self.q_cand_offsets[q], self.q_cand_offsets[q + 1])]

    def subset(self, qs) -> "Workload":
        """The questions ``qs`` (in that order) with their candidates."""
        pre, cands = [], []
        for q in qs:
            pre.append(self.prefix(q))
            cands.append(self.candidates(q))
        return from_lists(pre, cands)


def from_lists(prefixes: list, cands: list[list]) -> Workload:
    """Build the CSR arrays from per-question prefix and candidate token lists."""
    po = np.zeros(len(prefixes) + 1, np.int64)
    po[1:] = np.cumsum([len(p) for p in prefixes])
    qo = np.zeros(len(cands) + 1, np.int64)
    qo[1:] = np.cumsum([len(c) for c in cands])
    flat = [np.asarray(y, np.int32) for cs in cands for y in cs]
    co = np.zeros(len(flat) + 1, np.int64)
    co[1:] = np.cumsum([len(y) for y in flat])
    pt = np.concatenate([np.asarray(p, np.int32) for p in prefixes]) if prefixes else np.zeros(0, np.int32)
    ct = np.concatenate(flat) if flat else np.zeros(0, np.int32)
    return Workload(po, pt.astype(np.int32), qo, co, ct.astype(np.int32))


# Workload recipes. Lengths are discrete uniform, inclusive. "zipf" ids follow
# P(id = r) proportional to 1/(r+1) over [0, V); "uniform" ids are uniform.
WORKLOADS: dict[str, dict] = {
    "tiny": dict(model="tiny_dense_fp32", Q=16, P=(32, 32), ids="uniform", K=4, m=(1, 4)),
    "small": dict(model="small_gqa_bf16", Q=12, P=(40, 300), ids="zipf", K=4, m=(1, 24)),
    "dense_1p5b_k4": dict(model="dense_1p5b", Q=256, P=(150, 900), ids="zipf", K=4, m=(1, 24)),
    "dense_1p5b_binary": dict(model="dense_1p5b", Q=512, P=(300, 2000), ids="zipf", K=2, m=(1, 1)),
    "dense_1p5b_ordinal": dict(model="dense_1p5b", Q=512, P=(300, 2000), ids="zipf", K=5, m=(1, 3)),
    "hybrid_4b_k4": dict(model="hybrid_4b", Q=128, P=(200, 1500), ids="zipf", K=4, m=(1, 24)),
    "dense_27b_k10": dict(model="dense_27b", Q=64, P=(1024, 4096), ids="zipf", K=10, m=(8, 40)),
    "small_hybrid": dict(model="small_hybrid_bf16", Q=8, P=(20, 200), ids="zipf", K=4, m=(1, 12)),
    "micro_hybrid": dict(model="micro_hybrid_fp32", Q=4, P=(5, 20), ids="uniform", K=3, m=(1, 5)),
    "moe_35b_a3b_k4": dict(model="moe_35b_a3b", Q=128, P=(200, 1500), ids="zipf", K=4, m=(1, 24)),
    "small_moe": dict(model="small_moe_bf16", Q=8, P=(20, 200), ids="zipf", K=4, m=(1, 12)),
    "tiny_moe": dict(model="tiny_moe_bf16", Q=8, P=(20, 200), ids="zipf", K=4, m=(1, 12)),
    # enough prefix rows that the expert segments average over 1024 rows
    "tiny_moe_long": dict(model="tiny_moe_bf16", Q=16, P=(250, 400), ids="zipf", K=4, m=(1, 12)),
    "micro_moe": dict(model="micro_moe_fp32", Q=4, P=(5, 20), ids="uniform", K=3, m=(1, 5)),
    "small_q8": dict(model="small_gqa_q8", Q=12, P=(40, 300), ids="zipf", K=4, m=(1, 24)),
    "dense_1p5b_q8_k4": dict(model="dense_1p5b_q8", Q=256, P=(150, 900), ids="zipf", K=4, m=(1, 24)),
    "small_q4": dict(model="small_gqa_q4", Q=12, P=(40, 300), ids="zipf", K=4, m=(1, 24)),
    "dense_1p5b_q4_k4": dict(model="dense_1p5b_q4", Q=256, P=(150, 900), ids="zipf", K=4, m=(1, 24)),
    "dense_27b_q8_k10": dict(model="dense_27b_q8", Q=64, P=(1024, 4096), ids="zipf", K=10, m=(8, 40)),
}


def _stream(seed: int, label: str) -> np.random.Generator:
    return np.random.Generator(np.random.Philox(key=[seed, zlib.crc32(label.encode())]))


def zipf_ids(g: np.random.Generator, n: int, V: int) -> np.ndarray:
    w = 1.0 / np.arange(1, V + 1, dtype=np.float64)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    u = g.random(n)
    return np.minimum(np.searchsorted(cdf, u, side="right"), V - 1).astype(np.int32)


def make_workload(name: str, seed: int = MASTER_SEED, n_questions: int | None = None,
                  vocab: int | None = None, **over) -> Workload:
    """Generate the seeded workload ``name`` (see WORKLOADS)."""
    r = dict(WORKLOADS[name])
    r.update(over)
    V = vocab or full_spec(r["model"])["vocab"]
    Q = r["Q"] if n_questions is None else n_questions
    g_plen = _stream(seed, name + "/prefix_len")
    g_pid = _stream(seed, name + "/prefix_ids")
    g_mlen = _stream(seed, name + "/cand_len")
    g_cid = _stream(seed, name + "/cand_ids")
    plen = g_plen.integers(r["P"][0], r["P"][1] + 1, size=Q)
    prefixes = []
    for q in range(Q):
        if r["ids"] == "zipf":
            prefixes.append(zipf_ids(g_pid, int(plen[q]), V))
        else:
            prefixes.append(g_pid.integers(0, V, size=int(plen[q])).astype(np.int32))
    cands = []
    for q in range(Q):
        ml = g_mlen.integers(r["m"][0], r["m"][1] + 1, size=r["K"])
        cands.append([g_cid.integers(0, V, size=int(m)).astype(np.int32) for m in ml])
    return from_lists(prefixes, cands)


# --------------------------------------------------------------------------
# digests (to tie stored expected values to the exact inputs they came from)
# --------------------------------------------------------------------------

def tensor_digests(path: str, threads: int | None = None) -> dict[str, str]:
    """sha256 of every tensor's stored bytes, by tensor name."""
    import hashlib
    h = read_header(path)
    mm = np.memmap(path, dtype=np.uint8, mode="r")

    def one(t):
        d = hashlib.sha256()
        a, n = t["offset"], t["nbytes"]
        for o in range(a, a + n, 1 << 26):   # hashlib releases the GIL on large buffers
            d.update(memoryview(mm[o:min(o + (1 << 26), a + n)]))
        return t["name"], d.hexdigest()

    nthr = threads or max(1, min(16, len(os.sched_getaffinity(0))))
    with ThreadPoolExecutor(nthr) as ex:
        return dict(ex.map(one, h["tensors"]))


def workload_digest(wl: Workload) -> str:
    """sha256 over the five CSR arrays of a workload (fixed dtypes, in order)."""
    import hashlib
    d = hashlib.sha256()
    for a, dt in ((wl.prefix_offsets, np.int64), (wl.prefix_tokens, np.int32),
                  (wl.q_cand_offsets, np.int64), (wl.cand_tok_offsets, np.int64),
                  (wl.cand_tokens, np.int32)):
        d.update(np.ascontiguousarray(a, dtype=dt).tobytes())
    return d.hexdigest()
