"""The library's host code (request validation, row layout, decisions,
evaluation, model-file reader) built with AddressSanitizer and
UndefinedBehaviorSanitizer and run over valid and malformed inputs
(tests/host_checks.cpp). CPU only: g++ builds the host sources alone."""
import json
import os
import shutil
import struct
import subprocess

import pytest

import jet_synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_33874_amd", "csrc")


def _write_header(path, header, magic=b"JETMDL01", length=None):
    js = json.dumps(header).encode()
    with open(path, "wb") as f:
        f.write(magic + struct.pack("<Q", len(js) if length is None else length) + js)


def _malformed(valid, d):
    h = jet_synth.read_header(valid)
    out = []

    def variant(name, mutate=None, **kw):
        hh = json.loads(json.dumps(h))
        if mutate:
            mutate(hh)
        p = os.path.join(d, name + ".jetm")
        _write_header(p, hh, **kw)
        out.append(p)

    variant("bad_magic", magic=b"JETMDL02")
    variant("zero_length", length=0)
    variant("length_past_end", length=1 << 20)
    variant("huge_length", length=1 << 40)
    variant("few_layer_types", lambda x: x["layer_types"].pop())
    variant("negative_dim", lambda x: x.update(d_model=-5))
    variant("huge_dim", lambda x: x.update(n_layers=1e300))
    variant("fractional_dim", lambda x: x.update(head_dim=31.5))
    variant("string_dim", lambda x: x.update(vocab="1024"))
    variant("negative_shape", lambda x: x["tensors"][0].update(shape=[-1024, -128]))
    variant("fractional_shape", lambda x: x["tensors"][0].update(shape=[1024.5, 128]))
    variant("overflow_shape", lambda x: x["tensors"][0].update(shape=[2 ** 40, 2 ** 40, 2 ** 40]))
    variant("size_mismatch", lambda x: x["tensors"][1].update(nbytes=x["tensors"][1]["nbytes"] + 4))
    variant("bad_tensor_dtype", lambda x: x["tensors"][1].update(dtype="f8"))
    variant("nan_eps", lambda x: x.update(rms_eps=float("nan")))
    variant("unknown_arch", lambda x: x.update(arch="moe"))
    # unterminated and deeply nested JSON
    for name, js in (("unterminated", b'{"arch": "dense", "dtype'), ("deep", b"[" * 200 + b"]" * 200)):
        p = os.path.join(d, name + ".jetm")
        with open(p, "wb") as f:
            f.write(b"JETMDL01" + struct.pack("<Q", len(js)) + js)
        out.append(p)
    return out


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_code_under_address_and_ub_sanitizers(tmp_path):
    exe = str(tmp_path / "host_checks")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined,float-cast-overflow", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "host_checks.cpp"),
           os.path.join(CSRC, "host.cpp"), os.path.join(CSRC, "model_file.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    valid = jet_synth.ensure_model("tiny_dense_fp32", cache_dir=str(tmp_path))
    bad = _malformed(valid, str(tmp_path))
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe, valid, *bad], capture_output=True, text=True, env=env, timeout=300)
    print(r.stdout, r.stderr)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr
    assert "0 failure(s)" in r.stdout
