"""The C ABI from a plain C program (tests/c/abi_roundtrip.c): no Python
binding and no torch between the caller and the library.

(1) CPU: the program compiles with gcc (-Wall -Wextra -Werror) against
    include/msparse.h and links against the built libmsparse.so.
(2) GPU: it runs estimate -> index count -> index build -> forward ->
    backward on a 4K-token GQA workload and a head-dim-64 batch-2 one.  Its
    estimate sets match the oracle's top-k (Algorithm 1; outside the 1e-4 tie
    band) and the outputs built from the oracle's sets match the oracle's
    dense masked forward and backward (Eq. softmax_gradient, Eq.
    attention_backward) at the usual bars.
"""
import math
import os
import shutil
import subprocess

import numpy as np
import pytest
import torch

from oracle import attn as OA
from oracle import index as OI
from synth import WORKLOADS, make_inputs
from tests.helpers import assert_close, assert_lse_close, assert_topk_match, inputs_f64, oracle_indices

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c", "abi_roundtrip.c")
PKG = os.path.join(ROOT, "paper_2510_18830_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def _compile(out_dir: str) -> str:
    if shutil.which("gcc") is None:
        pytest.skip("gcc not installed")
    if not os.path.exists(os.path.join(PKG, "libmsparse.so")):
        pytest.skip("libmsparse.so not built")
    exe = os.path.join(out_dir, "abi_roundtrip")
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"), SRC,
           "-L", PKG, "-lmsparse", "-L", os.path.join(ROCM, "lib"), "-lamdhip64", f"-Wl,-rpath,{PKG}", "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def test_c_caller_compiles_and_links(tmp_path):
    exe = _compile(str(tmp_path))
    assert os.access(exe, os.X_OK)


def _bits(t: torch.Tensor) -> bytes:
    return t.contiguous().view(torch.int16).numpy().tobytes()


@pytest.mark.gpu
@pytest.mark.parametrize("name,wl", [
    ("gqa_4k_d128", WORKLOADS["layer_32k"].resized(seq=4096, heads_q=4, heads_kv=2, k_v=100, k_s=600)),
    ("b2_3k_d64", WORKLOADS["layer_32k"].resized(batch=2, seq=3072, heads_q=2, heads_kv=1, head_dim=64, k_v=70,
                                                 k_s=130)),
])
def test_c_caller_against_oracle(tmp_path, name, wl):
    print(f"C ABI round trip {name} {wl}", flush=True)
    exe = _compile(str(tmp_path))
    x = make_inputs(wl, "cpu")
    f = inputs_f64(x)
    vi, si, vs, ss = oracle_indices(f, wl)
    B, Hq, Hkv, N, d = wl.batch, wl.heads_q, wl.heads_kv, wl.seq, wl.head_dim
    hdr = np.array([B, N, Hq, Hkv, d, wl.last_q, wl.k_v, wl.k_s], np.int32)
    fin, fout = tmp_path / "in.bin", tmp_path / "out.bin"
    with open(fin, "wb") as fh:
        fh.write(hdr.tobytes())
        for n in ("q", "k", "v", "do"):
            fh.write(_bits(x[n]))
        fh.write(np.ascontiguousarray(vi, np.int32).tobytes())
        fh.write(np.ascontiguousarray(si, np.int32).tobytes())
    r = subprocess.run([exe, str(fin), str(fout)], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, r.stderr

    raw = open(fout, "rb").read()
    pos = 0

    def take(dtype, shape):
        nonlocal pos
        n = int(np.prod(shape)) * np.dtype(dtype).itemsize
        a = np.frombuffer(raw[pos:pos + n], dtype=dtype).reshape(shape)
        pos += n
        return a

    ev = take(np.int32, (B, Hq, wl.k_v))
    es = take(np.int32, (B, Hq, wl.k_s))
    out = take(np.uint16, (B, Hq, N, d))
    lse = take(np.float32, (B, Hq, N))
    dq = take(np.float32, (B, Hq, N, d))
    dk = take(np.float32, (B, Hkv, N, d))
    dv = take(np.float32, (B, Hkv, N, d))
    assert pos == len(raw)
    for b in range(B):
        for h in range(Hq):
            assert_topk_match(ev[b, h], vi[b, h], vs[b, h], wl.k_v)
            assert_topk_match(es[b, h], si[b, h], ss[b, h], wl.k_s)
    scale = 1 / math.sqrt(d)
    ref = OI.Index(vi, si, N)
    ro, rl = OA.layer_fwd(f["q"], f["k"], f["v"], ref, scale)
    rq, rk, rv = OA.layer_bwd(f["q"], f["k"], f["v"], f["do"], ref, scale)
    out32 = (out.astype(np.uint32) << 16).view(np.float32)   # bf16 bits -> fp32
    assert_close("out", out32, ro)
    assert_lse_close(lse, rl)
    for n, g, rr in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv)):
        assert_close(n, g, rr)
