"""Full-tensor parity at the 32K layer's shape.

(1) The 32K layer (16 query / 2 KV heads, GQA 8, N 32768, d 128, k_v 1000,
    k_s 6096) with every head's own sets from the fp64 estimator: the GPU runs
    index -> forward -> backward over all heads, and the oracle's dense masked
    forward and backward (Eq. softmax_gradient, Eq. attention_backward) give
    out, lse and dQ of the eight heads of KV group 0 and that group's dK and dV
    over every key, compared element by element.
(2) The same layer with a vertical budget of k_v 16384, which makes the
    column pass's work list split each chunk's query blocks into items of more
    than the minimum span: the span the kernel planned is read back from the
    workspace and checked against the plan recomputed here from the index,
    then KV group 0 is compared in full as in (1).  (With 4 query heads per KV
    head, k_v 8192 and k_s 1024 the generator's planted sink keys reach |dK|
    of about 15 over some 50K rows, and the fp16 rounding of dZ in the selected
    tiles, together with Delta taken from the forward's output, puts their dK
    error at 2.1e-2: a CPU emulation of exactly that rounding gives the same
    figure, so that case measures the precision of the fp16 second GEMM, not
    the column plan.  At head dim 64 the same layer gives span 55 and dK
    2.14e-2, by the same mechanism: the larger logit scale 1/8 concentrates
    more weight on the planted sink keys.)

The oracle runs one head per worker process (about 25 s per head on one core
pair), so each test takes about a minute of CPU time on the GPU host.
"""
import math

import numpy as np
import pytest
import torch

import paper_2510_18830_amd as ms
from synth import WORKLOADS, make_inputs
from tests.helpers import (assert_close, assert_lse_close, gpu_csr, inputs_f64, oracle_heads, oracle_indices,
                           weighted_identity_check)

pytestmark = pytest.mark.gpu

COL_ITEMS = 2048       # item budget of the column pass's plan
COL_MIN_SPAN = 16      # smallest span it uses


def _run_gpu(gpu, wl, x, vi, si, bwd_workspace=None):
    dims = ms.make_dims(wl.batch, wl.seq, wl.heads_q, wl.heads_kv, wl.head_dim)
    q, k, v, do = (x[n].to(gpu) for n in ("q", "k", "v", "do"))
    idx = ms.make_index(dims, torch.from_numpy(vi).to(gpu), torch.from_numpy(si).to(gpu))
    out32 = torch.empty(q.shape, dtype=torch.float32, device=gpu)
    out, lse = ms.attn_fwd(dims, q, k, v, idx, out_f32=out32)
    ws = bwd_workspace(dims, idx) if bwd_workspace else None
    dq, dk, dv = ms.attn_bwd(dims, q, k, v, out, do, lse, idx, out_f32=out32, workspace=ws)
    torch.cuda.synchronize()
    got = dict(out=out.float().cpu().numpy(), out32=out32.cpu().numpy(), lse=lse.cpu().numpy(),
               dq=dq.cpu().numpy(), dk=dk.cpu().numpy(), dv=dv.cpu().numpy())
    return got, idx, ws


def _identities(x, got):
    t = {n: torch.from_numpy(got[n]) for n in ("out32", "dq", "dk", "dv")}
    weighted_identity_check(x, t["out32"], t["dq"], t["dk"], t["dv"], 1e-5)


def _compare_group(got, ref, group, G):
    heads = range(group * G, (group + 1) * G)
    rk = sum(ref[h][3] for h in heads)
    rv = sum(ref[h][4] for h in heads)
    for h in heads:
        ro, rl, rq = ref[h][0], ref[h][1], ref[h][2]
        assert_close(f"out h{h}", got["out"][0, h], ro)
        assert_close(f"out32 h{h}", got["out32"][0, h], ro)
        assert_lse_close(got["lse"][0, h], rl)
        assert_close(f"dq h{h}", got["dq"][0, h], rq)
    for n, g, r in (("dk", got["dk"][0, group], rk), ("dv", got["dv"][0, group], rv)):
        e = np.abs(g - r)
        print(f"{n} kv{group}: max-abs {e.max():.3e} mean-abs {e.mean():.3e}", flush=True)
        assert_close(f"{n} kv{group}", g, r)


@pytest.mark.timeout(900)
def test_layer_32k_full_kv_group(gpu):
    wl = WORKLOADS["layer_32k"]
    print(f"32K full group {wl}", flush=True)
    x = make_inputs(wl, "cpu")
    f = inputs_f64(x)
    vi, si, _, _ = oracle_indices(f, wl)         # each head's own sets
    got, _, _ = _run_gpu(gpu, wl, x, vi, si)
    print("gpu done; oracle over the 8 heads of KV group 0", flush=True)
    G = wl.heads_q // wl.heads_kv
    _identities(x, got)
    ref = oracle_heads(f, vi, si, list(range(G)), 1 / math.sqrt(wl.head_dim))
    _compare_group(got, ref, 0, G)


def _bwd_offsets(dims, vcol_cap):
    """Byte offsets of the backward workspace's parts (256-byte aligned bump
    allocation in the library's order), for reading back the column plan."""
    B, Hq, Hkv, Nq, Nk, d = dims.batch, dims.heads_q, dims.heads_kv, dims.seq_q, dims.seq_k, dims.head_dim
    bh = B * Hq
    chunk_cap = (vcol_cap + 63) // 64 + bh
    parts = [("k16", B * Hkv * Nk * d * 2), ("v16", B * Hkv * Nk * d * 2), ("q16", bh * Nq * d * 2),
             ("g16", bh * Nq * d * 2), ("draw", bh * Nq * 4), ("delta", bh * Nq * 4), ("lse2", bh * Nq * 4),
             ("maxw", 16), ("choff", (bh + 1) * 4), ("e0", chunk_cap * 8), ("head", chunk_cap * 4),
             ("qlo", chunk_cap * 4), ("item", (chunk_cap + 1) * 4), ("span", 4)]
    off, out = 0, {}
    for name, size in parts:
        out[name] = off
        off = (off + size + 255) // 256 * 256
    return out, chunk_cap


def _diag_run(words) -> int:
    """Length of the run of set bits from bit 0 of a bitset (uint32 words)."""
    run = 0
    for w in words:
        w = int(w)
        if w == 0xFFFFFFFF:
            run += 32
            continue
        while w & 1:
            run += 1
            w >>= 1
        break
    return run


def _planned_span(csr, nqb, bh, chunk_cap):
    """The column pass's plan recomputed from the index: chunks of 64 entries of
    each head's vertical list, each seen by the query blocks from the first
    whose global block reaches the chunk's first column block plus the head's
    run of selected block-diagonals from 0 (every nearer query block covers
    the chunk's columns with selected blocks); span = max(16, ceil(candidates
    / budget))."""
    total = 0
    vp, vi = csr["vcol_ptr"], csr["vcol_idx"]
    qg = csr["q_blk_global"]
    db = csr["diag_bits"].reshape(bh, -1)
    for h in range(bh):
        run = _diag_run(db[h])
        for e0 in range(int(vp[h]), int(vp[h + 1]), 64):
            cg = int(csr["k_blk_global"][int(vi[e0]) >> 6])
            lo = int(np.searchsorted(qg, cg + run, side="left"))
            total += nqb - lo
    fine = chunk_cap * ((nqb + COL_MIN_SPAN - 1) // COL_MIN_SPAN)
    budget = min(COL_ITEMS, fine)
    return max(COL_MIN_SPAN, -(-total // budget))


@pytest.mark.timeout(900)
def test_column_pass_split_regime_full_tensors(gpu):
    wl = WORKLOADS["layer_32k"].resized(k_v=16384)
    print(f"column-pass regime {wl}", flush=True)
    x = make_inputs(wl, "cpu")
    f = inputs_f64(x)
    vi, si, _, _ = oracle_indices(f, wl)
    holder = {}

    def workspace(dims, idx):
        vcap = idx.struct.vcol_cap
        holder["dims"], holder["vcap"] = dims, vcap
        return ms._workspace(ms.attn_bwd_workspace_bytes(dims, vcap), gpu)

    got, idx, ws = _run_gpu(gpu, wl, x, vi, si, workspace)
    offs, chunk_cap = _bwd_offsets(holder["dims"], holder["vcap"])
    span_gpu = int(ws[offs["span"]:offs["span"] + 4].cpu().numpy().view(np.int32)[0])
    span_ref = _planned_span(gpu_csr(idx), wl.seq // 64, wl.batch * wl.heads_q, chunk_cap)
    print(f"column span: planned {span_gpu}, recomputed {span_ref}", flush=True)
    assert span_gpu == span_ref
    assert span_gpu > COL_MIN_SPAN
    G = wl.heads_q // wl.heads_kv
    ref = oracle_heads(f, vi, si, list(range(G)), 1 / math.sqrt(wl.head_dim))
    _compare_group(got, ref, 0, G)
