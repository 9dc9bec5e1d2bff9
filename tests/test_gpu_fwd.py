"""GPU sparse forward vs the fp64 oracle, given the oracle's index."""
import math

import numpy as np
import pytest
import torch

import paper_2510_18830_amd as ms
from oracle import attn as OA
from oracle import index as OI
from synth import WORKLOADS, make_inputs
from tests.helpers import assert_close, assert_lse_close, inputs_f64, oracle_indices

pytestmark = pytest.mark.gpu

SMALL = {
    "tiny_4k": WORKLOADS["tiny_4k"],
    "gqa_4k_d128": WORKLOADS["layer_32k"].resized(seq=4096, heads_q=4, heads_kv=2, k_v=100, k_s=600),
    "gqa_8k_b2": WORKLOADS["layer_128k"].resized(batch=2, seq=8192, heads_q=4, heads_kv=1, k_v=150, k_s=700),
    "d64_sparse": WORKLOADS["layer_32k"].resized(seq=6144, heads_q=2, heads_kv=2, head_dim=64, k_v=70, k_s=130),
    # odd block counts: the last workgroup of a block pair holds a lone block
    "odd_65_blocks_d64": WORKLOADS["layer_32k"].resized(seq=4160, heads_q=2, heads_kv=1, head_dim=64, k_v=90,
                                                        k_s=300),
    "odd_17_blocks_d128": WORKLOADS["layer_32k"].resized(seq=1088, heads_q=2, heads_kv=2, k_v=40, k_s=200),
}


def _run_fwd(dev, wl, vi, si, x, ring=None):
    dims = ms.make_dims(wl.batch, wl.seq // (ring.world if ring else 1), wl.heads_q, wl.heads_kv, wl.head_dim)
    idx = ms.make_index(dims, torch.from_numpy(vi).to(dev), torch.from_numpy(si).to(dev), ring)
    out, lse = ms.attn_fwd(dims, x["q"].to(dev), x["k"].to(dev), x["v"].to(dev), idx)
    torch.cuda.synchronize()
    return out.float().cpu().numpy(), lse.cpu().numpy()


@pytest.mark.parametrize("name", list(SMALL))
def test_fwd_full_parity(gpu, name):
    wl = SMALL[name]
    print(f"fwd {name} {wl}", flush=True)
    x = make_inputs(wl, "cpu", with_do=False)
    f = inputs_f64(x)
    vi, si, _, _ = oracle_indices(f, wl)
    scale = 1 / math.sqrt(wl.head_dim)
    ro, rl = OA.layer_fwd(f["q"], f["k"], f["v"], OI.Index(vi, si, wl.seq), scale)
    go, gl = _run_fwd(gpu, wl, vi, si, x)
    assert_close("out", go, ro)
    assert_lse_close(gl, rl)


def test_fwd_empty_rows(gpu):
    # slash offsets only in 70..; verticals only late: query block 0 sees no key
    wl = SMALL["gqa_4k_d128"]
    x = make_inputs(wl, "cpu", with_do=False)
    f = inputs_f64(x)
    B, Hq = wl.batch, wl.heads_q
    vi = np.tile(np.array([3000, 3500], np.int32), (B, Hq, 1))
    si = np.tile(np.array([70, 200, 1000], np.int32), (B, Hq, 1))
    ro, rl = OA.layer_fwd(f["q"], f["k"], f["v"], OI.Index(vi, si, wl.seq), 1 / math.sqrt(wl.head_dim))
    go, gl = _run_fwd(gpu, wl, vi, si, x)
    assert np.all(go[:, :, :64] == 0) and np.all(np.isneginf(gl[:, :, :64]))
    assert_close("out", go, ro)
    assert_lse_close(gl, rl)


def test_fwd_dense_budget(gpu):
    # every slash selected: the sparse kernel computes dense causal attention
    wl = SMALL["gqa_4k_d128"].resized(seq=2048)
    x = make_inputs(wl, "cpu", with_do=False)
    f = inputs_f64(x)
    vi = np.zeros((1, wl.heads_q, 1), np.int32)
    si = np.tile(np.arange(wl.seq, dtype=np.int32), (1, wl.heads_q, 1))
    ro, rl = OA.layer_fwd(f["q"], f["k"], f["v"], OI.Index(vi, si, wl.seq), 1 / math.sqrt(wl.head_dim))
    go, gl = _run_fwd(gpu, wl, vi, si, x)
    assert_close("out", go, ro)
    assert_lse_close(gl, rl)


# (striped, 2, 4480): 35 local blocks per shard, so the pair kernels see a lone block;
# inner > 0: the hierarchical step order of Algorithm 2 (inner cards per node)
@pytest.mark.parametrize("layout,W,seq,inner", [("striped", 4, 8192, 0), ("zigzag", 4, 8192, 0),
                                                ("striped", 2, 4480, 0), ("striped", 8, 8192, 4),
                                                ("zigzag", 4, 8192, 2)])
def test_fwd_ring_steps_merge(gpu, layout, W, seq, inner):
    wl = SMALL["gqa_8k_b2"].resized(batch=1, seq=seq)
    x = make_inputs(wl, "cpu", with_do=False)
    f = inputs_f64(x)
    vi, si, _, _ = oracle_indices(f, wl)
    scale = 1 / math.sqrt(wl.head_dim)
    nb = wl.seq // 64
    r = 1
    qg = OI.local_blocks(r, nb, W, layout)
    rows = (qg[:, None] * 64 + np.arange(64)[None]).reshape(-1)
    ref_o, ref_l = OA.layer_fwd(f["q"], f["k"], f["v"], OI.Index(vi, si, wl.seq), scale, rows=rows)
    T = wl.seq // W
    dims = ms.make_dims(1, T, wl.heads_q, wl.heads_kv, wl.head_dim)
    q_loc = x["q"][:, :, torch.from_numpy(rows)].contiguous().to(gpu)
    o_acc = torch.empty(q_loc.shape, dtype=torch.float32, device=gpu)
    l_acc = torch.empty(q_loc.shape[:-1], dtype=torch.float32, device=gpu)
    out = torch.empty_like(q_loc)
    # the same steps through the fused forward + merge
    f_acc = torch.empty_like(o_acc)
    fl_acc = torch.empty_like(l_acc)
    f_out = torch.empty_like(q_loc)
    tv, ts = torch.from_numpy(vi).to(gpu), torch.from_numpy(si).to(gpu)
    sched = OI.ring_schedule(W, inner)
    for t in range(W):
        ring = ms.make_ring(W, r, t, layout, inner)
        shard = int(sched[r, t])
        kg = OI.local_blocks(shard, nb, W, layout)
        krows = torch.from_numpy((kg[:, None] * 64 + np.arange(64)[None]).reshape(-1))
        k_loc = x["k"][:, :, krows].contiguous().to(gpu)
        v_loc = x["v"][:, :, krows].contiguous().to(gpu)
        idx = ms.make_index(dims, tv, ts, ring)
        po = torch.empty(q_loc.shape, dtype=torch.float32, device=q_loc.device)
        _, pl = ms.attn_fwd(dims, q_loc, k_loc, v_loc, idx, out_f32=po, bf16_out=False)
        ms.merge_out_lse(dims, po, pl, o_acc, l_acc, out if t == W - 1 else None, first=(t == 0))
        ms.attn_fwd_merge(dims, q_loc, k_loc, v_loc, idx, f_acc, fl_acc, f_out if t == W - 1 else None,
                          first=(t == 0))
    torch.cuda.synchronize()
    assert_close("ring out", out.float().cpu().numpy(), ref_o)
    assert_close("ring out fp32", o_acc.cpu().numpy(), ref_o)
    assert_lse_close(l_acc.cpu().numpy(), ref_l)
    assert_close("fused ring out", f_out.float().cpu().numpy(), ref_o)
    assert_close("fused ring out fp32", f_acc.cpu().numpy(), ref_o)
    assert_lse_close(fl_acc.cpu().numpy(), ref_l)
    # same arithmetic as the separate merge, up to the compiler's fma contraction
    assert torch.allclose(f_acc, o_acc, rtol=1e-5, atol=1e-6)
    assert torch.allclose(fl_acc, l_acc, rtol=1e-6, atol=1e-6)
