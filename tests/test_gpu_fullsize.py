"""Full-size parity in the benchmark's launch configuration.

The GPU runs index -> forward -> backward over every head of the workload's
full shape.  Every head's vertical and slash sets come from the oracle's fp64
estimator on that head (so no input comes from the GPU).  The oracle then
checks, on four heads spread over two KV groups, sampled query rows spread over
the sequence (out, lse and dQ need only the row itself), and the invariants
that hold at any size: sum over keys of dK is 0 and sum over keys of dV equals
the sum of dO over the group's query rows.  dK and dV of the last 128 keys of
two KV heads are checked element by element: only the last 128 query rows see
them, so the oracle's gradients over those rows are theirs in full.
"""
import math

import numpy as np
import pytest
import torch

import paper_2510_18830_amd as ms
from oracle import attn as OA
from oracle import index as OI
from synth import WORKLOADS, make_inputs
from tests.helpers import (assert_close, assert_lse_close, oracle_sets_every_head, to_f64,
                           weighted_identity_check)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["layer_32k", "layer_128k", "layer_512k"])
def test_fullsize_sampled_rows_and_invariants(gpu, name):
    wl = WORKLOADS[name]
    print(f"full-size {name}", flush=True)
    B, Hq, Hkv, N, d = wl.batch, wl.heads_q, wl.heads_kv, wl.seq, wl.head_dim
    G = Hq // Hkv
    scale = 1 / math.sqrt(d)
    x = make_inputs(wl, gpu)
    heads = [0, G - 1, Hq - G, Hq - 1]
    vi, si = oracle_sets_every_head(x, wl)
    print("oracle sets ready", flush=True)

    dims = ms.make_dims(B, N, Hq, Hkv, d)
    idx = ms.make_index(dims, torch.from_numpy(vi).to(gpu), torch.from_numpy(si).to(gpu))
    out32 = torch.empty(x["q"].shape, dtype=torch.float32, device=gpu)
    out, lse = ms.attn_fwd(dims, x["q"], x["k"], x["v"], idx, out_f32=out32)
    dq, dk, dv = ms.attn_bwd(dims, x["q"], x["k"], x["v"], out, x["do"], lse, idx, out_f32=out32)
    torch.cuda.synchronize()
    print("gpu done", flush=True)

    nb = N // 64
    blocks = np.unique(np.concatenate([[0, 1, nb - 1], np.linspace(2, nb - 2, 13).astype(np.int64)]))
    rows = np.unique(np.concatenate([blocks * 64, blocks * 64 + 37, blocks * 64 + 63]))
    sel = torch.from_numpy(rows).to(gpu)
    for h in heads:
        ref = OI.Index(vi[:, h:h + 1], si[:, h:h + 1], N)
        q = to_f64(x["q"][:, h:h + 1, sel].cpu())
        do = to_f64(x["do"][:, h:h + 1, sel].cpu())
        k = to_f64(x["k"][:, h // G:h // G + 1].cpu())
        v = to_f64(x["v"][:, h // G:h // G + 1].cpu())

        class Rows:      # the oracle's mask rows for the sampled rows, in sample order
            def mask_rows(self, bh, rr):
                return ref.mask_rows(0, rows[np.asarray(rr)])

        ro, rl = OA.layer_fwd(q, k, v, Rows(), scale)
        rq = OA.layer_dq(q, k, v, do, Rows(), scale, np.arange(len(rows)))
        assert_close(f"out h{h}", out[:, h:h + 1, sel].float().cpu().numpy(), ro)
        assert_close(f"out32 h{h}", out32[:, h:h + 1, sel].cpu().numpy(), ro)
        assert_lse_close(lse[:, h:h + 1, sel].cpu().numpy(), rl)
        assert_close(f"dq h{h}", dq[:, h:h + 1, sel].cpu().numpy(), rq)

    # invariants over every key of every KV head (fp64 sums of the GPU output)
    for g in range(Hkv):
        dk64 = dk[0, g].double()
        dv64 = dv[0, g].double()
        s_dk = dk64.sum(0)
        assert (s_dk.abs() <= 1e-4 * dk64.abs().sum(0) + 1e-3).all(), f"sum dK kv{g}"
        want = torch.zeros(d, dtype=torch.float64, device=gpu)
        for h in range(g * G, (g + 1) * G):
            want += x["do"][0, h].double().sum(0)
        s_dv = dv64.sum(0)
        assert ((s_dv - want).abs() <= 1e-4 * dv64.abs().sum(0) + 1e-3).all(), f"sum dV kv{g}"
    # the weighted identities over every key and row.  Both sides hold for
    # whatever dS and P the kernels use (dQ and dK share dS, O and dV share P
    # up to recomputation), so the residual is only the fp32 accumulation
    # order: 1e-10 to 2e-7 of the magnitude at 32K-512K; bar 1e-5.  A gradient
    # row moved to the wrong key shifts the sums by about its own weight, so
    # this catches misrouted partials in bulk (a few tens of rows at 512K);
    # single partials are compared element by element at 32K.
    weighted_identity_check(x, out32, dq, dk, dv, 1e-5)
    # element-wise dK / dV of the last 128 keys of two KV heads: only the last
    # 128 query rows (causal) of the group's heads see them, so the oracle's
    # gradients over those rows alone are the full gradients of these keys
    tail = np.arange(N - 128, N)
    tsel = torch.from_numpy(tail).to(gpu)
    for g in sorted({0, Hkv - 1}):
        k = to_f64(x["k"][:, g:g + 1].cpu())[0, 0]
        v = to_f64(x["v"][:, g:g + 1].cpu())[0, 0]
        rk = np.zeros((128, d))
        rv = np.zeros((128, d))
        for h in range(g * G, (g + 1) * G):
            ref = OI.Index(vi[:, h:h + 1], si[:, h:h + 1], N)
            M = ref.mask_rows(0, tail)
            _, gk, gv = OA.head_bwd(to_f64(x["q"][0, h, tsel].cpu()), k, v, to_f64(x["do"][0, h, tsel].cpu()), M,
                                    scale)
            rk += gk[N - 128:]
            rv += gv[N - 128:]
        assert_close(f"dk tail kv{g}", dk[0, g, N - 128:].cpu().numpy(), rk)
        assert_close(f"dv tail kv{g}", dv[0, g, N - 128:].cpu().numpy(), rv)
    del x, out, out32, dq, dk, dv
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["prefill_1m"])
def test_prefill_forward_sampled_rows(gpu, name):
    """Forward-only sparse prefill at 1M tokens: every head's sets from the
    oracle's estimator, GPU index and forward over every head, sampled rows of
    two heads checked."""
    wl = WORKLOADS[name]
    print(f"prefill {name}", flush=True)
    B, Hq, Hkv, N, d = wl.batch, wl.heads_q, wl.heads_kv, wl.seq, wl.head_dim
    G = Hq // Hkv
    scale = 1 / math.sqrt(d)
    x = make_inputs(wl, gpu, with_do=False)
    heads = [3, Hq - 2]
    vi, si = oracle_sets_every_head(x, wl)
    print("oracle sets ready", flush=True)
    dims = ms.make_dims(B, N, Hq, Hkv, d)
    idx = ms.make_index(dims, torch.from_numpy(vi).to(gpu), torch.from_numpy(si).to(gpu))
    out, lse = ms.attn_fwd(dims, x["q"], x["k"], x["v"], idx)
    torch.cuda.synchronize()
    print("gpu done", flush=True)
    nb = N // 64
    blocks = np.unique(np.concatenate([[0, nb - 1], np.linspace(1, nb - 2, 9).astype(np.int64)]))
    rows = np.unique(np.concatenate([blocks * 64 + 5, blocks * 64 + 63]))
    sel = torch.from_numpy(rows).to(gpu)
    for h in heads:
        ref = OI.Index(vi[:, h:h + 1], si[:, h:h + 1], N)
        q = to_f64(x["q"][:, h:h + 1, sel].cpu())
        k = to_f64(x["k"][:, h // G:h // G + 1].cpu())
        v = to_f64(x["v"][:, h // G:h // G + 1].cpu())

        class Rows:
            def mask_rows(self, bh, rr):
                return ref.mask_rows(0, rows[np.asarray(rr)])

        ro, rl = OA.layer_fwd(q, k, v, Rows(), scale)
        assert_close(f"out h{h}", out[:, h:h + 1, sel].float().cpu().numpy(), ro)
        assert_lse_close(lse[:, h:h + 1, sel].cpu().numpy(), rl)
    del x, out, lse
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name,rank", [("ring_512k_w8", 5)])
def test_ring_share_fullsize_sampled_rows(gpu, name, rank):
    """One worker's share of the striped ring at full size (Section 4.2,
    Algorithm 2): its query shard against all W KV shards as sequential steps,
    forward steps merged by log-sum-exp as they finish (the fused entry
    point), backward per step with dQ summed
    over the steps and later steps reusing the worker's query-side data.  The
    sampled global rows of the worker are checked against the oracle on the
    whole sequence (a row's out, lse and dQ do not depend on the partition);
    dK and dV are checked through invariants of the whole share: summed over
    the steps and keys, dK is 0 and dV equals the sum of dO over the worker's
    rows of the group's heads."""
    wl = WORKLOADS[name]
    print(f"ring share {name} rank {rank}", flush=True)
    B, Hq, Hkv, N, d, W = wl.batch, wl.heads_q, wl.heads_kv, wl.seq, wl.head_dim, wl.world
    G = Hq // Hkv
    scale = 1 / math.sqrt(d)
    x = make_inputs(wl, gpu)
    heads = [1, Hq - 1]
    vi, si = oracle_sets_every_head(x, wl)
    print("oracle sets ready", flush=True)

    T = N // W
    dims = ms.make_dims(B, T, Hq, Hkv, d)
    tv, ts = torch.from_numpy(vi).to(gpu), torch.from_numpy(si).to(gpu)
    lane = torch.arange(64, device=gpu)
    shards = []
    for t in range(W):
        idx = ms.make_index(dims, tv, ts, ms.make_ring(W, rank, t, wl.layout))
        kr = (idx["k_blk_global"].long()[:, None] * 64 + lane[None]).reshape(-1)
        shards.append((x["k"][:, :, kr].contiguous(), x["v"][:, :, kr].contiguous(), idx))
    qblk = shards[0][2]["q_blk_global"].long()
    assert np.array_equal(qblk.cpu().numpy(), OI.local_blocks(rank, N // 64, W, wl.layout))
    rr = (qblk[:, None] * 64 + lane[None]).reshape(-1)
    q_loc = x["q"][:, :, rr].contiguous()
    do_loc = x["do"][:, :, rr].contiguous()
    o_acc = torch.empty(q_loc.shape, dtype=torch.float32, device=gpu)
    l_acc = torch.empty(q_loc.shape[:-1], dtype=torch.float32, device=gpu)
    out = torch.empty_like(q_loc)
    for t, (k_s, v_s, idx) in enumerate(shards):   # forward steps merged as they finish
        ms.attn_fwd_merge(dims, q_loc, k_s, v_s, idx, o_acc, l_acc, out if t == W - 1 else None, first=(t == 0))
    dq = torch.empty(q_loc.shape, dtype=torch.float32, device=gpu)
    bws = ms._workspace(max(ms.attn_bwd_workspace_bytes(dims, s[2].struct.vcol_cap) for s in shards), gpu)
    sum_dk = torch.zeros(Hkv, d, dtype=torch.float64, device=gpu)
    sum_dv = torch.zeros_like(sum_dk)
    abs_dk = torch.zeros_like(sum_dk)
    abs_dv = torch.zeros_like(sum_dk)
    for t, (k_s, v_s, idx) in enumerate(shards):
        _, dk, dv = ms.attn_bwd(dims, q_loc, k_s, v_s, out, do_loc, l_acc, idx, dq=dq, dq_accumulate=(t > 0),
                                out_f32=o_acc, workspace=bws, reuse_qrows=(t > 0))
        sum_dk += dk[0].double().sum(1)
        sum_dv += dv[0].double().sum(1)
        abs_dk += dk[0].double().abs().sum(1)
        abs_dv += dv[0].double().abs().sum(1)
    torch.cuda.synchronize()
    print("gpu done", flush=True)

    nl = T // 64
    lblocks = np.unique(np.concatenate([[0, 1, nl - 1], np.linspace(2, nl - 2, 9).astype(np.int64)]))
    lrows = np.unique(np.concatenate([lblocks * 64 + 3, lblocks * 64 + 63]))
    grows = rr.cpu().numpy()[lrows]
    sel = torch.from_numpy(lrows).to(gpu)
    for h in heads:
        ref = OI.Index(vi[:, h:h + 1], si[:, h:h + 1], N)
        q = to_f64(q_loc[:, h:h + 1, sel].cpu())
        do = to_f64(do_loc[:, h:h + 1, sel].cpu())
        k = to_f64(x["k"][:, h // G:h // G + 1].cpu())
        v = to_f64(x["v"][:, h // G:h // G + 1].cpu())

        class Rows:      # the oracle's mask rows for the sampled global rows, in sample order
            def mask_rows(self, bh, r):
                return ref.mask_rows(0, grows[np.asarray(r)])

        ro, rl = OA.layer_fwd(q, k, v, Rows(), scale)
        rq = OA.layer_dq(q, k, v, do, Rows(), scale, np.arange(len(grows)))
        assert_close(f"out h{h}", out[:, h:h + 1, sel].float().cpu().numpy(), ro)
        assert_close(f"out32 h{h}", o_acc[:, h:h + 1, sel].cpu().numpy(), ro)
        assert_lse_close(l_acc[:, h:h + 1, sel].cpu().numpy(), rl)
        assert_close(f"dq h{h}", dq[:, h:h + 1, sel].cpu().numpy(), rq)
    want_dv = do_loc[0].double().sum(1).reshape(Hkv, G, d).sum(1)
    assert ((sum_dk).abs() <= 1e-4 * abs_dk + 1e-3).all(), "sum dK over the share"
    assert ((sum_dv - want_dv).abs() <= 1e-4 * abs_dv + 1e-3).all(), "sum dV over the share"
    del x, shards, q_loc, do_loc, out, o_acc, dq
    torch.cuda.empty_cache()


def test_layer_512k_deterministic(gpu):
    """The whole step at 512K (estimate, index, forward, backward) run twice on
    the same inputs gives bit-identical results: every reduction has a fixed
    order (no atomics on floating point)."""
    wl = WORKLOADS["layer_512k"]
    x = make_inputs(wl, gpu)
    dims = ms.make_dims(wl.batch, wl.seq, wl.heads_q, wl.heads_kv, wl.head_dim)
    runs = []
    for _ in range(2):
        vi, si = ms.estimate(dims, x["q"], x["k"], wl.last_q, wl.k_v, wl.k_s)
        idx = ms.make_index(dims, vi, si)
        of = torch.empty(x["q"].shape, dtype=torch.float32, device=gpu)
        out, lse = ms.attn_fwd(dims, x["q"], x["k"], x["v"], idx, out_f32=of)
        dq, dk, dv = ms.attn_bwd(dims, x["q"], x["k"], x["v"], out, x["do"], lse, idx, out_f32=of)
        torch.cuda.synchronize()
        runs.append({"v_idx": vi, "s_idx": si, "blk_ptr": idx["blk_ptr"], "col_ptr": idx["col_ptr"], "out": of,
                     "lse": lse, "dq": dq, "dk": dk, "dv": dv})
    for name in runs[0]:
        assert torch.equal(runs[0][name], runs[1][name]), name
    del x, runs
    torch.cuda.empty_cache()
