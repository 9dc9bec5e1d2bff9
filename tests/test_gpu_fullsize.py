"""Full-size parity in the benchmark's launch configuration.

The GPU runs index -> forward -> backward over every head of the workload's
full shape.  The index comes from the oracle's estimator on two sampled heads
(their sets are reused for the other heads, so no input comes from the GPU).
The oracle then checks, on the sampled heads, sampled query rows spread over
the sequence (out, lse and dQ need only the row itself), and the invariants
that hold at any size: sum over keys of dK is 0 and sum over keys of dV equals
the sum of dO over the group's query rows.
"""
import math

import numpy as np
import pytest
import torch

import paper_2510_18830_amd as ms
from oracle import attn as OA
from oracle import estimate as OE
from oracle import index as OI
from synth import WORKLOADS, make_inputs
from tests.helpers import assert_close, assert_lse_close, to_f64

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["layer_32k", "layer_128k", "layer_512k"])
def test_fullsize_sampled_rows_and_invariants(gpu, name):
    wl = WORKLOADS[name]
    print(f"full-size {name}", flush=True)
    B, Hq, Hkv, N, d = wl.batch, wl.heads_q, wl.heads_kv, wl.seq, wl.head_dim
    G = Hq // Hkv
    scale = 1 / math.sqrt(d)
    x = make_inputs(wl, gpu)
    heads = [0, Hq - 1]
    sets = {}
    for h in heads:
        q_last = to_f64(x["q"][0, h, N - wl.last_q:].cpu())
        k = to_f64(x["k"][0, h // G].cpu())
        vs, ss = OE.vs_scores(q_last, k, scale)
        sets[h] = (OE.topk_lower(vs, wl.k_v), OE.topk_lower(ss, wl.k_s))
    vi = np.stack([sets[heads[h % 2]][0] for h in range(Hq)])[None].astype(np.int32)
    si = np.stack([sets[heads[h % 2]][1] for h in range(Hq)])[None].astype(np.int32)
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
    del x, out, out32, dq, dk, dv
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["prefill_1m"])
def test_prefill_forward_sampled_rows(gpu, name):
    """Forward-only sparse prefill at 1M tokens: estimate sets from the oracle on
    two heads, GPU index and forward over every head, sampled rows checked."""
    wl = WORKLOADS[name]
    print(f"prefill {name}", flush=True)
    B, Hq, Hkv, N, d = wl.batch, wl.heads_q, wl.heads_kv, wl.seq, wl.head_dim
    G = Hq // Hkv
    scale = 1 / math.sqrt(d)
    x = make_inputs(wl, gpu, with_do=False)
    heads = [3, Hq - 2]
    sets = {}
    for h in heads:
        vs, ss = OE.vs_scores(to_f64(x["q"][0, h, N - wl.last_q:].cpu()), to_f64(x["k"][0, h // G].cpu()), scale)
        sets[h] = (OE.topk_lower(vs, wl.k_v), OE.topk_lower(ss, wl.k_s))
        del vs, ss
    vi = np.stack([sets[heads[h % 2]][0] for h in range(Hq)])[None].astype(np.int32)
    si = np.stack([sets[heads[h % 2]][1] for h in range(Hq)])[None].astype(np.int32)
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
