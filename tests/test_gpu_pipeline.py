"""The whole path with the online top-p budget: GPU top-p estimate -> padded
lists -> index -> forward -> backward, against the oracle doing the same
(Algorithm 1's score_cover and argtopk, then the index and attention).

The oracle's lists come from its own fp64 scores.  The seed is one whose
budgets are well separated from the neighbouring scores (checked below on the
oracle's scores alone), so the GPU must reproduce the oracle's budgets and
lists exactly; its forward and backward then run on its own lists.
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
from tests.helpers import assert_close, assert_lse_close, inputs_f64

pytestmark = pytest.mark.gpu


def _separated(score, p, k, rel=1e-4):
    """The budget k is not near a tie: the k-th and (k+1)-th largest scores
    differ, and the cumulative mass crosses p of the total, by more than `rel`
    (five times the score tolerance of the estimate tests)."""
    srt = np.sort(score)[::-1]
    c = np.cumsum(srt)
    theta = p * c[-1]
    gap = (srt[k - 1] - srt[k]) / srt[k - 1]
    mass = min(c[k - 1] - theta, theta - (c[k - 2] if k > 1 else 0.0)) / theta
    return gap > rel and mass > rel


@pytest.mark.parametrize("p_v,p_s", [(0.37, 0.37), (0.63, 0.69)])
def test_topp_pipeline(gpu, p_v, p_s):
    wl = WORKLOADS["layer_32k"].resized(seq=4096, heads_q=4, heads_kv=2)
    kmax_v, kmax_s = 1024, 2048
    print(f"top-p pipeline {wl} p {p_v} {p_s}", flush=True)
    x = make_inputs(wl, "cpu")
    f = inputs_f64(x)
    scale = 1 / math.sqrt(wl.head_dim)
    rvi, rsi, rvc, rsc, rvs, rss = OE.estimate_topp(f["q"], f["k"], wl.last_q, p_v, p_s, kmax_v, kmax_s, scale)
    for h in range(wl.heads_q):
        assert _separated(rvs[0, h], p_v, int(rvc[0, h])) and _separated(rss[0, h], p_s, int(rsc[0, h])), h
    assert (rvc < kmax_v).all() and (rsc < kmax_s).all()
    ref = OI.Index(rvi, rsi, wl.seq)
    ro, rl = OA.layer_fwd(f["q"], f["k"], f["v"], ref, scale)
    rq, rk, rv = OA.layer_bwd(f["q"], f["k"], f["v"], f["do"], ref, scale)

    dims = ms.make_dims(wl.batch, wl.seq, wl.heads_q, wl.heads_kv, wl.head_dim)
    q, k, v, do = (x[n].to(gpu) for n in ("q", "k", "v", "do"))
    vi, si, vc, sc = ms.estimate_topp(dims, q, k, wl.last_q, p_v, p_s, kmax_v, kmax_s)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(vc.cpu().numpy(), rvc)
    np.testing.assert_array_equal(sc.cpu().numpy(), rsc)
    np.testing.assert_array_equal(vi.cpu().numpy(), rvi)
    np.testing.assert_array_equal(si.cpu().numpy(), rsi)
    idx = ms.make_index(dims, vi, si)     # padded lists straight from the estimate
    of = torch.empty(q.shape, dtype=torch.float32, device=gpu)
    out, lse = ms.attn_fwd(dims, q, k, v, idx, out_f32=of)
    dq, dk, dv = ms.attn_bwd(dims, q, k, v, out, do, lse, idx, out_f32=of)
    torch.cuda.synchronize()
    assert_close("out", out.float().cpu().numpy(), ro)
    assert_lse_close(lse.cpu().numpy(), rl)
    for name, g, r in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv)):
        assert_close(name, g.cpu().numpy(), r)
