"""GPU pattern estimation vs the fp64 oracle estimator (Algorithm 1)."""
import math

import numpy as np
import pytest
import torch

import paper_2510_18830_amd as ms
from oracle import estimate as OE
from synth import WORKLOADS, make_inputs
from tests.helpers import assert_topk_match, inputs_f64, oracle_indices, to_f64

pytestmark = pytest.mark.gpu

SMALL = {
    "tiny_4k": WORKLOADS["tiny_4k"],
    "gqa_8k": WORKLOADS["layer_32k"].resized(seq=8192, heads_q=4, heads_kv=2, k_v=200, k_s=900),
    "last_q_17": WORKLOADS["layer_32k"].resized(seq=4096, heads_q=2, heads_kv=1, last_q=17, k_v=64, k_s=300),
    "d64_b2_ragged_chunk": WORKLOADS["tiny_4k"].resized(batch=2, seq=64 * 37, heads_q=2, heads_kv=1, k_v=50, k_s=90),
    "one_block": WORKLOADS["tiny_4k"].resized(seq=64, k_v=5, k_s=64, n_vert=0),
}


def _gpu_estimate(dev, wl, q, k):
    dims = ms.make_dims(wl.batch, wl.seq, wl.heads_q, wl.heads_kv, wl.head_dim)
    vs = torch.empty((wl.batch, wl.heads_q, wl.seq), dtype=torch.float32, device=dev)
    ss = torch.empty_like(vs)
    vi, si = ms.estimate(dims, q, k, wl.last_q, wl.k_v, wl.k_s, v_score=vs, s_score=ss)
    torch.cuda.synchronize()
    return vi.cpu().numpy(), si.cpu().numpy(), vs.cpu().numpy(), ss.cpu().numpy()


def _check(wl, got, ref):
    gvi, gsi, gvs, gss = got
    rvi, rsi, rvs, rss = ref
    for b in range(gvi.shape[0]):
        for h in range(gvi.shape[1]):
            for name, g, r in (("v_score", gvs[b, h], rvs[b, h]), ("s_score", gss[b, h], rss[b, h])):
                np.testing.assert_allclose(g, r, rtol=2e-5, atol=1e-6 * r.max(), err_msg=f"{name} b{b} h{h}")
            assert_topk_match(gvi[b, h], rvi[b, h], rvs[b, h], wl.k_v)
            assert_topk_match(gsi[b, h], rsi[b, h], rss[b, h], wl.k_s)
            # each observed row carries unit mass
            assert abs(gvs[b, h].sum() - wl.last_q) < 1e-3 * wl.last_q
            assert abs(gss[b, h].sum() - wl.last_q) < 1e-3 * wl.last_q


@pytest.mark.parametrize("name", list(SMALL))
def test_estimate_parity(gpu, name):
    wl = SMALL[name]
    print(f"estimate {name} {wl}", flush=True)
    x = make_inputs(wl, "cpu", with_do=False)
    f = inputs_f64(x, ("q", "k"))
    ref = oracle_indices(f, wl)
    got = _gpu_estimate(gpu, wl, x["q"].to(gpu), x["k"].to(gpu))
    _check(wl, got, ref)


def test_estimate_zero_query_ties(gpu):
    # q = 0: all columns m <= N - L tie exactly, as do all diagonals delta <= N - L
    wl = SMALL["gqa_8k"].resized(heads_q=2, heads_kv=1)
    x = make_inputs(wl, "cpu", with_do=False)
    q = torch.zeros_like(x["q"])
    f = {"q": np.zeros(q.shape), "k": to_f64(x["k"])}
    ref = oracle_indices(f, wl)
    assert ref[0][0, 0].tolist() == list(range(wl.k_v))
    got = _gpu_estimate(gpu, wl, q.to(gpu), x["k"].to(gpu))
    _check(wl, got, ref)


def test_estimate_full_budget_and_determinism(gpu):
    wl = SMALL["tiny_4k"].resized(seq=1024, k_v=1024, k_s=1024)
    x = make_inputs(wl, "cpu", with_do=False)
    a = _gpu_estimate(gpu, wl, x["q"].to(gpu), x["k"].to(gpu))
    b = _gpu_estimate(gpu, wl, x["q"].to(gpu), x["k"].to(gpu))
    assert a[0][0, 0].tolist() == list(range(1024)) and a[1][0, 0].tolist() == list(range(1024))
    for u, v in zip(a, b):
        assert np.array_equal(u, v)


@pytest.mark.parametrize("name,heads", [("layer_32k", [0, 9]), ("layer_128k", [5]), ("layer_512k", [27])])
def test_estimate_full_size_sampled_heads(gpu, name, heads):
    """The configuration's full shape on the GPU; the oracle checks sampled heads."""
    wl = WORKLOADS[name]
    print(f"estimate full {name} heads {heads}", flush=True)
    x = make_inputs(wl, gpu, with_do=False)
    got = _gpu_estimate(gpu, wl, x["q"], x["k"])
    G = wl.heads_q // wl.heads_kv
    for h in heads:
        q = to_f64(x["q"][:, h, -wl.last_q:].cpu())
        k = to_f64(x["k"][:, h // G].cpu())
        vs, ss = OE.vs_scores(q[0], k[0], 1 / math.sqrt(wl.head_dim))
        ref = (OE.topk_lower(vs, wl.k_v)[None, None], OE.topk_lower(ss, wl.k_s)[None, None], vs[None, None],
               ss[None, None])
        sub = tuple(g[:, h:h + 1] for g in got)
        _check(wl, sub, ref)
    del x
    torch.cuda.empty_cache()
