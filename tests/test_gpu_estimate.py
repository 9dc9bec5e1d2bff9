"""GPU pattern estimation vs the fp64 oracle estimator (Algorithm 1)."""
import math

import numpy as np
import pytest
import torch

import paper_2510_18830_amd as ms
from oracle import estimate as OE
from synth import WORKLOADS, make_inputs
from tests.helpers import (assert_budget_near, assert_topk_match, budget_fixed_point, inputs_f64, oracle_indices,
                           to_f64)

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


# ---- top-p budget (score_cover of Algorithm 1)

def _gpu_topp(dev, wl, q, k, p_v, p_s, kmax_v, kmax_s):
    dims = ms.make_dims(wl.batch, wl.seq, wl.heads_q, wl.heads_kv, wl.head_dim)
    vs = torch.empty((wl.batch, wl.heads_q, wl.seq), dtype=torch.float32, device=dev)
    ss = torch.empty_like(vs)
    out = ms.estimate_topp(dims, q, k, wl.last_q, p_v, p_s, kmax_v, kmax_s, v_score=vs, s_score=ss)
    torch.cuda.synchronize()
    return tuple(t.cpu().numpy() for t in out) + (vs.cpu().numpy(), ss.cpu().numpy())


def _check_topp(got, ref_scores, p_v, p_s, kmax_v, kmax_s, heads=None):
    """got = (v_idx, s_idx, v_cnt, s_cnt, v_score, s_score) from the GPU; ref_scores =
    (v_score, s_score) fp64 from the oracle for the same heads."""
    gvi, gsi, gvc, gsc, gvs, gss = got
    rvs, rss = ref_scores
    hs = range(gvi.shape[1]) if heads is None else heads
    for b in range(gvi.shape[0]):
        for j, h in enumerate(hs):
            for idx, cnt, g_sc, r_sc, p, kmax in ((gvi, gvc, gvs, rvs, p_v, kmax_v), (gsi, gsc, gss, rss, p_s, kmax_s)):
                c = int(cnt[b, h])
                # the decision, exactly, in the kernel's precision on its own scores
                assert c == min(budget_fixed_point(g_sc[b, h], p), kmax), (b, h, c)
                # the decision against the fp64 oracle scores, within the mass tolerance
                assert_budget_near(c, r_sc[b, j], p, kmax)
                # the selected set: the oracle's top-c, up to ties at the c-th score
                assert_topk_match(idx[b, h, :c], OE.topk_lower(r_sc[b, j], c), r_sc[b, j], c)
                assert (idx[b, h, c:] == -1).all()


TOPP = [("tiny_4k", 0.5, 0.9), ("gqa_8k", 0.9, 0.95), ("last_q_17", 0.95, 0.8), ("d64_b2_ragged_chunk", 0.99, 0.99),
        ("one_block", 0.7, 0.3)]


@pytest.mark.parametrize("name,p_v,p_s", TOPP)
def test_estimate_topp_parity(gpu, name, p_v, p_s):
    wl = SMALL[name]
    print(f"estimate_topp {name} p {p_v} {p_s}", flush=True)
    x = make_inputs(wl, "cpu", with_do=False)
    f = inputs_f64(x, ("q", "k"))
    N = wl.seq
    _, _, _, _, rvs, rss = OE.estimate_topp(f["q"], f["k"], wl.last_q, p_v, p_s, N, N, 1 / math.sqrt(wl.head_dim))
    got = _gpu_topp(gpu, wl, x["q"].to(gpu), x["k"].to(gpu), p_v, p_s, N, N)
    _check_topp(got, (rvs, rss), p_v, p_s, N, N)


def test_estimate_topp_cap_equals_fixed_k(gpu):
    wl = SMALL["gqa_8k"]
    x = make_inputs(wl, "cpu", with_do=False)
    q, k = x["q"].to(gpu), x["k"].to(gpu)
    got = _gpu_topp(gpu, wl, q, k, 0.999, 0.999, wl.k_v, wl.k_s)
    fixed = _gpu_estimate(gpu, wl, q, k)
    assert (got[2] == wl.k_v).all() and (got[3] == wl.k_s).all()
    assert np.array_equal(got[0], fixed[0]) and np.array_equal(got[1], fixed[1])
    # the same call with a tiny p stops at a budget of 1 for each list
    one = _gpu_topp(gpu, wl, q, k, 1e-9, 1e-9, wl.k_v, wl.k_s)
    assert (one[2] == 1).all() and (one[3] == 1).all()
    vs, ss = got[4], got[5]
    for b in range(wl.batch):
        for h in range(wl.heads_q):
            assert one[0][b, h, 0] == int(np.argmax(vs[b, h])) and one[1][b, h, 0] == int(np.argmax(ss[b, h]))


def test_estimate_topp_zero_query_closed_form(gpu):
    # q = 0: N - L + 1 columns (and diagonals) tie at c0 = H_N - H_{N-L}, so the
    # budget is ceil(p L / c0) (exact rationals) and the lower indices win
    from fractions import Fraction as Fr
    wl = SMALL["gqa_8k"].resized(heads_q=2, heads_kv=1)
    N, L = wl.seq, wl.last_q
    x = make_inputs(wl, "cpu", with_do=False)
    q = torch.zeros_like(x["q"]).to(gpu)
    c0 = sum(Fr(1, n + 1) for n in range(N - L, N))
    for p in (0.3, 0.77):
        r = Fr(p) * L / c0
        assert abs(float(r) - round(float(r))) > 1e-3     # not within rounding of a step
        want = math.ceil(r)
        got = _gpu_topp(gpu, wl, q, x["k"].to(gpu), p, p, N, N)
        assert (got[2] == want).all() and (got[3] == want).all(), (got[2], got[3], want)
        # the tied entries are equal only up to rounding on the GPU (each diagonal
        # is summed along its own path): the tie band decides
        ref = np.array([float(sum(Fr(1, n + 1) for n in range(max(m, N - L), N))) for m in range(N)])
        for b in range(wl.batch):
            for h in range(wl.heads_q):
                for idx in (got[0], got[1]):
                    assert_topk_match(idx[b, h, :want], np.arange(want), ref, want)


@pytest.mark.parametrize("name,heads", [("layer_128k", [5]), ("layer_512k", [0, 27])])
def test_estimate_topp_full_size_sampled_heads(gpu, name, heads):
    wl = WORKLOADS[name]
    print(f"estimate_topp full {name} heads {heads}", flush=True)
    x = make_inputs(wl, gpu, with_do=False)
    p_v, p_s = 0.9, 0.95
    got = _gpu_topp(gpu, wl, x["q"], x["k"], p_v, p_s, wl.k_v, wl.k_s)
    G = wl.heads_q // wl.heads_kv
    rv, rs = [], []
    for h in heads:
        q = to_f64(x["q"][:, h, -wl.last_q:].cpu())
        k = to_f64(x["k"][:, h // G].cpu())
        vs, ss = OE.vs_scores(q[0], k[0], 1 / math.sqrt(wl.head_dim))
        rv.append(vs)
        rs.append(ss)
    _check_topp(got, (np.array(rv)[None], np.array(rs)[None]), p_v, p_s, wl.k_v, wl.k_s, heads=heads)
    del x
    torch.cuda.empty_cache()


def test_mfma_peak_probe_runs(gpu):
    # the measurement kernel beside the attention path: a plausible dense fp16 rate
    t = ms.mfma_peak_tflops(2, 2000)
    assert 300.0 < t < 3000.0, t
    r = ms.mfma_peak_tflops(2, 2000, random=True)
    assert 300.0 < r < 3000.0, r


def test_estimate_graph_replay(gpu):
    """msparse_estimate captured in a HIP graph and replayed on three input sets
    (eager copies and synchronisations between the replays): every replay
    equals the eager call bit for bit."""
    wl = SMALL["gqa_8k"]
    dims = ms.make_dims(wl.batch, wl.seq, wl.heads_q, wl.heads_kv, wl.head_dim)
    xs = [make_inputs(wl.resized(seed=wl.seed + i), "cpu", with_do=False) for i in range(3)]
    q = xs[0]["q"].to(gpu)
    k = xs[0]["k"].to(gpu)
    shape = (wl.batch, wl.heads_q)
    vi = torch.empty(shape + (wl.k_v,), dtype=torch.int32, device=gpu)
    si = torch.empty(shape + (wl.k_s,), dtype=torch.int32, device=gpu)
    vs = torch.empty(shape + (wl.seq,), dtype=torch.float32, device=gpu)
    ss = torch.empty_like(vs)
    ws = ms._workspace(ms.lib().msparse_estimate_workspace(ms.ctypes.byref(dims), wl.last_q, wl.k_v, wl.k_s), gpu)

    def run(stream=None):
        ms.estimate(dims, q, k, wl.last_q, wl.k_v, wl.k_s, vi, si, v_score=vs, s_score=ss, workspace=ws,
                    stream=stream)

    refs = []
    for x in xs:
        q.copy_(x["q"].to(gpu))
        k.copy_(x["k"].to(gpu))
        run()
        torch.cuda.synchronize()
        refs.append([t.clone() for t in (vi, si, vs, ss)])
    stream = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, stream=stream):
        run(stream)
    for x, ref in zip(xs, refs):
        q.copy_(x["q"].to(gpu))
        k.copy_(x["k"].to(gpu))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for name, got, want in zip(("v_idx", "s_idx", "v_score", "s_score"), (vi, si, vs, ss), ref):
            assert torch.equal(got, want), name
