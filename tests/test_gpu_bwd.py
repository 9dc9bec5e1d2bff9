"""GPU sparse backward vs the fp64 oracle, given the oracle's index."""
import math

import numpy as np
import pytest
import torch

import paper_2510_18830_amd as ms
from oracle import attn as OA
from oracle import index as OI
from synth import WORKLOADS, make_inputs
from tests.helpers import assert_close, inputs_f64, oracle_indices

pytestmark = pytest.mark.gpu

SMALL = {
    "tiny_4k": WORKLOADS["tiny_4k"],
    "gqa_4k_d128": WORKLOADS["layer_32k"].resized(seq=4096, heads_q=4, heads_kv=2, k_v=100, k_s=600),
    "gqa_8k_g4": WORKLOADS["layer_128k"].resized(seq=8192, heads_q=4, heads_kv=1, k_v=150, k_s=700),
    "d64_b2": WORKLOADS["layer_32k"].resized(batch=2, seq=3072, heads_q=2, heads_kv=1, head_dim=64, k_v=70,
                                             k_s=130),
    # odd block counts: lone query block (dQ) and lone key block (dK/dV) per pair
    "odd_65_blocks_d64": WORKLOADS["layer_32k"].resized(seq=4160, heads_q=2, heads_kv=1, head_dim=64, k_v=90,
                                                        k_s=300),
    "odd_17_blocks_d128": WORKLOADS["layer_32k"].resized(seq=1088, heads_q=2, heads_kv=2, k_v=40, k_s=200),
}


def _gpu_fwd_bwd(dev, wl, vi, si, x):
    dims = ms.make_dims(wl.batch, wl.seq, wl.heads_q, wl.heads_kv, wl.head_dim)
    idx = ms.make_index(dims, torch.from_numpy(vi).to(dev), torch.from_numpy(si).to(dev))
    q, k, v, do = (x[n].to(dev) for n in ("q", "k", "v", "do"))
    of = torch.empty(q.shape, dtype=torch.float32, device=dev)
    out, lse = ms.attn_fwd(dims, q, k, v, idx, out_f32=of)
    dq, dk, dv = ms.attn_bwd(dims, q, k, v, out, do, lse, idx, out_f32=of)
    torch.cuda.synchronize()
    return dq.cpu().numpy(), dk.cpu().numpy(), dv.cpu().numpy()


@pytest.mark.parametrize("name", list(SMALL))
def test_bwd_full_parity(gpu, name):
    wl = SMALL[name]
    print(f"bwd {name} {wl}", flush=True)
    x = make_inputs(wl, "cpu")
    f = inputs_f64(x)
    vi, si, _, _ = oracle_indices(f, wl)
    rq, rk, rv = OA.layer_bwd(f["q"], f["k"], f["v"], f["do"], OI.Index(vi, si, wl.seq), 1 / math.sqrt(wl.head_dim))
    gq, gk, gv = _gpu_fwd_bwd(gpu, wl, vi, si, x)
    for n, g, r in (("dq", gq, rq), ("dk", gk, rk), ("dv", gv, rv)):
        e = np.abs(g - r)
        print(f"{n}: max-abs {e.max():.3e} mean-abs {e.mean():.3e} ref-rms {np.sqrt((r ** 2).mean()):.3e}", flush=True)
    assert_close("dq", gq, rq)
    assert_close("dk", gk, rk)
    assert_close("dv", gv, rv)


def test_bwd_empty_rows_and_dense_budget(gpu):
    wl = SMALL["gqa_4k_d128"].resized(seq=2048)
    x = make_inputs(wl, "cpu")
    f = inputs_f64(x)
    scale = 1 / math.sqrt(wl.head_dim)
    # (a) query block 0 sees nothing: its dQ rows are zero
    vi = np.tile(np.array([1500, 1700], np.int32), (1, wl.heads_q, 1))
    si = np.tile(np.array([70, 200, 1000], np.int32), (1, wl.heads_q, 1))
    rq, rk, rv = OA.layer_bwd(f["q"], f["k"], f["v"], f["do"], OI.Index(vi, si, wl.seq), scale)
    gq, gk, gv = _gpu_fwd_bwd(gpu, wl, vi, si, x)
    assert np.all(gq[:, :, :64] == 0)
    for n, g, r in (("dq", gq, rq), ("dk", gk, rk), ("dv", gv, rv)):
        assert_close(n, g, r)
    # (b) every slash selected: dense causal gradients
    vi = np.zeros((1, wl.heads_q, 1), np.int32)
    si = np.tile(np.arange(wl.seq, dtype=np.int32), (1, wl.heads_q, 1))
    rq, rk, rv = OA.layer_bwd(f["q"], f["k"], f["v"], f["do"], OI.Index(vi, si, wl.seq), scale)
    gq, gk, gv = _gpu_fwd_bwd(gpu, wl, vi, si, x)
    for n, g, r in (("dq", gq, rq), ("dk", gk, rk), ("dv", gv, rv)):
        assert_close(n, g, r)


@pytest.mark.parametrize("layout,inner,reuse", [("striped", 0, False), ("zigzag", 0, False), ("striped", 2, False),
                                                ("zigzag", 2, True), ("striped", 0, True)])
def test_bwd_ring_worker_share(gpu, layout, inner, reuse):
    """Worker r's steps: dQ of its rows summed over steps; each step's dK / dV of
    the step's shard equals the whole-sequence gradient restricted to worker r's
    query rows (dO zero elsewhere) and to the shard's keys."""
    W, r = 4, 2
    wl = SMALL["gqa_8k_g4"].resized(heads_q=2, k_v=120, k_s=500)
    x = make_inputs(wl, "cpu")
    f = inputs_f64(x)
    vi, si, _, _ = oracle_indices(f, wl)
    scale = 1 / math.sqrt(wl.head_dim)
    nb = wl.seq // 64
    qg = OI.local_blocks(r, nb, W, layout)
    rows = (qg[:, None] * 64 + np.arange(64)[None]).reshape(-1)
    do_r = np.zeros_like(f["do"])
    do_r[:, :, rows] = f["do"][:, :, rows]
    whole = OI.Index(vi, si, wl.seq)
    rq, rk, rv = OA.layer_bwd(f["q"], f["k"], f["v"], do_r, whole, scale)

    dev = gpu
    T = wl.seq // W
    dims = ms.make_dims(1, T, wl.heads_q, wl.heads_kv, wl.head_dim)
    sel = torch.from_numpy(rows)
    q_loc = x["q"][:, :, sel].contiguous().to(dev)
    do_loc = x["do"][:, :, sel].contiguous().to(dev)
    tv, ts = torch.from_numpy(vi).to(dev), torch.from_numpy(si).to(dev)
    # forward over the ring steps to get the final (merged) out and lse
    o_acc = torch.empty(q_loc.shape, dtype=torch.float32, device=dev)
    l_acc = torch.empty(q_loc.shape[:-1], dtype=torch.float32, device=dev)
    out = torch.empty_like(q_loc)
    shards = []
    sched = OI.ring_schedule(W, inner)      # inner > 0: hierarchical order (Algorithm 2)
    for t in range(W):
        ring = ms.make_ring(W, r, t, layout, inner)
        kg = OI.local_blocks(int(sched[r, t]), nb, W, layout)
        krows = (kg[:, None] * 64 + np.arange(64)[None]).reshape(-1)
        ks = torch.from_numpy(krows)
        k_loc = x["k"][:, :, ks].contiguous().to(dev)
        v_loc = x["v"][:, :, ks].contiguous().to(dev)
        idx = ms.make_index(dims, tv, ts, ring)
        shards.append((krows, k_loc, v_loc, idx))
        po = torch.empty(q_loc.shape, dtype=torch.float32, device=q_loc.device)
        _, pl = ms.attn_fwd(dims, q_loc, k_loc, v_loc, idx, out_f32=po, bf16_out=False)
        ms.merge_out_lse(dims, po, pl, o_acc, l_acc, out if t == W - 1 else None, first=(t == 0))
    dq = torch.empty(q_loc.shape, dtype=torch.float32, device=dev)
    # reuse: one workspace for the worker's steps; later steps keep its query-side data
    bws = ms._workspace(max(ms.attn_bwd_workspace_bytes(dims, s[3].struct.vcol_cap) for s in shards), dev)
    for t, (krows, k_loc, v_loc, idx) in enumerate(shards):
        _, dk, dv = ms.attn_bwd(dims, q_loc, k_loc, v_loc, out, do_loc, l_acc, idx, dq=dq, dq_accumulate=(t > 0),
                                out_f32=o_acc, workspace=bws, reuse_qrows=reuse and t > 0)
        torch.cuda.synchronize()
        assert_close(f"dk step {t}", dk.cpu().numpy(), rk[:, :, krows])
        assert_close(f"dv step {t}", dv.cpu().numpy(), rv[:, :, krows])
    assert_close("dq", dq.cpu().numpy(), rq[:, :, rows])


def test_bwd_independent_head_indices(gpu):
    """Every head gets its own random vertical / slash sets, so a kernel that
    mixes up per-head index data (lists, bitsets) cannot pass."""
    wl = SMALL["gqa_4k_d128"].resized(batch=2, seq=3072, heads_q=4, heads_kv=2)
    x = make_inputs(wl, "cpu")
    f = inputs_f64(x)
    rng = np.random.default_rng(77)
    N = wl.seq
    vi = np.stack([np.stack([np.sort(rng.choice(N, 90, replace=False)) for _ in range(4)]) for _ in range(2)])
    def slashes():
        run = int(rng.integers(50, 150))           # a band from the diagonal, then scattered offsets
        rest = rng.choice(np.arange(run, N), 160 - run, replace=False)
        return np.sort(np.concatenate([np.arange(run), rest]))
    si = np.stack([np.stack([slashes() for _ in range(4)]) for _ in range(2)])
    vi, si = vi.astype(np.int32), si.astype(np.int32)
    idx = OI.Index(vi, si, N)
    assert len({idx.diag_bits[bh].tobytes() for bh in range(8)}) == 8
    scale = 1 / math.sqrt(wl.head_dim)
    rq, rk, rv = OA.layer_bwd(f["q"], f["k"], f["v"], f["do"], idx, scale)
    gq, gk, gv = _gpu_fwd_bwd(gpu, wl, vi, si, x)
    for n, g, r in (("dq", gq, rq), ("dk", gk, rk), ("dv", gv, rv)):
        assert_close(n, g, r)


# degenerate sizes: one block (every tile is the causal diagonal), two blocks,
# unit budgets and a one-row estimation window, both head dims
@pytest.mark.parametrize("seq,head_dim,k_v,k_s,last_q", [(64, 128, 1, 1, 64), (64, 64, 1, 64, 16),
                                                          (128, 128, 1, 1, 1), (128, 64, 3, 2, 1)])
def test_fwd_bwd_minimal_sizes(gpu, seq, head_dim, k_v, k_s, last_q):
    wl = WORKLOADS["tiny_4k"].resized(seq=seq, heads_q=2, heads_kv=1, head_dim=head_dim, k_v=k_v, k_s=k_s,
                                      last_q=last_q, n_vert=0)
    print(f"minimal {wl}", flush=True)
    x = make_inputs(wl, "cpu")
    f = inputs_f64(x)
    vi, si, _, _ = oracle_indices(f, wl)
    scale = 1 / math.sqrt(wl.head_dim)
    ref = OI.Index(vi, si, wl.seq)
    ro, rl = OA.layer_fwd(f["q"], f["k"], f["v"], ref, scale)
    rq, rk, rv = OA.layer_bwd(f["q"], f["k"], f["v"], f["do"], ref, scale)
    dims = ms.make_dims(wl.batch, wl.seq, wl.heads_q, wl.heads_kv, wl.head_dim)
    idx = ms.make_index(dims, torch.from_numpy(vi).to(gpu), torch.from_numpy(si).to(gpu))
    q, k, v, do = (x[n].to(gpu) for n in ("q", "k", "v", "do"))
    of = torch.empty(q.shape, dtype=torch.float32, device=gpu)
    out, lse = ms.attn_fwd(dims, q, k, v, idx, out_f32=of)
    dq, dk, dv = ms.attn_bwd(dims, q, k, v, out, do, lse, idx, out_f32=of)
    torch.cuda.synchronize()
    assert_close("out", of.cpu().numpy(), ro)
    assert_close("dq", dq.cpu().numpy(), rq)
    assert_close("dk", dk.cpu().numpy(), rk)
    assert_close("dv", dv.cpu().numpy(), rv)


def test_fwd_bwd_graph_replay(gpu):
    """msparse_attn_fwd and msparse_attn_bwd captured in one HIP graph and
    replayed on three input sets (eager copies and synchronisations between
    the replays): every replay equals the eager calls bit for bit (the kernels
    are deterministic)."""
    wl = SMALL["gqa_4k_d128"].resized(seq=2048)
    dims = ms.make_dims(wl.batch, wl.seq, wl.heads_q, wl.heads_kv, wl.head_dim)
    xs = [make_inputs(wl.resized(seed=wl.seed + i), "cpu") for i in range(3)]
    f = inputs_f64(xs[0])
    vi, si, _, _ = oracle_indices(f, wl)
    idx = ms.make_index(dims, torch.from_numpy(vi).to(gpu), torch.from_numpy(si).to(gpu))
    fws = ms._workspace(ms.attn_fwd_workspace_bytes(dims), gpu)
    bws = ms._workspace(ms.attn_bwd_workspace_bytes(dims, idx.struct.vcol_cap), gpu)
    bufs = {n: xs[0][n].to(gpu) for n in ("q", "k", "v", "do")}
    out = torch.empty_like(bufs["q"])
    lse = torch.empty(bufs["q"].shape[:-1], dtype=torch.float32, device=gpu)
    of = torch.empty(bufs["q"].shape, dtype=torch.float32, device=gpu)
    dq = torch.empty(bufs["q"].shape, dtype=torch.float32, device=gpu)
    dk = torch.empty(bufs["k"].shape, dtype=torch.float32, device=gpu)
    dv = torch.empty(bufs["v"].shape, dtype=torch.float32, device=gpu)

    def step(stream=None):
        ms.attn_fwd(dims, bufs["q"], bufs["k"], bufs["v"], idx, out=out, lse=lse, out_f32=of, workspace=fws,
                    stream=stream)
        ms.attn_bwd(dims, bufs["q"], bufs["k"], bufs["v"], out, bufs["do"], lse, idx, dq, dk, dv, out_f32=of,
                    workspace=bws, stream=stream)

    refs = []
    for x in xs:
        for n in bufs:
            bufs[n].copy_(x[n].to(gpu))
        step()
        torch.cuda.synchronize()
        refs.append([t.clone() for t in (out, lse, dq, dk, dv)])
    stream = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, stream=stream):
        step(stream)
    for x, ref in zip(xs, refs):
        for n in bufs:
            bufs[n].copy_(x[n].to(gpu))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for name, got, want in zip(("out", "lse", "dq", "dk", "dv"), (out, lse, dq, dk, dv), ref):
            assert torch.equal(got, want), name
