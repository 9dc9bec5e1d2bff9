"""Benchmark of the vertical-slash sparse-attention hot path on one MI355X.

A step is one pass of the whole path over one synthetic layer already resident
in HBM: pattern estimation -> index build (prep, counts, offsets, fill; sized
in the warm-up, overflow flag checked after each step) -> sparse forward ->
sparse backward.  The metric is fwd+bwd TFLOP/s on the computed
blocks (counted FLOPs / step time, see below) and ms per layer.

Counted FLOPs (no credit for skipped tiles or for recomputation):
  fwd = sum over heads of 4 d (64^2 T + 64 C), T = selected 64x64 tiles
        (diagonal tiles in full), C = (query block, column) pairs;
  bwd = 2.5 fwd (the S, dP, dV, dK, dQ GEMMs).
value = (fwd + bwd) / ms_per_step, the step including estimation and the index.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
One JSON line is printed on stdout.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6     # MI355X dense bf16 / fp16 MFMA
PEAK_HBM_GBS = 8000.0


def kernel_source_hash() -> str:
    """sha256 over the kernel library sources (csrc: the kernels and their
    launchers; the public header holds declarations and documentation only)."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2510_18830_amd", "csrc")
    files = sorted(f for f in os.listdir(csrc) if f.endswith((".hip", ".h")))
    for f in files:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def kernel_symbol(label: str, d: int) -> str:
    """The kernel's name in rocprofv3 output for a trace label (the key/value-
    major backward runs its row-split kernel at head dim 128)."""
    if label == "bwd_dkdv" and d == 128:
        return f"bwd_dkdv_rows_kernel<{d}>"
    return f"{label}_kernel<{d}>"


def hbm_traffic(workload: str, kernel: str):
    """Bytes per launch of `kernel` from the committed PMC summary (FETCH_SIZE and
    WRITE_SIZE, copy-calibrated), or None when there is none for this workload
    or the kernel sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{workload}_hbm_traffic.md")
    if not os.path.exists(path):
        return None
    digest, table = None, {}
    with open(path) as fh:
        for line in fh:
            tok = line.split()
            if len(tok) == 2 and tok[0] == "source_sha256":
                digest = tok[1]
            elif len(tok) == 3 and tok[0] == "traffic":
                table[tok[1]] = float(tok[2])
    if digest != kernel_source_hash():
        return None
    return table.get(kernel)


def estimation_and_index_report(r) -> dict:
    """Estimation and index build against their rooflines.  Estimation: HBM
    fraction on algorithmic bytes (K once, the last query rows, the two score
    vectors written and read back, the selected indices), MFMA fraction on the
    two passes' FLOPs, and the measured HBM bytes of the estimation kernels
    from the committed counters (None when stale).  Index: HBM fraction on the
    bytes it reads (index lists) and writes (CSR entries and offsets)."""
    wl = r["wl"]
    B, Hq, Hkv, N, d, L = wl.batch, wl.heads_q, wl.heads_kv, wl.seq, wl.head_dim, wl.last_q
    est_bytes = (B * Hkv * N * d * 2 + B * Hq * L * d * 2 + 2 * (2 * B * Hq * N * 4)
                 + B * Hq * (wl.k_v + wl.k_s) * 4)
    est_flops = 2 * 2.0 * L * B * Hq * N * d
    t_est = r["stage_ms"]["estimate"] * 1e-3
    measured = hbm_traffic(wl.name, "estimation_total")   # every estimation launch of one step
    measured = None if measured is None else round(measured)
    nqb = N // 64
    idx_bytes = (B * Hq * (wl.k_v + wl.k_s) * 4                       # read the selected indices
                 + 4 * (2 * r["T"] + r["C"] + r["vcol"])             # block, transposed, column, vertical entries
                 + 8 * (2 * B * Hq * nqb + B * Hq * (N // 64) + B * Hq))   # offsets
    t_idx = r["stage_ms"]["index"] * 1e-3
    return {
        "estimation_ms": round(t_est * 1e3, 3),
        "estimation_algorithmic_bytes": int(est_bytes),
        "estimation_hbm_frac": round(est_bytes / t_est / (PEAK_HBM_GBS * 1e9), 4),
        "estimation_mfma_frac": round(est_flops / t_est / (PEAK_BF16_TFLOPS * 1e12), 4),
        "estimation_measured_hbm_bytes": measured,
        "index_ms": round(t_idx * 1e3, 3),
        "index_algorithmic_bytes": int(idx_bytes),
        "index_hbm_frac": round(idx_bytes / t_idx / (PEAK_HBM_GBS * 1e9), 4),
    }


def kernel_flops(name: str, d: int, T: int, C: int, BH: int, N: int, issued: bool = False) -> float:
    """GEMM work of each kernel on the computed blocks / columns.

    Counted (issued=False): the five backward GEMMs (S, dP, dV, dK, dQ) are
    counted once, with S and dP attributed to the key-major dK/dV kernels and
    only the dQ GEMM to the query-major dQ kernel, so the kernels' counted
    FLOPs add up to fwd + 2.5 fwd.  Issued (issued=True): what each kernel
    executes, including the S and dP that the dQ kernel recomputes."""
    pair = 2.0 * d            # one multiply-add over d per (row, key) per GEMM
    tiles = 4096.0 * T + 64.0 * C
    return {
        "attn_fwd": 2 * pair * tiles,                 # S, PV
        "bwd_dq": (3 if issued else 1) * pair * tiles,   # (S, dP recomputed,) dQ
        "bwd_dkdv": 4 * pair * 4096.0 * T,            # S, dP, dV, dK on tiles
        "bwd_dkdv_col": 4 * pair * 64.0 * C,          # the same on column pairs
        "est_pass1": pair * 64.0 * N * BH,            # last 64 rows x all keys
        "est_pass2": pair * 64.0 * N * BH,
    }.get(name, 0.0)


# The paper's own numbers for this path (context, other hardware): NVIDIA
# A100-40GB, 32 GPUs (4 nodes x 8), Qwen2.5-3B at 512K tokens, context
# parallel 32, bf16 (Section 5.4, latency breakdown).
PAPER_CONTEXT = {
    "hardware": "NVIDIA A100-40GB x 32 (4 nodes x 8, NVLink 3.0 + HDR InfiniBand), bf16",
    "workload": "Qwen2.5-3B continued pretraining at 512K tokens, context parallel 32",
    "index_building_ms_per_attention_forward": 1.13,
    "sparse_attention_compute_ms_per_ring_step_forward": 0.51,
    "forward_attention_total_ms_striped_ring_flat": 34.10,
    "forward_attention_total_ms_hierarchical_ring": 19.53,
    "note": "per-worker latencies inside a 32-GPU ring, not single-GPU throughput; the paper reports no "
            "backward timing and no TFLOP/s",
}

GEMM_DTYPES = {
    "fwd_QK^T": "bf16 MFMA (inputs as given)",
    "fwd_PV": "fp16 MFMA (P in fp16; V as an exact fp16 copy of the bf16 values times a power of two)",
    "bwd_all_GEMMs": "fp16 MFMA on exact fp16 copies of bf16 Q, K, V, dO (each times a power of two); "
                     "P and dZ in fp16, scaled by powers of two",
    "accumulate": "fp32",
    "softmax_and_outputs": "fp32 softmax; out bf16 (+ optional fp32), lse / dQ / dK / dV fp32",
}


def cpu_baseline(wl, x, vi, si, rows_wanted: int):
    """The fp64 oracle on a bounded sample of query rows of head 0."""
    import numpy as np
    from oracle import attn as OA, bf16 as OB, index as OI
    from synth import bf16_bits
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] or [os.cpu_count() or 1])
    except Exception:
        cores = os.cpu_count() or 1
    N, d = wl.seq, wl.head_dim
    G = wl.heads_q // wl.heads_kv
    idx = OI.Index(vi[:1, :1], si[:1, :1], N)
    nb = N // 64
    blocks = np.linspace(0, nb - 1, max(1, rows_wanted // 2)).astype(np.int64)
    rows = np.unique(np.concatenate([blocks * 64 + 5, blocks * 64 + 60]))
    q = OB.to_f64(bf16_bits(x["q"][0:1, 0:1, torch_index(rows)].cpu()))
    do = OB.to_f64(bf16_bits(x["do"][0:1, 0:1, torch_index(rows)].cpu()))
    k = OB.to_f64(bf16_bits(x["k"][0:1, 0:1].cpu()))
    v = OB.to_f64(bf16_bits(x["v"][0:1, 0:1].cpu()))

    class RowIndex:        # the oracle's mask for the sampled rows, in sample order
        def mask_rows(self, bh, rr):
            return idx.mask_rows(0, rows[np.asarray(rr)])

    scale = 1 / math.sqrt(d)
    t0 = time.perf_counter()
    OA.layer_fwd(q, k, v, RowIndex(), scale)
    OA.layer_dq(q, k, v, do, RowIndex(), scale, np.arange(len(rows)))
    dt = time.perf_counter() - t0
    pairs = sum(64 * len(idx.blocks[0][n // 64]) + len(idx.cols[0][n // 64]) for n in rows.tolist())
    flops = 3.5 * 4 * d * pairs     # fwd + bwd counted per row, as for the GPU
    full_s = dt / len(rows) * wl.batch * wl.heads_q * N
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{len(rows)} query rows of head 0 of {wl.name}: fp64 dense-masked forward and dQ, "
                      f"{dt:.1f} s",
            "extrapolated_full_layer_s": round(full_s, 1),
            "extrapolation": f"EXTRAPOLATED, not measured: the sample's time per row x {wl.batch * wl.heads_q * N} "
                             f"rows (every query row of every head; forward and dQ per row, the dK / dV "
                             f"accumulation not included)"}


def ring_leg(x, v_idx, s_idx, wl, world: int, rank: int, steps: int):
    """One worker's share of the striped ring (Section 4.2): its query shard
    against every KV shard as sequential steps (forward with LSE merge, then
    backward), plus the per-step and per-worker tile-work imbalance of the
    striped and zigzag layouts from the index alone."""
    import numpy as np
    import torch
    import paper_2510_18830_amd as ms
    dev = x["q"].device
    B, Hq, Hkv, N, d = wl.batch, wl.heads_q, wl.heads_kv, wl.seq, wl.head_dim
    T = N // world
    dims = ms.make_dims(B, T, Hq, Hkv, d)
    lane = torch.arange(64, device=dev)

    def rows_of(blk_global):
        # the shard's tokens in local order, from the library's local -> global block map
        return (blk_global.long()[:, None] * 64 + lane[None]).reshape(-1)

    # work per (layout, worker, step) from the index counts: tiles + columns / 64
    work = {}
    idx_ws = ms._workspace(ms.index_workspace_bytes(dims, wl.k_v, wl.k_s, ms.make_ring(world, 0, 1)), dev)
    for layout in ("striped", "zigzag"):
        m = np.zeros((world, world))
        for r in range(world):
            for t in range(world):
                blk, col, _ = ms.index_count(dims, v_idx, s_idx, ms.make_ring(world, r, t, layout),
                                             workspace=idx_ws)
                m[r, t] = blk + col / 64.0
        work[layout] = m
    # timed share of worker `rank`, striped (shard extraction stands in for the transfers)
    shards, nnz = [], []
    for t in range(world):
        ring = ms.Ring(world, rank, t, ms.STRIPED)
        blk, col, vcol = ms.index_count(dims, v_idx, s_idx, ring, workspace=idx_ws)
        idx = ms.alloc_index(dims, blk, col, vcol, dev, world)
        ms.build_index(dims, v_idx, s_idx, idx, ring, workspace=idx_ws)
        kr = rows_of(idx["k_blk_global"])
        shards.append((x["k"][:, :, kr].contiguous(), x["v"][:, :, kr].contiguous(), idx))
        nnz.append((blk, col))
    rr = rows_of(shards[0][2]["q_blk_global"])
    q_loc = x["q"][:, :, rr].contiguous()
    do_loc = x["do"][:, :, rr].contiguous()
    o_acc = torch.empty(q_loc.shape, dtype=torch.float32, device=dev)
    l_acc = torch.empty(q_loc.shape[:-1], dtype=torch.float32, device=dev)
    out = torch.empty_like(q_loc)
    fws = ms._workspace(ms.attn_fwd_workspace_bytes(dims), dev)
    dq = torch.empty(q_loc.shape, dtype=torch.float32, device=dev)
    dk = torch.empty(shards[0][0].shape, dtype=torch.float32, device=dev)
    dv = torch.empty_like(dk)
    bws = ms._workspace(max(ms.attn_bwd_workspace_bytes(dims, s[2].struct.vcol_cap) for s in shards), dev)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(world)]

    def run(timed):
        for t, (k_s, v_s, idx) in enumerate(shards):
            if timed:
                ev[t][0].record()
            ms.attn_fwd_merge(dims, q_loc, k_s, v_s, idx, o_acc, l_acc, out if t == world - 1 else None,
                              first=(t == 0), workspace=fws)
            if timed:
                ev[t][1].record()
        for t, (k_s, v_s, idx) in enumerate(shards):
            if timed:
                ev[t][2].record()
            ms.attn_bwd(dims, q_loc, k_s, v_s, out, do_loc, l_acc, idx, dq, dk, dv, dq_accumulate=(t > 0),
                        out_f32=o_acc, workspace=bws, reuse_qrows=(t > 0))
            if timed:
                ev[t][3].record()

    run(False)
    fwd_ms = np.zeros(world)
    bwd_ms = np.zeros(world)
    for _ in range(steps):
        run(True)
        torch.cuda.synchronize()
        fwd_ms += [ev[t][0].elapsed_time(ev[t][1]) for t in range(world)]
        bwd_ms += [ev[t][2].elapsed_time(ev[t][3]) for t in range(world)]
    fwd_ms /= steps
    bwd_ms /= steps
    flops = np.array([3.5 * 4.0 * d * (4096.0 * b + 64.0 * c) for b, c in nnz])
    total_ms = float(fwd_ms.sum() + bwd_ms.sum())

    def imb(v):
        v = np.asarray(v, dtype=np.float64)
        return round(float(v.max() / v.mean()), 3)
    return {
        "workload": wl.name, "world": world, "rank": rank, "layout": "striped",
        "step_ms_fwd": [round(float(v), 3) for v in fwd_ms], "step_ms_bwd": [round(float(v), 3) for v in bwd_ms],
        "share_ms": round(total_ms, 2),
        "share_tflops": round(float(flops.sum()) / (total_ms * 1e-3) / 1e12, 2),
        "step_imbalance_time": imb(fwd_ms + bwd_ms),
        "step_imbalance_work": {lay: imb(m[rank]) for lay, m in work.items()},
        "worker_imbalance_work_mean_over_steps": {lay: round(float(np.mean([m[:, t].max() / m[:, t].mean()
                                                                            for t in range(world)])), 3)
                                                  for lay, m in work.items()},
    }


def build_index_step(ms, dims, v_idx, s_idx, state, idx_ws, dev):
    """The index of one step.  The first step sizes it: one count-and-build
    call (one GPU wait) into an index grown to the counts plus 5 % headroom.
    Later steps build asynchronously into that index (msparse_build_index, no
    host wait inside the step) and its overflow flag is read after the step
    (check_index_step): the attention calls leave their outputs untouched on
    an overflowed index, so such a step would be invalid, and the sets, hence
    the sizes, are the same every step here.  Returns the counts."""
    if "idx" not in state:
        state["idx"] = ms.alloc_index(dims, 0, 0, 0, dev)
        built, nnz = ms.index_count_build(dims, v_idx, s_idx, state["idx"], workspace=idx_ws)
        if not built:
            blk, col, vcol = nnz
            state["idx"] = ms.alloc_index(dims, int(blk * 1.05) + 64, int(col * 1.05) + 64, vcol, dev)
            built, nnz = ms.index_count_build(dims, v_idx, s_idx, state["idx"], workspace=idx_ws)
            assert built
        state["nnz_index"] = nnz
        return nnz
    ms.build_index(dims, v_idx, s_idx, state["idx"], workspace=idx_ws)
    return state["nnz_index"]


def check_index_step(state):
    """After a step's final synchronisation: its index did not overflow and has
    the counts the step reported."""
    idx = state["idx"]
    assert int(idx["overflow"].item()) == 0, "index overflowed: the step's attention outputs are invalid"
    t = idx.tensors
    got = (int(t["blk_ptr"][-1].item()), int(t["col_ptr"][-1].item()), int(t["vcol_ptr"][-1].item()))
    assert got == tuple(state["nnz_index"]), (got, state["nnz_index"])


def prefill_leg(ms, torch, wl, x, steps: int, warmup: int) -> dict:
    """Forward-only sparse prefill (inference): estimate -> index -> forward per
    layer, inputs resident in HBM, stage times from HIP events on the stream."""
    dev = x["q"].device
    q, k, v = x["q"], x["k"], x["v"]
    B, Hq, N, d = wl.batch, wl.heads_q, wl.seq, wl.head_dim
    dims = ms.make_dims(B, N, Hq, wl.heads_kv, d)
    est_ws = ms._workspace(ms.lib().msparse_estimate_workspace(ms.ctypes.byref(dims), wl.last_q, wl.k_v, wl.k_s), dev)
    idx_ws = ms._workspace(ms.index_workspace_bytes(dims, wl.k_v, wl.k_s), dev)
    fwd_ws = ms._workspace(ms.attn_fwd_workspace_bytes(dims), dev)
    v_idx = torch.empty((B, Hq, wl.k_v), dtype=torch.int32, device=dev)
    s_idx = torch.empty((B, Hq, wl.k_s), dtype=torch.int32, device=dev)
    out = torch.empty_like(q)
    lse = torch.empty(q.shape[:-1], dtype=torch.float32, device=dev)
    ev = {s_: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for s_ in ("estimate", "index", "fwd")}
    acc = {s_: 0.0 for s_ in ev}
    state = {}

    def step(timed):
        def mark(stage, i):
            if timed:
                ev[stage][i].record()
        mark("estimate", 0)
        ms.estimate(dims, q, k, wl.last_q, wl.k_v, wl.k_s, v_idx, s_idx, workspace=est_ws)
        mark("estimate", 1)
        mark("index", 0)
        blk, col, vcol = build_index_step(ms, dims, v_idx, s_idx, state, idx_ws, dev)
        mark("index", 1)
        mark("fwd", 0)
        ms.attn_fwd(dims, q, k, v, state["idx"], out=out, lse=lse, workspace=fwd_ws)
        mark("fwd", 1)
        state["nnz"] = (blk, col)
        if timed:
            torch.cuda.synchronize()
            check_index_step(state)
            for s_, (a, b) in ev.items():
                acc[s_] += a.elapsed_time(b)

    for _ in range(warmup):
        step(False)
    torch.cuda.synchronize()
    for _ in range(steps):
        step(True)
    stage = {s_: acc[s_] / steps for s_ in acc}
    T, C = state["nnz"]
    fwd_flops = 4.0 * d * (4096.0 * T + 64.0 * C)
    nb = N // 64
    total = sum(stage.values())
    del state
    torch.cuda.empty_cache()
    return {"ms_per_layer": round(total, 3), "stage_ms": {s_: round(t, 3) for s_, t in stage.items()},
            "fwd_tflops_kernel": round(fwd_flops / (stage["fwd"] * 1e-3) / 1e12, 2),
            "fwd_tflops_layer": round(fwd_flops / (total * 1e-3) / 1e12, 2),
            "tokens_per_s": round(B * N / (total * 1e-3)),
            "counted_tiles": int(T), "counted_col_pairs": int(C),
            "tile_density_causal": round(T / (B * Hq * nb * (nb + 1) / 2.0), 4),
            "shape": {"seq_len": N, "heads_q": Hq, "heads_kv": wl.heads_kv, "head_dim": d, "k_v": wl.k_v,
                      "k_s": wl.k_s}}


def topp_leg(ms, torch, wl, x, ps, reps: int = 3) -> dict:
    """Estimation with the online top-p budget (score_cover): time per call and
    the budgets it picks, per fraction p (caps = N, so nothing is capped)."""
    dev = x["q"].device
    B, Hq, N, d = wl.batch, wl.heads_q, wl.seq, wl.head_dim
    dims = ms.make_dims(B, N, Hq, wl.heads_kv, d)
    ws = ms._workspace(ms.lib().msparse_estimate_topp_workspace(ms.ctypes.byref(dims), wl.last_q, N, N), dev)
    out = {}
    for p in ps:
        ms.estimate_topp(dims, x["q"], x["k"], wl.last_q, p, p, N, N, workspace=ws)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            vi, si, vc, sc = ms.estimate_topp(dims, x["q"], x["k"], wl.last_q, p, p, N, N, workspace=ws)
        b.record()
        torch.cuda.synchronize()
        vc = vc.float()
        sc = sc.float()
        out[str(p)] = {"estimate_ms": round(a.elapsed_time(b) / reps, 3),
                       "k_v_min_mean_max": [int(vc.min()), round(float(vc.mean()), 1), int(vc.max())],
                       "k_s_min_mean_max": [int(sc.min()), round(float(sc.mean()), 1), int(sc.max())]}
        del vi, si
    torch.cuda.empty_cache()
    return out


def balance_leg(ms, torch, wl, v_idx, s_idx, worlds, inner: int = 8) -> dict:
    """Striped vs zigzag ring balance from the index (Section 4.2; Section 5's
    workload balance analysis): per world size W, the worker x shard workload in
    tile-equivalents (tiles + columns / 64, msparse_ring_work) and its imbalance
    degrees max / mean under the flat ring and the hierarchical order with
    `inner` cards per node: worker level = mean over steps of max / mean over
    workers, step level = mean over workers of max / mean over steps."""
    import numpy as np
    dims = ms.make_dims(wl.batch, wl.seq, wl.heads_q, wl.heads_kv, wl.head_dim)
    ws = ms._workspace(ms.index_workspace_bytes(dims, v_idx.shape[-1], s_idx.shape[-1]), v_idx.device)

    def degrees(work, W, inn):
        sched = np.array([[ms.ring_shard(W, inn, r, t) for t in range(W)] for r in range(W)])
        per = work[np.arange(W)[:, None], sched]            # [worker, step]
        return (float(np.mean(per.max(0) / per.mean(0))), float(np.mean(per.max(1) / per.mean(1))))

    out = {}
    for layout in ("striped", "zigzag"):
        for W in worlds:
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            tiles, cols = ms.ring_work(dims, v_idx, s_idx, W, layout, workspace=ws)
            b.record()
            torch.cuda.synchronize()
            work = tiles.cpu().numpy().astype(np.float64) + cols.cpu().numpy() / 64.0
            fw, fs = degrees(work, W, 0)
            ent = {"ms": round(a.elapsed_time(b), 3), "worker_level_flat": round(fw, 4), "step_level": round(fs, 4),
                   "worker0_steps_flat": [round(float(work[0, ms.ring_shard(W, 0, 0, t)])) for t in range(min(W, 8))]}
            if W % inner == 0 and W > inner:
                hw, hs = degrees(work, W, inner)
                ent["worker_level_hierarchical"] = round(hw, 4)
                assert abs(hs - fs) < 1e-9       # a step order permutes each worker's row
            out[f"{layout}_w{W}"] = ent
    return out


def torch_index(rows):
    import torch
    return torch.from_numpy(rows)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="layer_512k")
    ap.add_argument("--also", default="layer_128k", help="second workload timed the same way ('' to skip)")
    ap.add_argument("--cpu-rows", type=int, default=1024)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--ring", type=int, default=1, help="also time worker 0's share of the 8-worker ring (512K)")
    ap.add_argument("--prefill", default="layer_128k,layer_512k,prefill_1m",
                    help="workloads timed as forward-only sparse prefill ('' to skip)")
    ap.add_argument("--topp", default="0.5,0.9", help="top-p fractions timed on the main workload ('' to skip)")
    ap.add_argument("--balance", default="8,32,128", help="ring sizes of the striped / zigzag balance sweep ('' to skip)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (HBM counter calibration) and exit")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_each_way": n * 4, "launches": 3}))
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the sparse path here runs on a single MI355X "
              "(a ring worker's share is timed as sequential steps); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2510_18830_amd as ms
    from synth import WORKLOADS, make_inputs

    dev = torch.device("cuda:0")
    results = {}
    for name in [args.workload] + ([args.also] if args.also else []):
        wl = WORKLOADS[name]
        print(f"[bench] {name}: generating inputs", file=sys.stderr, flush=True)
        x = make_inputs(wl, dev)
        q, k, v, do = x["q"], x["k"], x["v"], x["do"]
        B, Hq, N, d = wl.batch, wl.heads_q, wl.seq, wl.head_dim
        dims = ms.make_dims(B, N, Hq, wl.heads_kv, d)
        est_ws = ms._workspace(ms.lib().msparse_estimate_workspace(ms.ctypes.byref(dims), wl.last_q, wl.k_v, wl.k_s),
                               dev)
        idx_ws = ms._workspace(ms.index_workspace_bytes(dims, wl.k_v, wl.k_s), dev)
        bwd_ws = ms._workspace(ms.attn_bwd_workspace_bytes(dims, B * Hq * wl.k_v), dev)
        fwd_ws = ms._workspace(ms.attn_fwd_workspace_bytes(dims), dev)
        v_idx = torch.empty((B, Hq, wl.k_v), dtype=torch.int32, device=dev)
        s_idx = torch.empty((B, Hq, wl.k_s), dtype=torch.int32, device=dev)
        out = torch.empty_like(q)
        out32 = torch.empty(q.shape, dtype=torch.float32, device=dev)
        lse = torch.empty(q.shape[:-1], dtype=torch.float32, device=dev)
        dq = torch.empty(q.shape, dtype=torch.float32, device=dev)
        dk = torch.empty(k.shape, dtype=torch.float32, device=dev)
        dv = torch.empty(v.shape, dtype=torch.float32, device=dev)
        ev = {s: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for s in ("estimate", "index", "fwd", "bwd")}
        acc = {s: 0.0 for s in ev}
        per_step = []
        state = {}

        def step(timed):
            def mark(stage, i):
                if timed:
                    ev[stage][i].record()
            mark("estimate", 0)
            ms.estimate(dims, q, k, wl.last_q, wl.k_v, wl.k_s, v_idx, s_idx, workspace=est_ws)
            mark("estimate", 1)
            mark("index", 0)
            blk, col, vcol = build_index_step(ms, dims, v_idx, s_idx, state, idx_ws, dev)
            idx = state["idx"]
            mark("index", 1)
            mark("fwd", 0)
            ms.attn_fwd(dims, q, k, v, idx, out=out, lse=lse, out_f32=out32, workspace=fwd_ws)
            mark("fwd", 1)
            mark("bwd", 0)
            ms.attn_bwd(dims, q, k, v, out, do, lse, idx, dq, dk, dv, out_f32=out32, workspace=bwd_ws)
            mark("bwd", 1)
            state["nnz"] = (blk, col)
            state["vcol"] = vcol
            if timed:
                torch.cuda.synchronize()
                check_index_step(state)
                tot = 0.0
                for s, (a, b) in ev.items():
                    t = a.elapsed_time(b)
                    acc[s] += t
                    tot += t
                per_step.append(tot)

        print(f"[bench] {name}: warmup {args.warmup}", file=sys.stderr, flush=True)
        for _ in range(args.warmup):
            step(False)
        torch.cuda.synchronize()
        ms.trace_read()
        ms.trace_enable(True)
        print(f"[bench] {name}: timing {args.steps} steps", file=sys.stderr, flush=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            step(True)
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t0) * 1e3 / args.steps
        ms.trace_enable(False)
        kern = ms.trace_read()
        T, C = state["nnz"]
        fwd_flops = 4.0 * d * (4096.0 * T + 64.0 * C)
        step_ms = {s: acc[s] / args.steps for s in acc}
        ms_step = sum(step_ms.values())
        per_kernel = {}
        for kname, (n, tot) in kern.items():
            avg = tot / max(n, 1)
            fl = kernel_flops(kname, d, T, C, B * Hq, N)
            fi = kernel_flops(kname, d, T, C, B * Hq, N, issued=True)
            per_kernel[kname] = {"launches_per_step": n / args.steps, "avg_ms": round(avg, 4),
                                 "tflops_counted": round(fl / (avg * 1e-3) / 1e12, 2) if fl else None,
                                 "tflops_issued_incl_recompute": round(fi / (avg * 1e-3) / 1e12, 2) if fi else None}
        nb = N // 64
        results[name] = dict(
            wl=wl, ms_per_step=ms_step, wall_ms_per_step=wall, stage_ms=step_ms, kernels=per_kernel,
            median_ms_per_step=float(np.median(per_step)),
            fwd_flops=fwd_flops, T=T, C=C, vcol=state["vcol"],
            density=T / (B * Hq * nb * (nb + 1) / 2.0),
            v_idx=v_idx.cpu().numpy(), s_idx=s_idx.cpu().numpy(), x=x if name == args.workload else None)
        print(f"[bench] {name}: {ms_step:.2f} ms/step {json.dumps(step_ms)}", file=sys.stderr, flush=True)
        if name != args.workload:
            del x, q, k, v, do
        torch.cuda.empty_cache()

    main_r = results[args.workload]
    wl = main_r["wl"]
    tot_flops = 3.5 * main_r["fwd_flops"]
    value = tot_flops / (main_r["ms_per_step"] * 1e-3) / 1e12
    # dominant kernel by time per step
    kern = main_r["kernels"]
    dom = max(kern, key=lambda n: kern[n]["avg_ms"] * kern[n]["launches_per_step"])
    dk_ = kern[dom]
    achieved = dk_["tflops_counted"] if dk_["tflops_counted"] is not None else 0.0
    traffic = hbm_traffic(wl.name, kernel_symbol(dom, wl.head_dim))
    for r in results.values():
        r["est_idx"] = estimation_and_index_report(r)
    # achievable dense fp16 MFMA rate on this GPU (probe kernel, no memory traffic): constant
    # operands, and random operands (real data's switching; the power limit then lowers the clock)
    peak_meas = max(ms.mfma_peak_tflops(w) for w in (2, 4))
    peak_rand = max(ms.mfma_peak_tflops(w, random=True) for w in (2, 4))
    st = main_r["stage_ms"]
    ff = main_r["fwd_flops"]
    counted = {   # counted FLOPs (fwd; bwd = 2.5 fwd) over stage times, as fractions of the bf16 / fp16 peak
        "fwd_stage": round(ff / (st["fwd"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "bwd_stage": round(2.5 * ff / (st["bwd"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "fwd_plus_bwd_stages": round(3.5 * ff / ((st["fwd"] + st["bwd"]) * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "whole_step": round(3.5 * ff / (main_r["ms_per_step"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
    }
    roofline = {"bound": "mfma", "kernel": dom, "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "achieved_flops_per_launch": kernel_flops(dom, wl.head_dim, main_r["T"], main_r["C"],
                                                          wl.batch * wl.heads_q, wl.seq),
                "flops_attribution": "counted GEMMs: S, dP, dV, dK to the dK/dV kernels, dQ to the dQ kernel "
                                     "(its recomputed S, dP uncounted), S, PV to the forward",
                "counted_frac_of_peak": counted,
                "peak_measured": round(peak_meas, 1), "frac_of_measured": round(achieved / peak_meas, 4),
                "peak_measured_random_operands": round(peak_rand, 1),
                "frac_of_measured_random_operands": round(achieved / peak_rand, 4),
                "traffic": None if traffic is None else round(traffic), "traffic_unit": "HBM bytes per launch"}
    line = {
        "metric": "sparse attn fwd+bwd TFLOP/s on computed blocks + ms/layer at 128K and 512K",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(main_r["ms_per_step"], 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "gemm_dtypes": GEMM_DTYPES,
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": wl.batch, "seq_len": wl.seq, "heads_q": wl.heads_q,
                   "heads_kv": wl.heads_kv, "head_dim": wl.head_dim, "last_q": wl.last_q, "k_v": wl.k_v,
                   "k_s": wl.k_s, "parallelism": "single GPU"},
        "roofline": roofline,
        "detail": {
            n: {"ms_per_layer": round(r["ms_per_step"], 3), "median_ms_per_layer": round(r["median_ms_per_step"], 3),
                "wall_ms_per_layer": round(r["wall_ms_per_step"], 3),
                "stage_ms": {s: round(t, 3) for s, t in r["stage_ms"].items()},
                "fwd_tflops_kernel": round(r["fwd_flops"] / (r["stage_ms"]["fwd"] * 1e-3) / 1e12, 2),
                "bwd_tflops_kernel": round(2.5 * r["fwd_flops"] / (r["stage_ms"]["bwd"] * 1e-3) / 1e12, 2),
                "fwd_bwd_tflops_step": round(3.5 * r["fwd_flops"] / (r["ms_per_step"] * 1e-3) / 1e12, 2),
                "counted_tiles": int(r["T"]), "counted_col_pairs": int(r["C"]),
                "estimation_and_index": r["est_idx"],
                "tile_density_causal": round(r["density"], 4), "kernels": r["kernels"]}
            for n, r in results.items()},
    }
    line["detail"]["paper_context"] = PAPER_CONTEXT
    if args.ring and args.workload == "layer_512k":
        rw = WORKLOADS["ring_512k_w8"]
        print("[bench] ring share (worker 0 of 8, striped)", file=sys.stderr, flush=True)
        vi_t = torch.from_numpy(main_r["v_idx"]).to(dev)
        si_t = torch.from_numpy(main_r["s_idx"]).to(dev)
        line["detail"]["ring_512k_w8"] = ring_leg(main_r["x"], vi_t, si_t, rw, rw.world, 0, max(1, args.steps // 2))
        torch.cuda.empty_cache()
    if args.balance:
        print("[bench] ring balance sweep", file=sys.stderr, flush=True)
        line["detail"][f"{wl.name}_ring_balance"] = balance_leg(
            ms, torch, wl, torch.from_numpy(main_r["v_idx"]).to(dev), torch.from_numpy(main_r["s_idx"]).to(dev),
            [int(w) for w in args.balance.split(",")])
    if args.topp:
        print("[bench] top-p estimation", file=sys.stderr, flush=True)
        line["detail"][f"{wl.name}_topp"] = topp_leg(ms, torch, wl, main_r["x"],
                                                     [float(p) for p in args.topp.split(",")])
    if args.prefill:
        line["detail"]["prefill"] = {}
        for pname in args.prefill.split(","):
            pwl = WORKLOADS[pname]
            print(f"[bench] prefill {pname}", file=sys.stderr, flush=True)
            px = main_r["x"] if pname == wl.name else make_inputs(pwl, dev, with_do=False)
            line["detail"]["prefill"][pname] = prefill_leg(ms, torch, pwl, px, args.steps, args.warmup)
            if px is not main_r["x"]:
                del px
            torch.cuda.empty_cache()
    if not args.no_cpu:
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(wl, main_r["x"], main_r["v_idx"], main_r["s_idx"], args.cpu_rows)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
