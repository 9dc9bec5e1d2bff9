"""Benchmark of the vertical-slash sparse-attention hot path on one MI355X.

A step is one pass of the whole path over one synthetic layer already resident
in HBM: pattern estimation -> index count (one GPU wait) and build -> sparse
forward -> sparse backward.  The metric is fwd+bwd TFLOP/s on the computed
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


def kernel_flops(name: str, d: int, T: int, C: int, BH: int, N: int) -> float:
    """MFMA GEMM work each kernel must do on the computed blocks / columns."""
    pair = 2.0 * d            # one multiply-add over d per (row, key) per GEMM
    tiles = 4096.0 * T + 64.0 * C
    return {
        "attn_fwd": 2 * pair * tiles,                 # S, PV
        "bwd_dq": 3 * pair * tiles,                   # S, dP, dQ
        "bwd_dkdv": 4 * pair * 4096.0 * T,            # S, dP, dV, dK on tiles
        "bwd_dkdv_col": 4 * pair * 64.0 * C,          # the same on column pairs
        "est_pass1": pair * 64.0 * N * BH,            # last 64 rows x all keys
        "est_pass2": pair * 64.0 * N * BH,
    }.get(name, 0.0)


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
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{len(rows)} query rows of head 0 of {wl.name}: fp64 dense-masked forward and dQ, "
                      f"{dt:.1f} s"}


def torch_index(rows):
    import torch
    return torch.from_numpy(rows)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="layer_512k")
    ap.add_argument("--also", default="layer_128k", help="second workload timed the same way ('' to skip)")
    ap.add_argument("--cpu-rows", type=int, default=64)
    ap.add_argument("--no-cpu", action="store_true")
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
        state = {}

        def step(timed):
            def mark(stage, i):
                if timed:
                    ev[stage][i].record()
            mark("estimate", 0)
            ms.estimate(dims, q, k, wl.last_q, wl.k_v, wl.k_s, v_idx, s_idx, workspace=est_ws)
            mark("estimate", 1)
            mark("index", 0)
            blk, col, vcol = ms.index_count(dims, v_idx, s_idx, workspace=idx_ws)
            if state.get("caps", (0, 0, 0))[0] < blk or state["caps"][1] < col or state["caps"][2] < vcol:
                state["caps"] = (int(blk * 1.05) + 64, int(col * 1.05) + 64, vcol)
                state["idx"] = ms.alloc_index(dims, *state["caps"], dev)
            idx = state["idx"]
            ms.build_index(dims, v_idx, s_idx, idx, workspace=idx_ws)
            mark("index", 1)
            mark("fwd", 0)
            ms.attn_fwd(dims, q, k, v, idx, out=out, lse=lse, out_f32=out32, workspace=fwd_ws)
            mark("fwd", 1)
            mark("bwd", 0)
            ms.attn_bwd(dims, q, k, v, out, do, lse, idx, dq, dk, dv, out_f32=out32, workspace=bwd_ws)
            mark("bwd", 1)
            state["nnz"] = (blk, col)
            if timed:
                torch.cuda.synchronize()
                for s, (a, b) in ev.items():
                    acc[s] += a.elapsed_time(b)

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
            per_kernel[kname] = {"launches_per_step": n / args.steps, "avg_ms": round(avg, 4),
                                 "tflops": round(fl / (avg * 1e-3) / 1e12, 2) if fl else None}
        nb = N // 64
        results[name] = dict(
            wl=wl, ms_per_step=ms_step, wall_ms_per_step=wall, stage_ms=step_ms, kernels=per_kernel,
            fwd_flops=fwd_flops, T=T, C=C,
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
    achieved = dk_["tflops"] if dk_["tflops"] is not None else 0.0
    roofline = {"bound": "mfma", "kernel": dom, "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": None}
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
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": wl.batch, "seq_len": wl.seq, "heads_q": wl.heads_q,
                   "heads_kv": wl.heads_kv, "head_dim": wl.head_dim, "last_q": wl.last_q, "k_v": wl.k_v,
                   "k_s": wl.k_s, "parallelism": "single GPU"},
        "roofline": roofline,
        "detail": {
            n: {"ms_per_layer": round(r["ms_per_step"], 3), "stage_ms": {s: round(t, 3) for s, t in r["stage_ms"].items()},
                "fwd_tflops_kernel": round(r["fwd_flops"] / (r["stage_ms"]["fwd"] * 1e-3) / 1e12, 2),
                "bwd_tflops_kernel": round(2.5 * r["fwd_flops"] / (r["stage_ms"]["bwd"] * 1e-3) / 1e12, 2),
                "fwd_bwd_tflops_step": round(3.5 * r["fwd_flops"] / (r["ms_per_step"] * 1e-3) / 1e12, 2),
                "counted_tiles": int(r["T"]), "counted_col_pairs": int(r["C"]),
                "tile_density_causal": round(r["density"], 4), "kernels": r["kernels"]}
            for n, r in results.items()},
    }
    if not args.no_cpu:
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(wl, main_r["x"], main_r["v_idx"], main_r["s_idx"], args.cpu_rows)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
