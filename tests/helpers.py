"""Shared test plumbing: seeded inputs, oracle runs and GPU index extraction.

Inputs come only from synth/ (seeded generator); expected values only from
oracle/.  Tolerances follow the parity rules for this path: out / dQ / dK / dV
max-abs <= 2e-2 and mean-abs <= 2e-3 (bf16 inputs, fp32 accumulation); lse
max-abs <= 1e-3; index arrays bit-exact; estimated index sets equal except for
entries whose fp64 score lies within 1e-4 relative of the k-th score.
"""
from __future__ import annotations

import math

import numpy as np
import torch

from oracle import bf16 as OB
from oracle import estimate as OE
from oracle import index as OI
from synth import make_inputs, bf16_bits

MAX_ABS = 2e-2
MEAN_ABS = 2e-3
LSE_ABS = 1e-3
TOPK_REL = 1e-4


def to_f64(t: torch.Tensor) -> np.ndarray:
    return OB.to_f64(bf16_bits(t))


def inputs_f64(x: dict, names=("q", "k", "v", "do")) -> dict:
    return {n: to_f64(x[n]) for n in names if x.get(n) is not None}


def oracle_indices(f64: dict, wl, heads=None):
    """Reference (v_idx, s_idx, v_score, s_score) for every head (or the given heads)."""
    q, k = f64["q"], f64["k"]
    if heads is not None:
        G = q.shape[1] // k.shape[1]
        out = [OE.estimate(q[:, [h]], k[:, [h // G]], wl.last_q, wl.k_v, wl.k_s, 1 / math.sqrt(wl.head_dim))
               for h in heads]
        return tuple(np.concatenate([o[i] for o in out], axis=1) for i in range(4))
    return OE.estimate(q, k, wl.last_q, wl.k_v, wl.k_s, 1 / math.sqrt(wl.head_dim))


def oracle_sets_every_head(x: dict, wl) -> tuple[np.ndarray, np.ndarray]:
    """Each head's own (v_idx, s_idx) from the oracle's fp64 estimator (Alg. 1:
    the last last_q queries' column and diagonal sums, then the top k_v / k_s,
    lower index first), computed head by head from CPU copies of the inputs
    (which may live on the GPU)."""
    B, Hq, Hkv, N = wl.batch, wl.heads_q, wl.heads_kv, wl.seq
    G = Hq // Hkv
    scale = 1 / math.sqrt(wl.head_dim)
    vi = np.zeros((B, Hq, wl.k_v), np.int32)
    si = np.zeros((B, Hq, wl.k_s), np.int32)
    for b in range(B):
        for g in range(Hkv):
            k = to_f64(x["k"][b, g].cpu())
            for h in range(g * G, (g + 1) * G):
                vs, ss = OE.vs_scores(to_f64(x["q"][b, h, N - wl.last_q:].cpu()), k, scale)
                vi[b, h] = OE.topk_lower(vs, wl.k_v)
                si[b, h] = OE.topk_lower(ss, wl.k_s)
            del k
    return vi, si


def weighted_identity_check(x: dict, out32, dq, dk, dv, rel_tol: float) -> None:
    """Per KV group, the chain-rule identities of Eq. attention_backward on the
    GPU's own outputs (fp64 sums on the device): sum_j dK_j . k_j equals the sum
    of dQ_i . q_i over the group's heads and rows, and sum_j dV_j . v_j the sum
    of dO_i . O_i.  Unlike sum dK = 0 and sum dV = sum dO, they weight each
    key's gradient by that key's own row, so gradients accumulated into the
    wrong keys (systematically) break them.  The bar is relative to the sum of
    the terms' magnitudes."""
    B, Hq = x["q"].shape[:2]
    Hkv = x["k"].shape[1]
    G = Hq // Hkv
    for b in range(B):
        for g in range(Hkv):
            kk, vv = x["k"][b, g].double(), x["v"][b, g].double()
            dkk, dvv = dk[b, g].double() * kk, dv[b, g].double() * vv
            tk, tv = float(dkk.sum()), float(dvv.sum())
            mk, mv = float(dkk.abs().sum()), float(dvv.abs().sum())
            del kk, vv, dkk, dvv
            tq = to = 0.0
            for h in range(g * G, (g + 1) * G):
                a = dq[b, h].double() * x["q"][b, h].double()
                c = x["do"][b, h].double() * out32[b, h].double()
                tq += float(a.sum())
                to += float(c.sum())
                mk += float(a.abs().sum())
                mv += float(c.abs().sum())
                del a, c
            print(f"identities b{b} kv{g}: dK.k - dQ.q = {tk - tq:.3e} (rel {abs(tk - tq) / mk:.2e}), "
                  f"dV.v - dO.O = {tv - to:.3e} (rel {abs(tv - to) / mv:.2e})", flush=True)
            assert abs(tk - tq) <= rel_tol * mk, f"dK.k identity b{b} kv{g}"
            assert abs(tv - to) <= rel_tol * mv, f"dV.v identity b{b} kv{g}"


def gpu_csr(idx) -> dict:
    """Copy a GPU SparseIndex to host arrays trimmed to their used lengths."""
    t = {k: v.cpu().numpy() for k, v in idx.tensors.items()}
    nb = int(t["blk_ptr"][-1])
    nc = int(t["col_ptr"][-1])
    nv = int(t["vcol_ptr"][-1])
    return dict(blk_ptr=t["blk_ptr"], blk_idx=t["blk_idx"][:nb], col_ptr=t["col_ptr"], col_idx=t["col_idx"][:nc],
                kblk_ptr=t["kblk_ptr"], kblk_idx=t["kblk_idx"][:nb], vcol_ptr=t["vcol_ptr"],
                vcol_idx=t["vcol_idx"][:nv], diag_bits=t["diag_bits"].view(np.uint32),
                q_blk_global=t["q_blk_global"], k_blk_global=t["k_blk_global"])


def head_csr(c: dict, bh: int, nqb: int, nkb: int) -> dict:
    """Per-head slices of a CSR dict (offsets rebased to 0)."""
    def seg(ptr, idx, n):
        p = ptr[bh * n: bh * n + n + 1]
        return p - p[0], idx[p[0]:p[-1]]
    bp, bi = seg(c["blk_ptr"], c["blk_idx"], nqb)
    cp, ci = seg(c["col_ptr"], c["col_idx"], nqb)
    kp, ki = seg(c["kblk_ptr"], c["kblk_idx"], nkb)
    vp, vi = seg(c["vcol_ptr"], c["vcol_idx"], 1)
    return dict(blk_ptr=bp, blk_idx=bi, col_ptr=cp, col_idx=ci, kblk_ptr=kp, kblk_idx=ki, vcol_ptr=vp, vcol_idx=vi)


def assert_close(name, got, ref, max_abs=MAX_ABS, mean_abs=MEAN_ABS):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    err = np.abs(got - ref)
    assert np.isfinite(err).all(), f"{name}: non-finite difference"
    assert err.max() <= max_abs and err.mean() <= mean_abs, \
        f"{name}: max-abs {err.max():.3e} mean-abs {err.mean():.3e}"


def assert_lse_close(got, ref, tol=LSE_ABS):
    got = np.asarray(got, dtype=np.float64)
    inf_r = np.isneginf(ref)
    assert (np.isneginf(got) == inf_r).all(), "lse -inf pattern differs"
    err = np.abs(got[~inf_r] - ref[~inf_r])
    assert err.size == 0 or err.max() <= tol, f"lse max-abs {err.max():.3e}"


def assert_topk_match(got, ref, score, k, rel=TOPK_REL):
    """Sets equal except entries within `rel` of the oracle's k-th score."""
    order = np.sort(score)[::-1]
    t_k = order[k - 1]
    diff = np.setxor1d(np.asarray(got), np.asarray(ref))
    bad = diff[np.abs(score[diff] - t_k) > rel * abs(t_k)]
    assert bad.size == 0, f"{bad.size} index differences outside the tie band (t_k={t_k:.6e})"
    assert len(np.unique(got)) == k and np.all(np.diff(got) > 0)


TOPP_MASS_REL = 1e-4


def budget_fixed_point(score32, p: float) -> int:
    """score_cover (Algorithm 1) taken in the kernel's precision, so that the GPU's
    budget can be checked exactly on its own scores: every fp32 score x counts
    floor(x 2^40) (exact integers, summed in any order), the threshold is
    ceil(p T) rounded in fp64, and k is the first count of the descending list
    whose cumulative mass reaches it."""
    x = np.asarray(score32, dtype=np.float32).astype(np.float64)
    q = np.floor(x * 2.0 ** 40).astype(np.int64)
    theta = math.ceil(p * float(int(q.sum())))
    order = np.lexsort((np.arange(x.size), -x))
    c = np.cumsum(q[order])
    return int(np.searchsorted(c, theta, side="left")) + 1


def assert_budget_near(cnt: int, score, p: float, kmax: int, rel=TOPP_MASS_REL):
    """The budget against the oracle's fp64 scores: the mass of the cnt largest
    reaches p of the total and that of the cnt - 1 largest stays below it, both
    within `rel` of the threshold (a cap at kmax only needs the second)."""
    srt = np.sort(np.asarray(score, dtype=np.float64))[::-1]
    c = np.cumsum(srt)
    theta = p * c[-1]
    assert 1 <= cnt <= kmax
    if cnt < kmax:
        assert c[cnt - 1] >= theta * (1 - rel), f"mass {c[cnt - 1]:.6e} below p of the total {theta:.6e}"
    assert cnt == 1 or c[cnt - 2] < theta * (1 + rel), f"cnt {cnt} larger than needed"


def assert_close_rows(name, got, ref, max_abs=MAX_ABS, mean_abs=MEAN_ABS):
    """The parity bars per row, in units of max(1, RMS of that row of the
    reference): a row built from inputs scaled far from unity (an outlier value
    row of size 2^10, say) carries rounding errors proportional to its own
    size, so the absolute bars apply relative to each row's magnitude."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    unit = np.maximum(1.0, np.sqrt(np.mean(ref ** 2, axis=-1, keepdims=True)))
    err = np.abs(got - ref) / unit
    assert np.isfinite(err).all(), f"{name}: non-finite difference"
    assert err.max() <= max_abs and err.mean() <= mean_abs, \
        f"{name}: row-scaled max-abs {err.max():.3e} mean-abs {err.mean():.3e}"


def _head_reference(job):
    """Full oracle forward and backward of one query head (a process-pool worker)."""
    q, k, v, do, vi, si, N, scale, threads = job
    from threadpoolctl import threadpool_limits
    from oracle import attn as OA_
    with threadpool_limits(threads):
        idx = OI.Index(vi, si, N)
        o, lse = OA_.layer_fwd(q, k, v, idx, scale)
        dq, dk, dv = OA_.layer_bwd(q, k, v, do, idx, scale)
    return o[0, 0], lse[0, 0], dq[0, 0], dk[0, 0], dv[0, 0]


def oracle_heads(f: dict, vi, si, heads, scale, workers=8, threads=2):
    """The oracle's out, lse, dQ and the per-head dK, dV contributions of the
    given query heads (batch 0), one head per worker process (spawned, so no
    GPU state is inherited): {h: (out, lse, dq, dk_h, dv_h)}."""
    import multiprocessing as mp
    q, k = f["q"], f["k"]
    G = q.shape[1] // k.shape[1]
    N = q.shape[2]
    jobs = [(q[:1, [h]], k[:1, [h // G]], f["v"][:1, [h // G]], f["do"][:1, [h]], vi[:1, [h]], si[:1, [h]], N,
             scale, threads) for h in heads]
    with mp.get_context("spawn").Pool(min(workers, len(jobs))) as pool:
        res = pool.map(_head_reference, jobs)
    return dict(zip(heads, res))
