"""Pins for the reference attention: a library masked SDPA with autograd (fp64),
finite differences, brute-force loops, invariants, empty rows and the ring merge."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import attn as A
from oracle import index as I


def _case(seed, B=1, Hq=4, Hkv=2, N=256, d=16, nv=6, ns=9):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, Hq, N, d))
    k = rng.standard_normal((B, Hkv, N, d))
    v = rng.standard_normal((B, Hkv, N, d))
    do = rng.standard_normal((B, Hq, N, d))
    V = np.stack([np.stack([np.sort(rng.choice(N, nv, replace=False)) for _ in range(Hq)]) for _ in range(B)])
    S = np.stack([np.stack([np.sort(np.concatenate([[0], rng.choice(np.arange(1, N), ns - 1, replace=False)]))
                            for _ in range(Hq)]) for _ in range(B)])
    return q, k, v, do, I.Index(V, S, N)


def _sdpa(q, k, v, do, idx, scale):
    B, Hq, N, d = q.shape
    G = Hq // k.shape[1]
    mask = torch.stack([torch.stack([torch.from_numpy(idx.mask_rows(b * Hq + h, np.arange(N)))
                                     for h in range(Hq)]) for b in range(B)])
    tq, tk, tv = (torch.from_numpy(x).requires_grad_() for x in (q, k, v))
    o = F.scaled_dot_product_attention(tq, tk.repeat_interleave(G, 1), tv.repeat_interleave(G, 1),
                                       attn_mask=mask, scale=scale)
    o.backward(torch.from_numpy(do))
    return o.detach().numpy(), tq.grad.numpy(), tk.grad.numpy(), tv.grad.numpy()


@pytest.mark.parametrize("seed", [0, 1])
def test_against_library_sdpa(seed):
    q, k, v, do, idx = _case(seed)
    scale = 1 / math.sqrt(q.shape[-1])
    out, lse = A.layer_fwd(q, k, v, idx, scale)
    dq, dk, dv = A.layer_bwd(q, k, v, do, idx, scale)
    o2, dq2, dk2, dv2 = _sdpa(q, k, v, do, idx, scale)
    for a, b in ((out, o2), (dq, dq2), (dk, dk2), (dv, dv2)):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-11)


def test_full_budget_equals_dense_causal():
    rng = np.random.default_rng(4)
    B, Hq, Hkv, N, d = 1, 2, 1, 192, 8
    q, k, v, do = (rng.standard_normal(s) for s in [(B, Hq, N, d), (B, Hkv, N, d), (B, Hkv, N, d), (B, Hq, N, d)])
    idx = I.Index(np.zeros((B, Hq, 1), np.int64), np.tile(np.arange(N), (B, Hq, 1)), N)
    out, lse = A.layer_fwd(q, k, v, idx, 0.4)
    dq, dk, dv = A.layer_bwd(q, k, v, do, idx, 0.4)
    tq, tk, tv = (torch.from_numpy(x).requires_grad_() for x in (q, k, v))
    o = F.scaled_dot_product_attention(tq, tk.repeat_interleave(2, 1), tv.repeat_interleave(2, 1),
                                       is_causal=True, scale=0.4)
    o.backward(torch.from_numpy(do))
    np.testing.assert_allclose(out, o.detach().numpy(), atol=1e-12)
    np.testing.assert_allclose(dq, tq.grad.numpy(), atol=1e-12)
    np.testing.assert_allclose(dk, tk.grad.numpy(), atol=1e-12)
    np.testing.assert_allclose(dv, tv.grad.numpy(), atol=1e-12)
    # lse of the dense causal row is a log-sum-exp over m <= n
    z = 0.4 * q[0, 0] @ k[0, 0].T
    n = 150
    assert abs(lse[0, 0, n] - math.log(np.exp(z[n, :n + 1]).sum())) < 1e-12


def test_brute_force_loops_tiny():
    q, k, v, do, idx = _case(5, B=1, Hq=1, Hkv=1, N=128, d=4, nv=3, ns=4)
    scale = 0.5
    out, lse = A.layer_fwd(q, k, v, idx, scale)
    M = idx.mask_rows(0, np.arange(128))
    for n in range(0, 128, 7):
        ms = [m for m in range(128) if M[n, m]]
        zs = [scale * sum(q[0, 0, n, t] * k[0, 0, m, t] for t in range(4)) for m in ms]
        mx = max(zs)
        w = [math.exp(z - mx) for z in zs]
        s = sum(w)
        assert abs(lse[0, 0, n] - (mx + math.log(s))) < 1e-12
        for t in range(4):
            o = sum(wi * v[0, 0, m, t] for wi, m in zip(w, ms)) / s
            assert abs(out[0, 0, n, t] - o) < 1e-12


def test_finite_differences():
    q, k, v, do, idx = _case(6, B=1, Hq=2, Hkv=1, N=128, d=4, nv=3, ns=5)
    scale = 0.7
    dq, dk, dv = A.layer_bwd(q, k, v, do, idx, scale)

    def loss(q_, k_, v_):
        return float((A.layer_fwd(q_, k_, v_, idx, scale)[0] * do).sum())

    eps = 1e-6
    rng = np.random.default_rng(0)
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        for _ in range(4):
            pos = tuple(int(rng.integers(0, s)) for s in x.shape)
            xp, xm = x.copy(), x.copy()
            xp[pos] += eps
            xm[pos] -= eps
            args = {"q": (q, k, v), "k": (q, k, v), "v": (q, k, v)}[name]
            ap = [xp if a is x else a for a in args]
            am = [xm if a is x else a for a in args]
            fd = (loss(*ap) - loss(*am)) / (2 * eps)
            assert abs(fd - g[pos]) <= 1e-6 * max(1.0, abs(g[pos])), (name, pos, fd, g[pos])


def test_stochastic_rows_and_invariants():
    q, k, v, do, idx = _case(8)
    scale = 0.25
    P = A.head_probs(q[0, 1], k[0, 0], idx.mask_rows(1, np.arange(256)), scale)
    np.testing.assert_allclose(P.sum(axis=1), 1.0, atol=1e-13)
    dq, dk, dv = A.layer_bwd(q, k, v, do, idx, scale)
    np.testing.assert_allclose(dk.sum(axis=2), 0.0, atol=1e-11)
    np.testing.assert_allclose(dv.sum(axis=2)[0, 0], do[0, 0:2].sum(axis=(0, 1)), atol=1e-11)


def weighted_gradient_residuals(q, k, v, do, out, dq, dk, dv):
    """Per KV group g, the two identities that follow from the chain rule of
    Eq. attention_backward (S = scale Q K^T, O = P V):
      sum_j dK_j . k_j = sum over the group's heads and rows of dQ_i . q_i
        (both equal sum_ij dS_ij S_ij), and
      sum_j dV_j . v_j = sum over the group's heads and rows of dO_i . O_i.
    Returns [(residual_k, magnitude_k, residual_v, magnitude_v)] per (b, g)."""
    B, Hq = q.shape[:2]
    Hkv = k.shape[1]
    G = Hq // Hkv
    res = []
    for b in range(B):
        for g in range(Hkv):
            hs = slice(g * G, (g + 1) * G)
            tk, tq = (dk[b, g] * k[b, g]).sum(), (dq[b, hs] * q[b, hs]).sum()
            tv, to = (dv[b, g] * v[b, g]).sum(), (do[b, hs] * out[b, hs]).sum()
            mk = np.abs(dk[b, g] * k[b, g]).sum() + np.abs(dq[b, hs] * q[b, hs]).sum()
            mv = np.abs(dv[b, g] * v[b, g]).sum() + np.abs(do[b, hs] * out[b, hs]).sum()
            res.append((tk - tq, mk, tv - to, mv))
    return res


def test_weighted_gradient_identities():
    """The oracle's gradients satisfy both identities to rounding, and a dK or
    dV row added to the wrong key (a misrouted partial) breaks them."""
    q, k, v, do, idx = _case(21)
    scale = 0.3
    out, _ = A.layer_fwd(q, k, v, idx, scale)
    dq, dk, dv = A.layer_bwd(q, k, v, do, idx, scale)
    for rk, mk, rv, mv in weighted_gradient_residuals(q, k, v, do, out, dq, dk, dv):
        assert abs(rk) <= 1e-12 * mk and abs(rv) <= 1e-12 * mv
    for name in ("dk", "dv"):
        bad = {"dk": dk.copy(), "dv": dv.copy()}
        t = bad[name]
        t[0, 1, 200] += t[0, 1, 37]       # key 37's gradient moved to key 200
        t[0, 1, 37] = 0.0
        r = weighted_gradient_residuals(q, k, v, do, out, dq, bad["dk"], bad["dv"])[1]
        rel = abs(r[0]) / r[1] if name == "dk" else abs(r[2]) / r[3]
        assert rel > 1e-3, (name, rel)


def test_empty_row():
    # no slash at the diagonal and no vertical in the first block: rows of block 0 see nothing
    N, d = 128, 4
    rng = np.random.default_rng(9)
    q, k, v, do = (rng.standard_normal((1, 1, N, d)) for _ in range(4))
    idx = I.Index(np.array([[[100]]]), np.array([[[70]]]), N)
    out, lse = A.layer_fwd(q, k, v, idx, 0.5)
    assert np.all(out[0, 0, :64] == 0) and np.all(np.isneginf(lse[0, 0, :64]))
    dq, dk, dv = A.layer_bwd(q, k, v, do, idx, 0.5)
    assert np.all(dq[0, 0, :64] == 0)
    assert np.isfinite(dk).all() and np.isfinite(dv).all()


@pytest.mark.parametrize("layout,W", [("striped", 2), ("striped", 4), ("zigzag", 2)])
def test_ring_merge_equals_single_pass(layout, W):
    rng = np.random.default_rng(13)
    N, d, Hq, Hkv = 1024, 8, 2, 1
    nb = N // 64
    q, k, v = (rng.standard_normal((1, h, N, d)) for h in (Hq, Hkv, Hkv))
    V = np.stack([np.sort(rng.choice(N, 12, replace=False)) for _ in range(Hq)])[None]
    S = np.stack([np.sort(rng.choice(N, 20, replace=False)) for _ in range(Hq)])[None]
    whole = I.Index(V, S, N)
    ref_o, ref_l = A.layer_fwd(q, k, v, whole, 0.3)
    for r in range(W):
        qg = I.local_blocks(r, nb, W, layout)
        rows = (qg[:, None] * 64 + np.arange(64)[None]).reshape(-1)
        o = np.zeros((1, Hq, len(rows), d))
        l = np.full((1, Hq, len(rows)), -np.inf)
        for t in range(W):
            st = I.Index(V, S, N, world=W, rank=r, step=t, layout=layout)
            kg = st.k_blk_global
            krows = (kg[:, None] * 64 + np.arange(64)[None]).reshape(-1)
            po, pl = A.layer_fwd(q[:, :, rows], k[:, :, krows], v[:, :, krows], st, 0.3)
            o, l = A.merge(o, l, po, pl)
        np.testing.assert_allclose(o, ref_o[:, :, rows], atol=1e-12)
        np.testing.assert_allclose(l, ref_l[:, :, rows], atol=1e-12)


def test_merge_with_empty_partial():
    rng = np.random.default_rng(2)
    o = rng.standard_normal((3, 4))
    l = rng.standard_normal(3)
    mo, ml = A.merge(o, l, np.zeros((3, 4)), np.full(3, -np.inf))
    np.testing.assert_array_equal(ml, l)
    np.testing.assert_allclose(mo, o, atol=0)


# ---- layer_dq: dQ of sampled rows only (Eq. attention_backward restricted to
# those rows; a row's dQ needs only that row's probabilities and gradients)
def test_layer_dq_equals_full_backward_rows():
    q, k, v, do, idx = _case(21, B=2, Hq=4, Hkv=2, N=256, d=8, nv=7, ns=6)
    scale = 0.35
    dq_full = A.layer_bwd(q, k, v, do, idx, scale)[0]
    rows = np.array([255, 3, 64, 63, 130, 0, 191, 64])     # unsorted, with a repeat
    dq = A.layer_dq(q[:, :, rows], k, v, do[:, :, rows], _RowsOf(idx, rows), scale, np.arange(len(rows)))
    np.testing.assert_allclose(dq, dq_full[:, :, rows], rtol=0, atol=1e-12)


class _RowsOf:
    """An index whose mask row r is row rows[r] of `idx` (the sampled-row form
    the full-size tests hand to the oracle)."""

    def __init__(self, idx, rows):
        self.idx, self.rows = idx, np.asarray(rows)

    def mask_rows(self, bh, rr):
        return self.idx.mask_rows(bh, self.rows[np.asarray(rr)])


def test_layer_dq_brute_force_loops():
    # dQ_n = scale sum_m P[n,m] (dO_n . v_m - dO_n . O_n) k_m over the executed
    # keys, written as plain loops; Delta is taken as dO . O here (the oracle
    # uses the row sum of dA o A: the two agree only if the code is right)
    q, k, v, do, idx = _case(22, B=1, Hq=2, Hkv=1, N=128, d=4, nv=3, ns=4)
    scale = 0.6
    rows = np.array([0, 1, 17, 63, 64, 100, 127])
    dq = A.layer_dq(q, k, v, do, idx, scale, rows)
    for h in range(2):
        M = idx.mask_rows(h, np.arange(128))
        for r, n in enumerate(rows.tolist()):
            ms = [m for m in range(128) if M[n, m]]
            z = [scale * sum(q[0, h, n, t] * k[0, 0, m, t] for t in range(4)) for m in ms]
            mx = max(z)
            w = [math.exp(zz - mx) for zz in z]
            s = sum(w)
            p = [wi / s for wi in w]
            o = [sum(pi * v[0, 0, m, t] for pi, m in zip(p, ms)) for t in range(4)]
            delta = sum(do[0, h, n, t] * o[t] for t in range(4))
            for t in range(4):
                want = scale * sum(pi * (sum(do[0, h, n, u] * v[0, 0, m, u] for u in range(4)) - delta)
                                   * k[0, 0, m, t] for pi, m in zip(p, ms))
                assert abs(dq[0, h, r, t] - want) < 1e-12, (h, n, t, dq[0, h, r, t], want)


def test_layer_dq_finite_differences():
    # d/dq_n of sum over the sampled rows of O o dO, one row's forward at a time
    q, k, v, do, idx = _case(23, B=1, Hq=2, Hkv=1, N=128, d=4, nv=3, ns=5)
    scale = 0.8
    rows = np.array([5, 70, 127])
    dq = A.layer_dq(q, k, v, do, idx, scale, rows)

    def loss(q_):
        return float((A.layer_fwd(q_, k, v, idx, scale, rows=rows)[0] * do[:, :, rows]).sum())

    eps = 1e-6
    for h in range(2):
        for r, n in enumerate(rows.tolist()):
            for t in range(4):
                qp, qm = q.copy(), q.copy()
                qp[0, h, n, t] += eps
                qm[0, h, n, t] -= eps
                fd = (loss(qp) - loss(qm)) / (2 * eps)
                assert abs(fd - dq[0, h, r, t]) <= 1e-6 * max(1.0, abs(fd)), (h, n, t, fd, dq[0, h, r, t])


def test_layer_dq_empty_row_is_zero():
    N, d = 128, 4
    rng = np.random.default_rng(24)
    q, k, v, do = (rng.standard_normal((1, 1, N, d)) for _ in range(4))
    idx = I.Index(np.array([[[100]]]), np.array([[[70]]]), N)   # block 0 sees nothing
    dq = A.layer_dq(q, k, v, do, idx, 0.5, np.array([0, 40, 63, 64, 127]))
    assert np.all(dq[0, 0, :3] == 0)
    assert np.abs(dq[0, 0, 3:]).max() > 0
