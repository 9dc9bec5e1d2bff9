"""Reference masked attention forward / backward and the partial-result merge.

Test infrastructure; see oracle/__init__.py.  All arithmetic is fp64.

For one query head with executed mask M (a boolean [rows, keys] array, see
index.Index.mask_rows), scale = 1 / sqrt(d):

  forward   z = scale * Q K^T, masked entries -inf (additive mask);
            lse_n = log sum_{m in M_n} exp(z[n, m]);  A = exp(z - lse);
            O = A V.  A row with no visible key gives O = 0 and lse = -inf.
  backward  (Eq. softmax_gradient and Eq. attention_backward)
            dV = A^T dO;  dA = dO V^T;
            dZ = A o (dA - rowsum(dA o A));
            dQ = scale * dZ K;  dK = scale * dZ^T Q.
            The index is a constant: no gradient flows into the estimator.
  GQA       query head h reads KV head h // (Hq / Hkv); dK and dV of a KV head
            are the sums over its query heads.
  merge     (merge_out_and_lse of Algorithm 2) two partial results over disjoint
            key sets combine as lse = logaddexp(lse1, lse2),
            O = exp(lse1 - lse) O1 + exp(lse2 - lse) O2.
"""
import numpy as np

ROW_CHUNK = 512


def head_fwd(q, k, v, mask, scale):
    """q [R, d], k/v [Nk, d], mask [R, Nk] -> out [R, d], lse [R]."""
    z = np.where(mask, scale * (q @ k.T), -np.inf)
    zmax = z.max(axis=1)
    empty = ~np.isfinite(zmax)
    ref = np.where(empty, 0.0, zmax)
    e = np.exp(z - ref[:, None])
    s = e.sum(axis=1)
    with np.errstate(divide="ignore", invalid="ignore"):
        lse = np.where(empty, -np.inf, ref + np.log(s))
        out = np.where(empty[:, None], 0.0, (e @ v) / s[:, None])
    return out, lse


def head_probs(q, k, mask, scale):
    _, lse = head_fwd(q, k, np.zeros((k.shape[0], 1)), mask, scale)
    z = np.where(mask, scale * (q @ k.T), -np.inf)
    with np.errstate(invalid="ignore"):
        a = np.exp(z - np.where(np.isfinite(lse), lse, 0.0)[:, None])
    return np.where(mask, a, 0.0)


def head_bwd(q, k, v, do, mask, scale):
    """Gradients of one head over the rows given (all rows for dK / dV)."""
    a = head_probs(q, k, mask, scale)
    dv = a.T @ do
    da = do @ v.T
    dz = a * (da - (da * a).sum(axis=1, keepdims=True))
    dq = scale * (dz @ k)
    dk = scale * (dz.T @ q)
    return dq, dk, dv


def seen_keys(mask):
    """Keys that some row of the mask sees.  A masked entry has weight exactly
    0 (additive -inf before the softmax), so leaving out keys that no row of a
    chunk sees changes no sum; it only skips work."""
    return np.flatnonzero(mask.any(axis=0))


def layer_fwd(q, k, v, index, scale, rows=None):
    """q [B, Hq, Nq, d], k/v [B, Hkv, Nk, d] fp64 -> out [B, Hq, R, d], lse [B, Hq, R].

    rows: local query rows to evaluate (default all), each from its own mask row.
    """
    B, Hq, Nq, d = q.shape
    G = Hq // k.shape[1]
    rows = np.arange(Nq) if rows is None else np.asarray(rows)
    out = np.zeros((B, Hq, len(rows), d))
    lse = np.zeros((B, Hq, len(rows)))
    for b in range(B):
        for h in range(Hq):
            bh = b * Hq + h
            for c0 in range(0, len(rows), ROW_CHUNK):
                rr = rows[c0:c0 + ROW_CHUNK]
                M = index.mask_rows(bh, rr)
                sk = seen_keys(M)
                o, l = head_fwd(q[b, h, rr], k[b, h // G][sk], v[b, h // G][sk], M[:, sk], scale)
                out[b, h, c0:c0 + len(rr)] = o
                lse[b, h, c0:c0 + len(rr)] = l
    return out, lse


def layer_dq(q, k, v, do, index, scale, rows):
    """dQ of the given local query rows only (a row's dQ needs only that row)."""
    B, Hq, Nq, d = q.shape
    G = Hq // k.shape[1]
    rows = np.asarray(rows)
    dq = np.zeros((B, Hq, len(rows), d))
    for b in range(B):
        for h in range(Hq):
            M = index.mask_rows(b * Hq + h, rows)
            sk = seen_keys(M)
            dq[b, h] = head_bwd(q[b, h, rows], k[b, h // G][sk], v[b, h // G][sk], do[b, h, rows], M[:, sk],
                                scale)[0]
    return dq


def layer_bwd(q, k, v, do, index, scale):
    """Full dQ [B,Hq,Nq,d], dK, dV [B,Hkv,Nk,d]; rows processed in chunks."""
    B, Hq, Nq, d = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for b in range(B):
        for h in range(Hq):
            for c0 in range(0, Nq, ROW_CHUNK):
                rr = np.arange(c0, min(Nq, c0 + ROW_CHUNK))
                M = index.mask_rows(b * Hq + h, rr)
                sk = seen_keys(M)
                gq, gk, gv = head_bwd(q[b, h, rr], k[b, h // G][sk], v[b, h // G][sk], do[b, h, rr], M[:, sk],
                                      scale)
                dq[b, h, rr] = gq
                dk[b, h // G, sk] += gk
                dv[b, h // G, sk] += gv
    return dq, dk, dv


def merge(o1, lse1, o2, lse2):
    """Log-sum-exp merge of two partial (O, lse) pairs over disjoint key sets."""
    lse = np.logaddexp(lse1, lse2)
    safe = np.where(np.isfinite(lse), lse, 0.0)
    w1 = np.where(np.isfinite(lse1), np.exp(lse1 - safe), 0.0)
    w2 = np.where(np.isfinite(lse2), np.exp(lse2 - safe), 0.0)
    return w1[..., None] * o1 + w2[..., None] * o2, lse
