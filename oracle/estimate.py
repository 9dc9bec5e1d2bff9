"""Reference vertical-slash pattern estimator (test infrastructure; see oracle/__init__.py).

Algorithm 1 of the paper, on one GPU (no broadcast or gather), per batch b and
query head h, with G = Hq / Hkv and KV head h // G:

  1. Q_last = the last L query rows, positions n in R = {N - L, ..., N - 1}.
  2. Scores z[n, m] = scale * q_n . k_m, with the causal mask applied additively
     (m > n gets -inf; the paper writes the mask as a product, read here as the
     usual additive mask before the softmax).
  3. Row-wise softmax over all causal keys of the whole sequence:
     P[n, m] = exp(z[n, m] - lse_n), lse_n = log sum_{m <= n} exp(z[n, m]).
  4. Vertical scores: v_score[m] = sum_{n in R} P[n, m]            (sum_v).
  5. Slash scores:    s_score[delta] = sum_{n in R, n >= delta} P[n, n - delta],
     delta = n - m the distance below the main diagonal            (sum_s).
  6. i_v = the k_v largest v_score, i_s = the k_s largest s_score (argtopk with a
     fixed budget); equal scores are broken by the lower index; both are
     returned in ascending order.

The online top-p budget (score_cover of Algorithm 1) replaces the fixed k_v,
k_s of step 6 by the smallest count whose largest scores reach a fraction p of
the list's total attention mass (the total is L for both lists: every observed
softmax row sums to 1 and each of its entries lies in exactly one column and
one diagonal).  The paper prints no value of p; the caller gives p and a cap.
"""
import numpy as np


def vs_scores(q_last: np.ndarray, k: np.ndarray, scale: float):
    """Steps 2-5 for one head.  q_last [L, d] (rows N-L..N-1), k [N, d], fp64."""
    L = q_last.shape[0]
    N = k.shape[0]
    rows = np.arange(N - L, N)
    z = scale * (q_last @ k.T)                                   # [L, N]
    causal = np.arange(N)[None, :] <= rows[:, None]
    z = np.where(causal, z, -np.inf)
    zmax = z.max(axis=1, keepdims=True)
    lse = zmax + np.log(np.exp(z - zmax).sum(axis=1, keepdims=True))
    p = np.exp(z - lse)                                          # masked -> 0
    v_score = p.sum(axis=0)
    s_score = np.zeros(N)
    for r, n in enumerate(rows):
        # row n touches delta = n - m for m = 0..n; delta runs n..0 as m runs 0..n
        s_score[: n + 1] += p[r, : n + 1][::-1]
    return v_score, s_score


def topk_lower(score: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k largest scores, ties to the lower index, ascending."""
    n = score.shape[0]
    order = np.lexsort((np.arange(n), -score))      # by -score, then by index
    return np.sort(order[:k]).astype(np.int32)


def estimate(q: np.ndarray, k: np.ndarray, last_q: int, k_v: int, k_s: int, scale: float):
    """Whole-layer estimator.  q [B, Hq, N, d], k [B, Hkv, N, d] fp64.

    Returns v_idx [B, Hq, k_v], s_idx [B, Hq, k_s] (int32, ascending) and
    v_score, s_score [B, Hq, N] (fp64).
    """
    B, Hq, N, d = q.shape
    G = Hq // k.shape[1]
    v_idx = np.zeros((B, Hq, k_v), np.int32)
    s_idx = np.zeros((B, Hq, k_s), np.int32)
    v_sc = np.zeros((B, Hq, N))
    s_sc = np.zeros((B, Hq, N))
    for b in range(B):
        for h in range(Hq):
            vs, ss = vs_scores(q[b, h, N - last_q:], k[b, h // G], scale)
            v_sc[b, h], s_sc[b, h] = vs, ss
            v_idx[b, h] = topk_lower(vs, k_v)
            s_idx[b, h] = topk_lower(ss, k_s)
    return v_idx, s_idx, v_sc, s_sc


def score_cover(score: np.ndarray, p: float) -> int:
    """Top-p budget of Algorithm 1: the smallest k such that the k largest scores
    (sorted descending, ties to the lower index) sum to at least p times the
    total of all scores; 0 < p < 1."""
    n = score.shape[0]
    order = np.lexsort((np.arange(n), -score))
    cum = np.cumsum(score[order])
    theta = p * cum[-1]
    return int(np.searchsorted(cum, theta, side="left")) + 1


def estimate_topp(q: np.ndarray, k: np.ndarray, last_q: int, p_v: float, p_s: float, kmax_v: int, kmax_s: int,
                  scale: float):
    """Whole-layer estimator with the top-p budget (Algorithm 1).

    Per head: k_v = min(score_cover(v_score, p_v), kmax_v), k_s likewise (kmax is
    the caller's capacity), then the argtopk of step 6 with those budgets.
    Returns v_idx [B, Hq, kmax_v] (the k_v selected positions ascending, then -1
    in the unused slots), s_idx [B, Hq, kmax_s] alike, v_cnt, s_cnt [B, Hq]
    (int32) and v_score, s_score [B, Hq, N] (fp64).
    """
    B, Hq, N, d = q.shape
    G = Hq // k.shape[1]
    v_idx = np.full((B, Hq, kmax_v), -1, np.int32)
    s_idx = np.full((B, Hq, kmax_s), -1, np.int32)
    v_cnt = np.zeros((B, Hq), np.int32)
    s_cnt = np.zeros((B, Hq), np.int32)
    v_sc = np.zeros((B, Hq, N))
    s_sc = np.zeros((B, Hq, N))
    for b in range(B):
        for h in range(Hq):
            vs, ss = vs_scores(q[b, h, N - last_q:], k[b, h // G], scale)
            v_sc[b, h], s_sc[b, h] = vs, ss
            kv = min(score_cover(vs, p_v), kmax_v)
            ks = min(score_cover(ss, p_s), kmax_s)
            v_cnt[b, h], s_cnt[b, h] = kv, ks
            v_idx[b, h, :kv] = topk_lower(vs, kv)
            s_idx[b, h, :ks] = topk_lower(ss, ks)
    return v_idx, s_idx, v_cnt, s_cnt, v_sc, s_sc
