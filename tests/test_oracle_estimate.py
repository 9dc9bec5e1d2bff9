"""Pins for the reference estimator (Algorithm 1): closed forms, invariants,
a library softmax, and brute force on tiny inputs."""
import math

import numpy as np
import pytest
import torch

from oracle import estimate as E
from oracle import bf16


def test_bf16_patterns():
    bits = np.array([0x3F80, 0xC000, 0x7F80, 0x0001, 0x8000, 0x4049], dtype=np.uint16)
    x = bf16.to_f64(bits)
    assert x[0] == 1.0 and x[1] == -2.0 and x[2] == np.inf
    assert x[3] == 2.0 ** -133 and x[4] == 0.0 and np.signbit(x[4])
    assert x[5] == 3.140625


def test_zero_query_closed_form_and_tie_break():
    # q = 0: every causal logit is 0, so P[n, m] = 1 / (n + 1) for m <= n.
    N, L, d = 96, 16, 8
    rng = np.random.default_rng(0)
    k = rng.standard_normal((N, d))
    vs, ss = E.vs_scores(np.zeros((L, d)), k, 1 / math.sqrt(d))
    rows = range(N - L, N)
    want_v = np.array([sum(1.0 / (n + 1) for n in rows if n >= m) for m in range(N)])
    want_s = np.array([sum(1.0 / (n + 1) for n in rows if n >= dl) for dl in range(N)])
    np.testing.assert_allclose(vs, want_v, rtol=0, atol=1e-14)
    np.testing.assert_allclose(ss, want_s, rtol=0, atol=1e-14)
    # all m <= N - L tie exactly: the lower index must win
    assert E.topk_lower(vs, 20).tolist() == list(range(20))
    assert E.topk_lower(ss, 33).tolist() == list(range(33))


def _closed(N, L, hot, a):
    """P for one planted logit a at (n, hot(n)) per row, all other causal logits 0."""
    P = np.zeros((N, N))
    for n in range(N):
        h = hot(n)
        den = (n + 1) + (math.exp(a) - 1 if h is not None else 0.0)
        for m in range(n + 1):
            P[n, m] = (math.exp(a) if m == h else 1.0) / den
    return P[N - L:]


def test_planted_slash_closed_form():
    # q_n = e_n, k_m = c e_{m + 5}: the only non-zero logit of row n sits at m = n - 5.
    N, L, d, c, d0 = 40, 12, 64, 20.0, 5
    q = np.eye(d)[:N]
    k = np.zeros((N, d))
    for m in range(N):
        if m + d0 < d:
            k[m, m + d0] = c
    scale = 1 / math.sqrt(d)
    vs, ss = E.vs_scores(q[N - L:], k, scale)
    P = _closed(N, L, lambda n: n - d0 if n >= d0 else None, c * scale)
    want_v = P.sum(axis=0)
    want_s = np.array([sum(P[r, n - dl] for r, n in enumerate(range(N - L, N)) if n >= dl)
                       for dl in range(N)])
    np.testing.assert_allclose(vs, want_v, atol=1e-13)
    np.testing.assert_allclose(ss, want_s, atol=1e-13)
    assert E.topk_lower(ss, 1).tolist() == [d0]


def test_planted_vertical_closed_form():
    N, L, d, c, m0 = 48, 10, 16, 30.0, 7
    u = np.zeros(d)
    u[3] = 1.0
    q = np.tile(u, (N, 1))
    k = np.zeros((N, d))
    k[m0] = c * u
    scale = 1 / math.sqrt(d)
    vs, ss = E.vs_scores(q[N - L:], k, scale)
    P = _closed(N, L, lambda n: m0 if n >= m0 else None, c * scale)
    np.testing.assert_allclose(vs, P.sum(axis=0), atol=1e-13)
    assert E.topk_lower(vs, 1).tolist() == [m0]
    # the vertical's mass lands on the offsets n - m0 of the observed rows
    want_s6 = sum(P[r, n - (N - 1 - m0)] for r, n in enumerate(range(N - L, N)) if n >= N - 1 - m0)
    assert abs(ss[N - 1 - m0] - want_s6) < 1e-13


def test_against_library_softmax_and_loops():
    rng = np.random.default_rng(1)
    N, L, d = 70, 9, 12
    q = rng.standard_normal((N, d))
    k = rng.standard_normal((N, d))
    scale = 0.3
    vs, ss = E.vs_scores(q[N - L:], k, scale)
    z = torch.from_numpy(scale * q[N - L:] @ k.T)
    rows = torch.arange(N - L, N)[:, None]
    z = z.masked_fill(torch.arange(N)[None, :] > rows, float("-inf"))
    P = torch.softmax(z, dim=-1).numpy()
    want_v = [sum(P[r, m] for r in range(L)) for m in range(N)]
    want_s = [0.0] * N
    for r in range(L):
        n = N - L + r
        for m in range(n + 1):
            want_s[n - m] += P[r, m]
    np.testing.assert_allclose(vs, want_v, atol=1e-14)
    np.testing.assert_allclose(ss, want_s, atol=1e-14)
    # each observed row carries unit mass
    assert abs(vs.sum() - L) < 1e-12 and abs(ss.sum() - L) < 1e-12


def test_topk_brute_force_and_full_budget():
    rng = np.random.default_rng(2)
    for _ in range(20):
        n = int(rng.integers(5, 60))
        sc = rng.integers(0, 6, n).astype(np.float64)   # many exact ties
        k = int(rng.integers(1, n + 1))
        want = sorted(sorted(range(n), key=lambda i: (-sc[i], i))[:k])
        assert E.topk_lower(sc, k).tolist() == want
    assert E.topk_lower(rng.random(17), 17).tolist() == list(range(17))


def test_layer_estimate_gqa_mapping():
    rng = np.random.default_rng(3)
    B, Hq, Hkv, N, d, L = 2, 4, 2, 64, 8, 8
    q = rng.standard_normal((B, Hq, N, d))
    k = rng.standard_normal((B, Hkv, N, d))
    vi, si, vs, ss = E.estimate(q, k, L, 5, 7, 0.35)
    for b in range(B):
        for h in range(Hq):
            v1, s1 = E.vs_scores(q[b, h, N - L:], k[b, h // 2], 0.35)
            np.testing.assert_array_equal(vs[b, h], v1)
            assert vi[b, h].tolist() == E.topk_lower(v1, 5).tolist()
            assert si[b, h].tolist() == E.topk_lower(s1, 7).tolist()


# ---- top-p budget (score_cover of Algorithm 1)

def test_score_cover_zero_query_exact_rational():
    # q = 0: v_score[m] = H_N - H_{N-L} =: c0 for every m <= N - L (N - L + 1 equal
    # entries), and the total mass is L.  While p L <= (N - L + 1) c0 the budget
    # is ceil(p L / c0), computed here in exact rationals.
    from fractions import Fraction as Fr
    N, L, d = 200, 16, 8
    rng = np.random.default_rng(4)
    vs, ss = E.vs_scores(np.zeros((L, d)), rng.standard_normal((N, d)), 1 / math.sqrt(d))
    c0 = sum(Fr(1, n + 1) for n in range(N - L, N))
    for p in (Fr(1, 10), Fr(3, 10), Fr(1, 2), Fr(77, 100), Fr(9, 10)):
        want = math.ceil(p * L / c0)
        assert want <= N - L + 1
        assert E.score_cover(vs, float(p)) == want
        assert E.score_cover(ss, float(p)) == want   # same closed form in delta


def test_score_cover_hand_example():
    # scores 0.1 0.4 0.2 0.2 0.1 (total 1): sorted 0.4 (1), 0.2 (2), 0.2 (3),
    # 0.1 (0), 0.1 (4); cumulative 0.4 0.6 0.8 0.9 1.0
    sc = np.array([0.1, 0.4, 0.2, 0.2, 0.1])
    for p, k in ((0.05, 1), (0.39, 1), (0.5, 2), (0.7, 3), (0.85, 4), (0.95, 5)):
        assert E.score_cover(sc, p) == k, p
    # with k = 4 the tie at 0.1 goes to the lower index
    assert E.topk_lower(sc, E.score_cover(sc, 0.85)).tolist() == [0, 1, 2, 3]
    # "at least": reaching the threshold exactly is enough (binary-exact values)
    sc = np.array([0.25, 0.25, 0.5])
    assert E.score_cover(sc, 0.5) == 1 and E.score_cover(sc, 0.75) == 2


def test_score_cover_brute_force_subsets():
    # the budget is the smallest size of ANY subset reaching p of the total mass
    import itertools
    rng = np.random.default_rng(5)
    checked = 0
    for _ in range(60):
        n = int(rng.integers(1, 9))
        sc = rng.random(n) ** 3
        p = float(rng.uniform(0.02, 0.98))
        theta = p * sc.sum()
        best = [max(math.fsum(sc[list(c)]) for c in itertools.combinations(range(n), r)) for r in range(1, n + 1)]
        if min(abs(x - theta) for x in best) < 1e-9:     # too close to call in floating point
            continue
        want = 1 + min(r for r in range(n) if best[r] >= theta)
        assert E.score_cover(sc, p) == want, (sc, p)
        checked += 1
    assert checked > 40


def test_score_cover_invariants():
    rng = np.random.default_rng(6)
    sc = rng.exponential(size=3000) ** 4
    srt = np.sort(sc)[::-1]
    last = 0
    for p in np.linspace(0.01, 0.99, 50):
        k = E.score_cover(sc, p)
        assert srt[:k].sum() >= p * sc.sum() * (1 - 1e-12)
        assert k == 1 or srt[:k - 1].sum() < p * sc.sum()
        assert k >= last
        last = k


def test_estimate_topp_cap_padding_and_fixed_k():
    rng = np.random.default_rng(7)
    B, Hq, Hkv, N, d, L = 1, 4, 2, 256, 8, 16
    q = 2 * rng.standard_normal((B, Hq, N, d))
    k = rng.standard_normal((B, Hkv, N, d))
    vi, si, vc, sc_, vs, ss = E.estimate_topp(q, k, L, 0.6, 0.8, 40, 60, 0.35)
    for h in range(Hq):
        kv = min(E.score_cover(vs[0, h], 0.6), 40)
        ks = min(E.score_cover(ss[0, h], 0.8), 60)
        assert (vc[0, h], sc_[0, h]) == (kv, ks)
        assert vi[0, h, :kv].tolist() == E.topk_lower(vs[0, h], kv).tolist()
        assert si[0, h, :ks].tolist() == E.topk_lower(ss[0, h], ks).tolist()
        assert (vi[0, h, kv:] == -1).all() and (si[0, h, ks:] == -1).all()
    # a cap below the budget gives exactly the fixed-k estimate
    vi2, si2, vc2, sc2, _, _ = E.estimate_topp(q, k, L, 0.99, 0.99, 3, 5, 0.35)
    vi3, si3, _, _ = E.estimate(q, k, L, 3, 5, 0.35)
    assert (vc2 == 3).all() and (sc2 == 5).all()
    np.testing.assert_array_equal(vi2, vi3)
    np.testing.assert_array_equal(si2, si3)
