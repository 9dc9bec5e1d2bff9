"""Pins for the reference index (Section 4.1 (ii), Section 4.2): tile enumeration
by brute force against the token-level vertical-slash mask, special cases and
the ring-shard decomposition."""
import numpy as np
import pytest

from oracle import index as I

B64 = 64


def test_diag_set_cases():
    nb = 8
    assert I.diag_set([0], nb).tolist() == [0]
    assert I.diag_set([63], nb).tolist() == [0, 1]
    assert I.diag_set([64], nb).tolist() == [1]
    assert I.diag_set([65], nb).tolist() == [1, 2]
    assert I.diag_set([nb * 64 - 1], nb).tolist() == [nb - 1]   # ceil = nb has no tile


def _token_vs(N, V, S):
    n = np.arange(N)[:, None]
    m = np.arange(N)[None, :]
    return (m <= n) & (np.isin(m, V) | np.isin(n - m, S))


@pytest.mark.parametrize("seed", range(6))
def test_tiles_brute_force(seed):
    rng = np.random.default_rng(seed)
    N = 512
    nb = N // B64
    V = np.sort(rng.choice(N, 9, replace=False))
    S = np.sort(rng.choice(N, 7, replace=False))
    idx = I.Index(V[None, None], S[None, None], N)
    M = idx.mask_rows(0, np.arange(N))
    tok = _token_vs(N, V, S)
    assert not (tok & ~M).any()                        # covers every selected token
    assert not (M & ~np.tri(N, dtype=bool)).any()      # causal
    for i in range(nb):
        blocks = idx.blocks[0][i].tolist()
        cols = idx.cols[0][i].tolist()
        assert blocks == sorted(set(blocks)) and cols == sorted(set(cols))
        for j in blocks:                               # minimal: each tile meets a slash
            sub = tok[i * 64:(i + 1) * 64, j * 64:(j + 1) * 64]
            n = np.arange(i * 64, i * 64 + 64)[:, None]
            m = np.arange(j * 64, j * 64 + 64)[None, :]
            assert ((m <= n) & np.isin(n - m, S)).any()
        for c in cols:
            assert c // 64 not in blocks and c <= 64 * i + 63 and c in V
        for v in V:                                    # every visible vertical is covered
            if v <= 64 * i + 63:
                assert v in cols or v // 64 in blocks


def test_full_budget_is_dense_causal():
    N = 256
    idx = I.Index(np.array([[[3, 100]]]), np.arange(N)[None, None], N)
    M = idx.mask_rows(0, np.arange(N))
    assert (M == np.tri(N, dtype=bool)).all()
    assert all(len(c) == 0 for c in idx.cols[0])


def test_csr_layout_and_transpose():
    rng = np.random.default_rng(7)
    N = 1024
    V = np.stack([np.sort(rng.choice(N, 20, replace=False)) for _ in range(3)])[None]
    S = np.stack([np.sort(rng.choice(N, 30, replace=False)) for _ in range(3)])[None]
    idx = I.Index(V, S, N)
    c = idx.csr()
    nqb = N // 64
    assert c["blk_ptr"].shape == (3 * nqb + 1,)
    for bh in range(3):
        for i in range(nqb):
            a, b = c["blk_ptr"][bh * nqb + i], c["blk_ptr"][bh * nqb + i + 1]
            assert c["blk_idx"][a:b].tolist() == idx.blocks[bh][i].tolist()
            for j in c["blk_idx"][a:b]:
                ka, kb = c["kblk_ptr"][bh * nqb + j], c["kblk_ptr"][bh * nqb + j + 1]
                assert i in c["kblk_idx"][ka:kb].tolist()
        bits = c["diag_bits"].reshape(3, -1)[bh]
        D = [x for x in range(nqb) if bits[x // 32] >> (x % 32) & 1]
        assert D == I.diag_set(S[0, bh], nqb).tolist()
    assert c["kblk_idx"].size == c["blk_idx"].size


@pytest.mark.parametrize("layout,W", [("striped", 2), ("striped", 4), ("zigzag", 2), ("zigzag", 4)])
def test_ring_steps_partition_the_whole_index(layout, W):
    rng = np.random.default_rng(11)
    N = 2048
    nb = N // 64
    V = np.sort(rng.choice(N, 40, replace=False))[None, None]
    S = np.sort(rng.choice(N, 60, replace=False))[None, None]
    whole = I.Index(V, S, N)
    for r in range(W):
        qg = I.local_blocks(r, nb, W, layout)
        got_b = {int(g): [] for g in qg}
        got_c = {int(g): [] for g in qg}
        for t in range(W):
            st = I.Index(V, S, N, world=W, rank=r, step=t, layout=layout)
            kg = st.k_blk_global
            assert (np.array([I.owner(int(g), nb, W, layout) for g in kg]) == (r - t) % W).all()
            for qi, g in enumerate(st.q_blk_global.tolist()):
                got_b[g] += [int(kg[j]) for j in st.blocks[0][qi]]
                got_c[g] += [int(kg[c // 64]) * 64 + int(c) % 64 for c in st.cols[0][qi]]
        for g in qg.tolist():
            assert sorted(got_b[g]) == whole.blocks[0][g].tolist()
            assert sorted(got_c[g]) == whole.cols[0][g].tolist()


def test_ring_world_one_is_identity():
    rng = np.random.default_rng(12)
    N = 1024
    V = np.sort(rng.choice(N, 30, replace=False))[None, None]
    S = np.sort(rng.choice(N, 30, replace=False))[None, None]
    a = I.Index(V, S, N).csr()
    b = I.Index(V, S, N, world=1, rank=0, step=0, layout="zigzag").csr()
    for key in a:
        np.testing.assert_array_equal(a[key], b[key])


def test_layouts_owner_counts():
    nb = 64
    for layout in ("striped", "zigzag"):
        for W in (1, 2, 4, 8):
            counts = [len(I.local_blocks(w, nb, W, layout)) for w in range(W)]
            assert counts == [nb // W] * W
    # zigzag worker 0 holds the first and the last chunk
    assert I.local_blocks(0, 16, 2, "zigzag").tolist() == [0, 1, 2, 3, 12, 13, 14, 15]
    assert I.local_blocks(1, 16, 4, "striped").tolist() == [1, 5, 9, 13]


def test_unused_slots_are_dropped():
    # top-p lists are padded with -1 to the caller's capacity
    rng = np.random.default_rng(11)
    N = 1024
    v = np.sort(rng.choice(N, 20, replace=False)).astype(np.int32)
    s = np.sort(rng.choice(N, 30, replace=False)).astype(np.int32)
    vp = np.concatenate([v, np.full(7, -1, np.int32)])
    sp = np.concatenate([s, np.full(5, -1, np.int32)])
    assert I.diag_set(sp, N // B64).tolist() == I.diag_set(s, N // B64).tolist()
    for W, layout in ((1, "striped"), (4, "striped"), (2, "zigzag")):
        for t in range(W):
            a = I.Index(v[None, None], s[None, None], N, W, 1 % W, t, layout).csr()
            b = I.Index(vp[None, None], sp[None, None], N, W, 1 % W, t, layout).csr()
            for key in a:
                np.testing.assert_array_equal(a[key], b[key], err_msg=key)


# ---- hierarchical step order (Section 4.3, Algorithm 2) and workload matrix

@pytest.mark.parametrize("W,inner", [(2, 0), (4, 2), (8, 4), (8, 2), (12, 3), (12, 4), (6, 6), (6, 1)])
def test_ring_schedule_properties(W, inner):
    S = I.ring_schedule(W, inner)
    ar = np.arange(W)
    for r in range(W):
        assert sorted(S[r].tolist()) == ar.tolist()           # every shard once per worker
        assert S[r, 0] == r                                  # step 0: own KV
    for t in range(W):
        assert sorted(S[:, t].tolist()) == ar.tolist()       # each shard held once per step
    w = W if inner in (0, 1, W) else inner
    nodes = W // w
    for r in range(W):
        n, c = divmod(r, w)
        for t in range(W):
            i, j = divmod(t, w)
            # the inner loop only circulates one node's shards, one card back per step
            assert S[r, t] == ((n - i) % nodes) * w + (c - j) % w, (r, t)


def test_ring_schedule_flat_limits():
    for W in (3, 4, 8):
        flat = np.array([[(r - t) % W for t in range(W)] for r in range(W)])
        for inner in (0, 1, W):
            np.testing.assert_array_equal(I.ring_schedule(W, inner), flat)


@pytest.mark.parametrize("W,layout,inner", [(2, "striped", 0), (4, "striped", 0), (4, "striped", 2),
                                            (2, "zigzag", 0), (4, "zigzag", 2)])
def test_ring_work_matches_ring_indices(W, layout, inner):
    rng = np.random.default_rng(60 + W)
    N = 2048
    v = rng.integers(0, N, (1, 2, 40)).astype(np.int32)
    s = np.concatenate([np.tile(np.arange(70), (1, 2, 1)), rng.integers(0, N, (1, 2, 30))], -1).astype(np.int32)
    tiles, cols = I.ring_work(v, s, N, W, layout)
    S = I.ring_schedule(W, inner)
    for r in range(W):
        for t in range(W):
            c = I.Index(v, s, N, W, r, t, layout, inner=inner).csr()
            assert c["blk_ptr"][-1] == tiles[r, S[r, t]] and c["col_ptr"][-1] == cols[r, S[r, t]], (r, t)
    whole = I.Index(v, s, N).csr()
    assert tiles.sum() == whole["blk_ptr"][-1] and cols.sum() == whole["col_ptr"][-1]


def test_ring_work_dense_causal_brute_force():
    N, W = 1024, 4
    nb = N // B64
    v = np.zeros((1, 1, 1), np.int32)
    s = np.arange(N, dtype=np.int32)[None, None]         # every offset: the full causal grid, no columns
    for layout in ("striped", "zigzag"):
        tiles, cols = I.ring_work(v, s, N, W, layout)
        want = np.zeros((W, W), np.int64)
        for i in range(nb):
            for j in range(i + 1):
                want[I.owner(i, nb, W, layout), I.owner(j, nb, W, layout)] += 1
        np.testing.assert_array_equal(tiles, want)
        assert cols.sum() == 0


def test_imbalance_degrees_hand_example():
    work = np.array([[3.0, 1.0], [2.0, 2.0]])
    # flat ring: worker 0 sees shards 0, 1 (3, 1); worker 1 sees 1, 0 (2, 2)
    wl, sl = I.imbalance_degrees(work, I.ring_schedule(2))
    assert abs(wl - (3 / 2.5 + 2 / 1.5) / 2) < 1e-15
    assert abs(sl - (3 / 2 + 1.0) / 2) < 1e-15
