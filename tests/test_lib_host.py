"""Host-side checks of the C ABI: the library loads, exports every declared
symbol, and rejects bad arguments before touching the GPU."""
import ctypes
import os
import re

import pytest

import paper_2510_18830_amd as ms

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "msparse.h")


def declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(msparse_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    so = ms.lib()
    names = declared()
    assert len(names) >= 11
    for n in names:
        assert hasattr(so, n), n


def test_strerror():
    L = ms.lib()
    assert L.msparse_strerror(0) == b"ok"
    assert L.msparse_strerror(-3) == b"index capacity too small"


def _bad(status_expected, fn, *args):
    st = fn(*args)
    assert st == status_expected, (st, ms.lib().msparse_last_error())


def test_validation_before_launch():
    L = ms.lib()
    d = ms.make_dims(1, 4096, 4, 2, 128)
    fake = ctypes.c_void_p(16)   # never dereferenced: validation fails first
    iv = ctypes.c_void_p(32)
    # bad head_dim / block / causal / N % 64 / GQA
    for field, val, st in (("head_dim", 96, -2), ("block", 128, -2), ("causal", 0, -2), ("seq_q", 4000, -2),
                           ("heads_kv", 3, -1)):
        dd = ms.make_dims(1, 4096, 4, 2, 128)
        setattr(dd, field, val)
        if field == "seq_q":
            dd.seq_k = val
        _bad(st, L.msparse_estimate, ctypes.byref(dd), fake, fake, 64, 10, 10, iv, iv, None, None, fake, 1 << 30,
             None)
    # budgets and last_q
    _bad(-1, L.msparse_estimate, ctypes.byref(d), fake, fake, 0, 10, 10, iv, iv, None, None, fake, 1 << 30, None)
    _bad(-1, L.msparse_estimate, ctypes.byref(d), fake, fake, 64, 0, 10, iv, iv, None, None, fake, 1 << 30, None)
    _bad(-1, L.msparse_estimate, ctypes.byref(d), fake, fake, 64, 10, 4097, iv, iv, None, None, fake, 1 << 30, None)
    _bad(-2, L.msparse_estimate, ctypes.byref(d), fake, fake, 65, 10, 10, iv, iv, None, None, fake, 1 << 30, None)
    _bad(-1, L.msparse_estimate, ctypes.byref(d), None, fake, 64, 10, 10, iv, iv, None, None, fake, 1 << 30, None)
    # workspace too small
    _bad(-4, L.msparse_estimate, ctypes.byref(d), fake, fake, 64, 10, 10, iv, iv, None, None, fake, 8, None)
    # ring descriptors
    r = ms.Ring(4, 4, 0, 0)
    _bad(-1, L.msparse_index_count, ctypes.byref(d), iv, 10, iv, 10, ctypes.byref(r), ctypes.byref(ctypes.c_int64()),
         ctypes.byref(ctypes.c_int64()), ctypes.byref(ctypes.c_int64()), fake, 1 << 30, None)
    r = ms.Ring(4, 1, 0, 7)
    _bad(-1, L.msparse_index_count, ctypes.byref(d), iv, 10, iv, 10, ctypes.byref(r), ctypes.byref(ctypes.c_int64()),
         ctypes.byref(ctypes.c_int64()), ctypes.byref(ctypes.c_int64()), fake, 1 << 30, None)
    # a null index
    _bad(-1, L.msparse_attn_fwd, ctypes.byref(d), fake, fake, fake, None, fake, fake, None, fake, 1 << 40, None)
    # fused forward + merge: a null index, a null accumulator, a bad head_dim
    _bad(-1, L.msparse_attn_fwd_merge, ctypes.byref(d), fake, fake, fake, None, fake, fake, None, 0, fake, 1 << 40,
         None)
    _bad(-1, L.msparse_attn_fwd_merge, ctypes.byref(d), fake, fake, fake, None, None, fake, None, 1, fake, 1 << 40,
         None)
    dd = ms.make_dims(1, 4096, 4, 2, 128)
    dd.head_dim = 96
    _bad(-2, L.msparse_attn_fwd_merge, ctypes.byref(dd), fake, fake, fake, None, fake, fake, None, 0, fake, 1 << 40,
         None)
    # tensors off 16-byte alignment (checked before the index and workspace)
    odd = ctypes.c_void_p(24)
    _bad(-1, L.msparse_attn_fwd, ctypes.byref(d), fake, odd, fake, None, fake, fake, None, fake, 1 << 40, None)
    _bad(-1, L.msparse_attn_fwd_merge, ctypes.byref(d), fake, fake, fake, None, odd, fake, None, 0, fake, 1 << 40,
         None)
    _bad(-1, L.msparse_attn_bwd, ctypes.byref(d), fake, fake, fake, fake, None, odd, fake, None, fake, fake, fake, 0,
         fake, 1 << 40, None)
    _bad(-1, L.msparse_estimate, ctypes.byref(d), odd, fake, 64, 10, 10, iv, iv, None, None, fake, 1 << 30, None)
    _bad(-1, L.msparse_merge_out_lse, ctypes.byref(d), fake, fake, fake, fake, odd, 0, None)
    assert "16-byte" in L.msparse_last_error().decode()


def test_index_capacity_needs_overflow_flag_or_bound():
    L = ms.lib()
    d = ms.make_dims(1, 4096, 1, 1, 64)
    fake = ctypes.c_void_p(16)
    x = ms.IndexStruct(fake, fake, 10, fake, fake, 10, fake, fake, fake, fake, 10, fake, fake, fake, None, 1)
    ws = L.msparse_index_workspace(ctypes.byref(d), 8, 8, None)
    assert ws > 0
    _bad(-3, L.msparse_build_index, ctypes.byref(d), fake, 8, fake, 8, None, ctypes.byref(x), fake, ws, None)


def test_workspace_queries_are_positive():
    L = ms.lib()
    d = ms.make_dims(1, 131072, 32, 8, 128)
    assert L.msparse_estimate_workspace(ctypes.byref(d), 64, 2048, 8192) >= 2 * 32 * 131072 * 4
    assert L.msparse_attn_bwd_workspace(ctypes.byref(d), 32 * 2048) >= 32 * 131072 * 4
    assert L.msparse_index_workspace(ctypes.byref(d), 2048, 8192, ctypes.byref(ms.Ring(8, 0, 3, 1))) > 0


def test_topp_validation_before_launch():
    L = ms.lib()
    d = ms.make_dims(1, 4096, 4, 2, 128)
    fake = ctypes.c_void_p(16)
    iv = ctypes.c_void_p(32)

    def call(p_v, p_s, kv=10, ks=10, cnt=iv, ws=1 << 30):
        return L.msparse_estimate_topp(ctypes.byref(d), fake, fake, 64, p_v, p_s, kv, ks, iv, iv, cnt, cnt, None,
                                       None, fake, ws, None)

    for p in (0.0, 1.0, -0.5, 1.5, float("nan")):
        _bad(-1, call, p, 0.5)
        _bad(-1, call, 0.5, p)
    _bad(-1, lambda: call(0.5, 0.5, cnt=None))
    _bad(-1, lambda: call(0.5, 0.5, kv=0))
    _bad(-1, lambda: call(0.5, 0.5, ks=4097))
    _bad(-4, lambda: call(0.5, 0.5, ws=8))
    assert L.msparse_estimate_topp_workspace(ctypes.byref(d), 64, 100, 100) == \
        L.msparse_estimate_workspace(ctypes.byref(d), 64, 100, 100)


def test_ring_shard_matches_oracle_schedule():
    from oracle import index as OI
    for W, inner in ((1, 0), (2, 0), (4, 2), (8, 4), (8, 2), (12, 3), (16, 16), (6, 1)):
        S = OI.ring_schedule(W, inner)
        for r in range(W):
            for t in range(W):
                assert ms.ring_shard(W, inner, r, t) == S[r, t], (W, inner, r, t)
    assert ms.ring_shard(8, 3, 0, 0) == -1 and ms.ring_shard(8, 4, 8, 0) == -1 and ms.ring_shard(8, 4, 0, -1) == -1


def test_ring_validation_before_launch():
    L = ms.lib()
    d = ms.make_dims(1, 8192, 2, 1, 128)
    fake = ctypes.c_void_p(16)
    iv = ctypes.c_void_p(32)
    # hierarchical inner must divide world
    r = ms.Ring(8, 1, 0, 0, 3)
    _bad(-1, L.msparse_index_count, ctypes.byref(d), iv, 10, iv, 10, ctypes.byref(r), ctypes.byref(ctypes.c_int64()),
         ctypes.byref(ctypes.c_int64()), ctypes.byref(ctypes.c_int64()), fake, 1 << 30, None)

    def work(world, layout, tiles=iv, ws=1 << 30):
        return L.msparse_ring_work(ctypes.byref(d), iv, 10, iv, 10, world, layout, tiles, iv, fake, ws, None)
    _bad(-1, lambda: work(0, 0))
    _bad(-1, lambda: work(8, 5))
    _bad(-1, lambda: work(8, 0, tiles=None))
    _bad(-2, lambda: work(3, 0))         # 128 blocks do not split into 3 shards
    _bad(-2, lambda: work(128, 1))       # zigzag needs 2 * 128 chunks
    _bad(-4, lambda: work(8, 0, ws=8))


def test_peak_probe_validation():
    L = ms.lib()
    fake = ctypes.c_void_p(16)
    for w, it, out in ((0, 16, fake), (9, 16, fake), (2, 0, fake), (2, 12, fake), (2, 16, None)):
        for rnd in (0, 1):
            assert L.msparse_mfma_peak_probe(w, it, rnd, out, None) == -1


def test_bwd_flags_validation():
    L = ms.lib()
    d = ms.make_dims(1, 4096, 4, 2, 128)
    fake = ctypes.c_void_p(16)
    idx = ms.IndexStruct()
    for f in ("blk_ptr", "blk_idx", "col_ptr", "col_idx", "kblk_ptr", "kblk_idx", "vcol_ptr", "vcol_idx", "diag_bits",
              "q_blk_global", "k_blk_global"):
        setattr(idx, f, 64)
    idx.blk_cap = idx.col_cap = idx.vcol_cap = 1
    idx.world = 1
    st = L.msparse_attn_bwd(ctypes.byref(d), fake, fake, fake, fake, None, fake, fake, ctypes.byref(idx), fake, fake,
                            fake, 4, fake, 1 << 40, None)
    assert st == -1, ms.lib().msparse_last_error()


def test_header_compiles_as_c_and_cpp():
    """include/msparse.h is a plain C header (C99 and C++)."""
    import shutil
    import subprocess
    hdr = os.path.join(os.path.dirname(__file__), "..", "include", "msparse.h")
    for cc, lang, std in (("gcc", "c", "-std=c99"), ("g++", "c++", "-std=c++17")):
        if shutil.which(cc) is None:
            pytest.skip(f"{cc} not installed")
        r = subprocess.run([cc, "-fsyntax-only", "-Wall", "-Werror", "-x", lang, std, hdr], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr
