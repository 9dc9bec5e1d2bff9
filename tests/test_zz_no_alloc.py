"""The allocation-free index build (msparse_build_index_noalloc, for callers
that cannot allocate) against msparse_build_index with a caller workspace:
bit-identical index arrays on two calls in a row, the second smaller (the
fixed scratch keeps the first call's contents), for the whole sequence and a
ring step; and a size beyond the fixed scratch rejected before any launch."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2510_18830_amd as ms
from tests.helpers import gpu_csr


def _sets(rng, B, Hq, Ng, k_v, k_s):
    v = np.stack([np.stack([np.sort(rng.choice(Ng, k_v, replace=False)) for _ in range(Hq)]) for _ in range(B)])
    s = np.stack([np.stack([np.sort(rng.choice(Ng, k_s, replace=False)) for _ in range(Hq)]) for _ in range(B)])
    return v.astype(np.int32), s.astype(np.int32)


@pytest.mark.gpu
def test_noalloc_index_build_matches_workspace_build(gpu):
    rng = np.random.default_rng(77)
    cases = [  # (B, Hq, Hkv, N_global, k_v, k_s, ring): the second call is smaller than the first
        (2, 6, 2, 65536, 700, 3000, None),
        (1, 3, 1, 8192, 90, 500, (4, 1, 2, "striped")),
        (1, 2, 1, 4096, 40, 300, None),
    ]
    for B, Hq, Hkv, Ng, k_v, k_s, rg in cases:
        print(f"noalloc index B{B} Hq{Hq} N{Ng} k_v{k_v} k_s{k_s} ring {rg}", flush=True)
        ring = ms.make_ring(*rg) if rg else None
        W = rg[0] if rg else 1
        dims = ms.make_dims(B, Ng // W, Hq, Hkv, 128)
        v, s = _sets(rng, B, Hq, Ng, k_v, k_s)
        tv, ts = torch.from_numpy(v).to(gpu), torch.from_numpy(s).to(gpu)
        ref = ms.make_index(dims, tv, ts, ring)
        blk, col, vcol = (int(ref.struct.blk_cap), int(ref.struct.col_cap), int(ref.struct.vcol_cap))
        got = ms.alloc_index(dims, blk, col, vcol, gpu, W)
        for t in got.tensors.values():       # stale contents must not leak into the result
            t.fill_(-7) if t.dtype != torch.int64 else t.fill_(-9)
        ms.build_index_noalloc(dims, tv, ts, got, ring)
        torch.cuda.synchronize()
        a, b = gpu_csr(ref), gpu_csr(got)
        for key in a:
            assert np.array_equal(a[key], b[key]), key
        assert int(got["overflow"].item()) == 0


def test_noalloc_rejects_more_than_its_scratch():
    L = ms.lib()
    d = ms.make_dims(8, 1 << 20, 64, 8, 128)     # about 0.4 GB of index scratch
    fake = ctypes.c_void_p(16)
    x = ms.IndexStruct(fake, fake, 1 << 40, fake, fake, 1 << 40, fake, fake, fake, fake, 1 << 40, fake, fake, fake,
                       None, 1)
    st = L.msparse_build_index_noalloc(ctypes.byref(d), fake, 4096, fake, 16384, None, ctypes.byref(x), None)
    assert st == -4, L.msparse_last_error()
    assert b"fixed scratch" in L.msparse_last_error()
