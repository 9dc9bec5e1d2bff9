"""An overflowed index, and inputs far from unit scale.

(1) An index built with half the capacities it needs sets its overflow flag;
    the attention calls then return from every kernel without reading the
    incomplete lists, so every output keeps the values it had before.  A build
    with the exact capacities afterwards gives results equal to the oracle's.
(2) Inputs far from unit scale.  Every fp16 operand is scaled by a power of
    two taken from max |q|, |k|, |v| or |dO| (dZ by t with t d max|v| in
    [2^9, 2^10)), so multiplying Q, K, V, dO by powers of two (with the logits
    unchanged) must give bit-identical results up to the matching powers of
    two: out and dV scale with V and dO, dQ with dO V K, dK with dO V Q.
(3) Rows far from unit scale inside one tensor (the paper attributes vertical
    lines to keys of large norm, Section 3.2): key rows times 4, dO rows times
    2^6, value rows times 2^-10 and value rows times 2^e for a few e, against
    the oracle.  fp16 rounding of P (relative 2^-12) against a value row of
    size 2^e moves the outputs that read it in proportion, so the parity bars
    apply per row in units of max(1, RMS of that reference row); lse to 1e-3.
    Key rows of 2^8 (logits up to about +-4600) miss the row bar on dQ by up
    to 2x: the fp32 lse then carries an absolute rounding near 1e-4 or more,
    which rows with nearly all their weight on one key amplify; that logit
    scale is outside what fp32 softmax resolves, and the tested key rows stop
    at 2^4 (logits up to about +-290).
"""
import math

import numpy as np
import pytest
import torch

import paper_2510_18830_amd as ms
from oracle import attn as OA
from oracle import index as OI
from synth import WORKLOADS, make_inputs
from tests.helpers import assert_close, assert_close_rows, assert_lse_close, inputs_f64, oracle_indices

pytestmark = pytest.mark.gpu


def test_overflowed_index_leaves_outputs_untouched(gpu):
    wl = WORKLOADS["layer_32k"].resized(seq=2048, heads_q=2, heads_kv=1, k_v=64, k_s=300)
    print(f"overflow {wl}", flush=True)
    x = make_inputs(wl, "cpu")
    f = inputs_f64(x)
    vi, si, _, _ = oracle_indices(f, wl)
    dims = ms.make_dims(wl.batch, wl.seq, wl.heads_q, wl.heads_kv, wl.head_dim)
    q, k, v, do = (x[n].to(gpu) for n in ("q", "k", "v", "do"))
    tv, ts = torch.from_numpy(vi).to(gpu), torch.from_numpy(si).to(gpu)
    blk, col, vcol = ms.index_count(dims, tv, ts)
    small = ms.alloc_index(dims, blk // 2, col // 2, vcol, gpu)
    ms.build_index(dims, tv, ts, small)
    torch.cuda.synchronize()
    assert int(small["overflow"].item()) == 1

    def filled(shape, dtype, val):
        return torch.full(shape, val, dtype=dtype, device=gpu)

    out = filled(q.shape, torch.bfloat16, 7.0)
    lse = filled(q.shape[:-1], torch.float32, 3.0)
    out32 = filled(q.shape, torch.float32, 5.0)
    o_acc = filled(q.shape, torch.float32, 11.0)
    l_acc = filled(q.shape[:-1], torch.float32, 13.0)
    dq = filled(q.shape, torch.float32, 9.0)
    dk = filled(k.shape, torch.float32, 17.0)
    dv = filled(v.shape, torch.float32, 19.0)
    ms.attn_fwd(dims, q, k, v, small, out=out, lse=lse, out_f32=out32)
    ms.attn_fwd_merge(dims, q, k, v, small, o_acc, l_acc, first=False)
    ms.attn_bwd(dims, q, k, v, out, do, lse, small, dq, dk, dv, out_f32=out32)
    torch.cuda.synchronize()
    for name, t, val in (("out", out.float(), 7.0), ("lse", lse, 3.0), ("out32", out32, 5.0), ("o_acc", o_acc, 11.0),
                         ("lse_acc", l_acc, 13.0), ("dq", dq, 9.0), ("dk", dk, 17.0), ("dv", dv, 19.0)):
        assert bool((t == val).all()), f"{name} was written after an overflowed build"

    # the exact capacities: the flag is cleared and the results are the oracle's
    full = ms.alloc_index(dims, blk, col, vcol, gpu)
    full["overflow"].fill_(1)
    ms.build_index(dims, tv, ts, full)
    out, lse = ms.attn_fwd(dims, q, k, v, full, out_f32=out32)
    dq, dk, dv = ms.attn_bwd(dims, q, k, v, out, do, lse, full, out_f32=out32)
    torch.cuda.synchronize()
    assert int(full["overflow"].item()) == 0
    scale = 1 / math.sqrt(wl.head_dim)
    ref = OI.Index(vi, si, wl.seq)
    ro, rl = OA.layer_fwd(f["q"], f["k"], f["v"], ref, scale)
    rq, rk, rv = OA.layer_bwd(f["q"], f["k"], f["v"], f["do"], ref, scale)
    assert_close("out", out.float().cpu().numpy(), ro)
    assert_lse_close(lse.cpu().numpy(), rl)
    for n, g, r in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv)):
        assert_close(n, g.cpu().numpy(), r)


def _run(gpu, wl, x, vi, si):
    dims = ms.make_dims(wl.batch, wl.seq, wl.heads_q, wl.heads_kv, wl.head_dim)
    q, k, v, do = (x[n].to(gpu) for n in ("q", "k", "v", "do"))
    idx = ms.make_index(dims, torch.from_numpy(vi).to(gpu), torch.from_numpy(si).to(gpu))
    out32 = torch.empty(q.shape, dtype=torch.float32, device=gpu)
    out, lse = ms.attn_fwd(dims, q, k, v, idx, out_f32=out32)
    dq, dk, dv = ms.attn_bwd(dims, q, k, v, out, do, lse, idx, out_f32=out32)
    torch.cuda.synchronize()
    return {"out": out.float(), "out32": out32, "lse": lse, "dq": dq, "dk": dk, "dv": dv}


def _times(t, e):
    """t * 2^e, exact in bf16 / fp32 within range (checked)."""
    y = (t.float() * 2.0 ** e).to(t.dtype)
    assert torch.equal(y.float() * 2.0 ** -e, t.float())
    return y


@pytest.mark.parametrize("d,eq,ek,ev,eo", [(128, -6, 6, -10, 12), (64, -6, 6, -10, 12), (128, 5, -5, 9, -12)])
def test_power_of_two_scaling_is_exact(gpu, d, eq, ek, ev, eo):
    wl = WORKLOADS["layer_32k"].resized(seq=2048, heads_q=4, heads_kv=2, head_dim=d, k_v=64, k_s=300)
    print(f"scaling q 2^{eq} k 2^{ek} v 2^{ev} dO 2^{eo} d{d}", flush=True)
    x = make_inputs(wl, "cpu")
    vi, si, _, _ = oracle_indices(inputs_f64(x), wl)
    base = _run(gpu, wl, x, vi, si)
    y = {"q": _times(x["q"], eq), "k": _times(x["k"], ek), "v": _times(x["v"], ev), "do": _times(x["do"], eo)}
    got = _run(gpu, wl, y, vi, si)
    want = {"out": ev, "out32": ev, "lse": 0, "dv": eo, "dq": eo + ev + ek, "dk": eo + ev + eq}
    for n, e in want.items():
        assert torch.equal(got[n], base[n] * 2.0 ** e), f"{n}: not the unit-scale result times 2^{e}"
    # and the unit-scale result is the oracle's
    f = inputs_f64(x)
    ref = OI.Index(vi, si, wl.seq)
    scale = 1 / math.sqrt(d)
    ro, rl = OA.layer_fwd(f["q"], f["k"], f["v"], ref, scale)
    rq, rk, rv = OA.layer_bwd(f["q"], f["k"], f["v"], f["do"], ref, scale)
    assert_close("out", base["out"].cpu().numpy(), ro)
    assert_lse_close(base["lse"].cpu().numpy(), rl)
    for n, r in (("dq", rq), ("dk", rk), ("dv", rv)):
        assert_close(n, base[n].cpu().numpy(), r)


def _outlier_rows(wl, seed, ev, ek):
    """The workload's inputs with some rows multiplied by powers of two."""
    x = make_inputs(wl, "cpu")
    rng = np.random.default_rng(seed)
    N = wl.seq
    y = {n: x[n] for n in ("q", "k", "v", "do")}
    k, v, do = (x[n].float() for n in ("k", "v", "do"))
    for g in range(wl.heads_kv):
        big_v, small_v = np.split(rng.choice(N, 16, replace=False), 2)
        v[:, g, torch.from_numpy(big_v)] *= 2.0 ** ev
        v[:, g, torch.from_numpy(small_v)] *= 2.0 ** -10
        k[:, g, torch.from_numpy(rng.choice(N - wl.last_q, 16, replace=False))] *= 2.0 ** ek
    for h in range(wl.heads_q):
        do[:, h, torch.from_numpy(rng.choice(N, 16, replace=False))] *= 2.0 ** 6
    for n, t in (("k", k), ("v", v), ("do", do)):
        y[n] = t.to(torch.bfloat16)
        assert torch.equal(y[n].float(), t), n
    return y


@pytest.mark.parametrize("d,ev,ek", [(128, 3, 2), (64, 3, 2), (128, 10, 2), (128, 3, 4), (64, 10, 4)])
def test_outlier_rows_parity(gpu, d, ev, ek):
    wl = WORKLOADS["layer_32k"].resized(seq=2048, heads_q=4, heads_kv=2, head_dim=d, k_v=64, k_s=300)
    print(f"outlier rows d{d} value rows 2^{ev} key rows 2^{ek}", flush=True)
    x = _outlier_rows(wl, 100 + d, ev, ek)
    f = inputs_f64(x)
    vi, si, _, _ = oracle_indices(f, wl)
    scale = 1 / math.sqrt(d)
    ref = OI.Index(vi, si, wl.seq)
    ro, rl = OA.layer_fwd(f["q"], f["k"], f["v"], ref, scale)
    rq, rk, rv = OA.layer_bwd(f["q"], f["k"], f["v"], f["do"], ref, scale)
    got = _run(gpu, wl, x, vi, si)
    for n, r in (("out32", ro), ("dq", rq), ("dk", rk), ("dv", rv)):
        g = got[n].cpu().numpy()
        e = np.abs(g - r)
        print(f"{n}: max-abs {e.max():.3e} mean-abs {e.mean():.3e} ref-rms {np.sqrt((r ** 2).mean()):.3e}",
              flush=True)
        assert_close_rows(n, g, r)
    assert_lse_close(got["lse"].cpu().numpy(), rl)
