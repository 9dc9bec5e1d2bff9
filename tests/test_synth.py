"""The synthetic generator: determinism, shapes, the Theorem 3.1 band identity and
planted-vertical recovery by the reference estimator on the tiny workload."""
import math

import numpy as np
import torch

from synth import WORKLOADS, make_inputs, bf16_bits
from synth.gen import _rope_band, slash_theta
from oracle import bf16, estimate as E


def test_band_mean_logit_depends_only_on_offset():
    # rho(n) w . rho(m) w = sum_i (w_i^2 + w_{i+d/2}^2) cos((n - m) theta_i)   (Theorem 3.1)
    d, n = 16, 300
    wl = WORKLOADS["tiny_4k"].resized(head_dim=d, k_s=100)
    th = slash_theta(wl)
    w = torch.randn(d, dtype=torch.float64)
    band = _rope_band(n, d, w, torch.from_numpy(th), "cpu").double()
    gram = band @ band.T
    pw = (w[: d // 2] ** 2 + w[d // 2:] ** 2).numpy()
    for a, b in [(0, 0), (5, 2), (299, 17), (100, 250)]:
        want = float((pw * np.cos((a - b) * th)).sum())
        assert abs(gram[a, b].item() - want) < 1e-4 * max(1, abs(want))


def test_deterministic_and_shaped():
    wl = WORKLOADS["layer_32k"].resized(seq=1024, heads_q=4, heads_kv=2, k_s=128, k_v=16)
    a = make_inputs(wl)
    b = make_inputs(wl)
    for key in ("q", "k", "v", "do"):
        assert a[key].dtype == torch.bfloat16
        assert torch.equal(a[key], b[key])
    assert a["q"].shape == (1, 4, 1024, 128) and a["k"].shape == (1, 2, 1024, 128)
    assert (a["planted_cols"] < 1024 - wl.last_q).all()


def test_tiny_planted_verticals_recovered():
    wl = WORKLOADS["tiny_4k"]
    x = make_inputs(wl, with_do=False)
    q = bf16.to_f64(bf16_bits(x["q"]))
    k = bf16.to_f64(bf16_bits(x["k"]))
    vs, _ = E.vs_scores(q[0, 0, -wl.last_q:], k[0, 0], 1 / math.sqrt(wl.head_dim))
    vi = E.topk_lower(vs, wl.k_v)
    assert np.isin(x["planted_cols"][0, 0].numpy(), vi).mean() >= 0.9
