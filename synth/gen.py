"""Seeded planted-pattern generator for the vertical-slash sparse-attention workloads.

The paper trains Qwen2.5-3B / Llama-3.1-8B on ProLong at 512K tokens (Sections 5.1-5.2);
neither the data nor the weights are available, so the benchmark inputs are
synthetic tensors with the paper's shapes and a planted vertical-slash structure:

* slash band -- Theorem 3.1 (Section 3.2, proof in the appendix) says that with
  RoPE the expected logit depends only on n - m.  We add the same rotary-rotated
  unit vector w_g (rotate-half RoPE, pair i at frequency theta_i) to every query
  and key of a KV group, so E[z_{n,m}] gains
  (a_s^2 / sqrt(d)) * sum_i (w_i^2 + w_{i+d/2}^2) * cos((n - m) theta_i),
  a band along the main diagonal.  The RoPE base is b_gen = 4 * k_s and only
  the low-frequency pairs theta_i <= 2 / k_s carry energy, so the mean boost
  stays above about half its peak out to |n - m| = k_s and its later lobes stay
  below about a quarter of the peak: the top-k_s slashes form a nearly
  contiguous run from the main diagonal.  The peak boost is
  a_s^2 / sqrt(d) = 8.
* verticals -- outlier keys (Section 3.2): n_vert seed-chosen key positions per
  KV group, drawn without replacement from [0, N - last_q), get
  3 * sqrt(d) * u added, u the unit mean of the group's queries (taken before
  the slash band is added).  The literal 3 * u would move a logit by only about
  3 / sqrt(d) standard deviations; sqrt(d) is the norm of an N(0, I) key.

Draw order with one torch.Generator seeded with the workload seed, on the
device the tensors are made on:
  1. Q [B,Hq,N,d], K [B,Hkv,N,d], V [B,Hkv,N,d], dO [B,Hq,N,d] ~ N(0,1) fp32,
     each drawn one (b, h) slice at a time in (b, h) order;
  2. for each (b, g) in order: w_g ~ N(0, I_d) (slash workloads only),
     then the vertical positions (randperm(N - last_q)[:n_vert]);
  3. Q, K, V, dO are rounded to bf16 (round to nearest even).
The CPU and the GPU generators give different streams: a test draws once on one
device and copies what it needs to the other.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, replace

import numpy as np
import torch

SLASH_BETA = 8.0          # peak logit boost a_s^2 / sqrt(d) of the slash band
SLASH_THETA_SPAN = 2.0    # keep rotary pairs with theta_i <= SLASH_THETA_SPAN / k_s
VERT_GAIN = 3.0           # vertical outlier strength, in units of sqrt(d)


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    heads_q: int
    heads_kv: int
    seq: int
    head_dim: int
    last_q: int
    k_v: int
    k_s: int
    n_vert: int
    slash: bool
    seed: int
    world: int = 1        # ring workers (1 = whole sequence on one GPU)
    layout: str = "striped"

    def resized(self, **kw) -> "Workload":
        return replace(self, **kw)


WORKLOADS = {
    "tiny_4k": Workload("tiny_4k", 1, 1, 1, 4096, 64, 64, 128, 256, 16, False, 1),
    "layer_32k": Workload("layer_32k", 1, 16, 2, 32768, 128, 64, 1000, 6096, 64, True, 2),
    "layer_128k": Workload("layer_128k", 1, 32, 8, 131072, 128, 64, 2048, 8192, 64, True, 3),
    "ring_512k_w8": Workload("ring_512k_w8", 1, 28, 4, 524288, 128, 64, 4096, 16384, 64, True, 5,
                             world=8, layout="striped"),
    "layer_512k": Workload("layer_512k", 1, 28, 4, 524288, 128, 64, 4096, 16384, 64, True, 5),
    # forward-only sparse prefill (inference) at 1M tokens, the 512K layer's heads and budgets
    "prefill_1m": Workload("prefill_1m", 1, 28, 4, 1048576, 128, 64, 4096, 16384, 64, True, 6),
}


def _rope_band(n: int, d: int, w: torch.Tensor, theta: torch.Tensor, device) -> torch.Tensor:
    """rho(p) w for p = 0..n-1 with rotate-half RoPE; returns [n, d] fp32."""
    half = d // 2
    pos = torch.arange(n, device=device, dtype=torch.float64)
    ang = pos[:, None] * theta[None, :].to(device=device, dtype=torch.float64)
    c, s = torch.cos(ang), torch.sin(ang)
    x = w[:half].to(torch.float64)
    y = w[half:].to(torch.float64)
    out = torch.empty((n, d), device=device, dtype=torch.float64)
    out[:, :half] = x * c - y * s
    out[:, half:] = x * s + y * c
    return out.to(torch.float32)


def slash_theta(wl: Workload) -> np.ndarray:
    d = wl.head_dim
    b_gen = 4.0 * wl.k_s
    return b_gen ** (-2.0 * np.arange(d // 2) / d)


def make_inputs(wl: Workload, device="cpu", with_do: bool = True) -> dict:
    """Draw the workload's bf16 tensors (see the module docstring for the recipe)."""
    device = torch.device(device)
    g = torch.Generator(device=device)
    g.manual_seed(wl.seed)
    B, Hq, Hkv, N, d = wl.batch, wl.heads_q, wl.heads_kv, wl.seq, wl.head_dim
    G = Hq // Hkv

    def draw(h):
        t = torch.empty((B, h, N, d), device=device, dtype=torch.float32)
        for b in range(B):
            for i in range(h):
                t[b, i] = torch.randn((N, d), generator=g, device=device, dtype=torch.float32)
        return t

    q = draw(Hq)
    k = draw(Hkv)
    v = draw(Hkv).to(torch.bfloat16)
    do = draw(Hq).to(torch.bfloat16) if with_do else None

    theta = slash_theta(wl)
    keep = theta <= SLASH_THETA_SPAN / wl.k_s
    a_s = math.sqrt(SLASH_BETA * math.sqrt(d))
    planted = torch.empty((B, Hkv, wl.n_vert), dtype=torch.int64)
    slash_w = torch.zeros((B, Hkv, d), dtype=torch.float32)
    keep_t = torch.from_numpy(np.concatenate([keep, keep])).to(device)
    for b in range(B):
        for kh in range(Hkv):
            heads = slice(kh * G, (kh + 1) * G)
            u = q[b, heads].mean(dim=(0, 1))
            u = u / torch.linalg.vector_norm(u)
            if wl.slash:
                w = torch.randn((d,), generator=g, device=device, dtype=torch.float32)
                w = torch.where(keep_t, w, torch.zeros_like(w))
                w = w / torch.linalg.vector_norm(w)
                slash_w[b, kh] = w.cpu()
                band = a_s * _rope_band(N, d, w, torch.from_numpy(theta), device)
                q[b, heads] += band[None]
                k[b, kh] += band
                del band
            cols = torch.randperm(N - wl.last_q, generator=g, device=device)[: wl.n_vert]
            planted[b, kh] = cols.cpu()
            k[b, kh, cols] += VERT_GAIN * math.sqrt(d) * u
    out = {
        "q": q.to(torch.bfloat16),
        "k": k.to(torch.bfloat16),
        "v": v,
        "do": do,
        "planted_cols": planted,
        "slash_w": slash_w,
        "slash_a": a_s if wl.slash else 0.0,
        "slash_theta": theta,
        "slash_keep": keep,
    }
    return out


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """Raw bf16 bit patterns of a tensor as a host uint16 array (marshalling only)."""
    assert t.dtype == torch.bfloat16
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
