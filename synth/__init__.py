"""Seeded synthetic inputs shared by the oracle-side tests and the GPU path.

This package holds no arithmetic of the sparse-attention method itself: it only
draws Q/K/V/dO tensors with a planted vertical-slash structure (Section 3.2,
Theorem 3.1 of the paper) and describes the benchmark workloads.
"""
from .gen import WORKLOADS, Workload, make_inputs, bf16_bits  # noqa: F401
