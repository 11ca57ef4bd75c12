"""Seeded synthetic inputs for the ESPACE projected linear layer.

This package is shared by the CPU oracle's tests and by the GPU path's tests and
benchmark.  It draws random numbers and builds matrices of the shapes and value
distributions of the paper's layers; it computes none of the projected-linear
arithmetic (no W·P, no Pᵀ·X, no product of the two).
"""
from .bf16 import bf16_bits_from_f64, f64_from_bf16_bits  # noqa: F401
from .configs import CONFIGS, Workload, workloads, workload  # noqa: F401
from .generate import (  # noqa: F401
    haar_orthogonal,
    index_pattern,
    spectrum,
    symmetric_with_spectrum,
    upstream_gradient,
    gaussian_tokens,
    structured_tokens,
    silu_gated_tokens,
    principal_subspace,
    weights,
    make_inputs,
)
