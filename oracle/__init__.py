"""CPU oracle for the ESPACE projected linear layer.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package; the library and its Python binding
never do, and this package imports nothing from them.
"""
from .espace_ref import (  # noqa: F401
    fold,
    project,
    expand,
    projected_linear,
    projected_linear_from_weights,
    dense,
    reconstruct,
    rel_fro,
    sampled_projected_linear,
    sampled_dense,
    autocorrelation,
    principal_components,
    normalized_autocorrelation,
    gomse_matrix,
    nlmse_matrix,
    principal_components_by_magnitude,
    train_forward,
    train_backward,
    dense_backward,
)
from .mxfp8_ref import (  # noqa: F401
    e4m3_round,
    e4m3_decode,
    e4m3_encode,
    mx_quantize,
    mx_scale,
    mx_dequantize,
    mx_project,
    mx_expand,
    mx_projected_linear,
)
from .brute import (  # noqa: F401
    bf_fold,
    bf_project,
    bf_expand,
    bf_dense,
    bf_reconstruct,
)
