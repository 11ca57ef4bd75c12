"""ESPACE projected linear layer on MI355X (gfx950): Python binding of libespace.so.

Y = (W·P)·(Pᵀ·X)  (Sakr & Khailany, ESPACE, Section 2.2, Eq. 3), with the
folded weight W·P computed once and the projection and expansion computed per
call by hand-written HIP kernels.  Importing the package loads the library;
there is no other implementation behind these functions.
"""
from ._lib import (  # noqa: F401
    ABI_VERSION,
    BF16,
    F32,
    OP_AUTOCORR,
    OP_BACKWARD,
    OP_DENSE,
    OP_DENSE_BACKWARD,
    OP_EXPAND,
    OP_FOLD,
    OP_PROJECT,
    OP_PCA,
    OP_SYMPRODUCT,
    OP_PROJECTED_LINEAR,
    OP_PROJECTED_LINEAR_MXFP8,
    MXTensor,
    mx_empty,
    espace_quantize_mxfp8,
    espace_project_mxfp8,
    espace_expand_mxfp8,
    espace_projected_linear_mxfp8,
    EspaceError,
    espace_autocorrelation_update,
    espace_dense_linear,
    espace_dense_linear_backward,
    espace_expand,
    espace_fold_weights,
    espace_principal_components,
    espace_project,
    espace_projected_linear,
    espace_projected_linear_backward,
    espace_projected_linear_noalloc,
    espace_set_wait_limit,
    espace_symmetrized_product,
    espace_wait_timeouts,
    espace_workspace_bytes,
    header_functions,
    lib,
    padded_empty,
)
