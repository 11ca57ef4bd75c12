"""Parameter, flop and byte accounting of the projected linear layer.

Storage letters: a layer maps K input features to M output features for N
tokens, and keeps L principal components.
"""


def dense_params(K, M):
    """Weights of the dense layer (Section 2.1, Eq. 1)."""
    return K * M


def inference_params(K, M, L):
    """Weights needed at inference: P (K×L) and the folded weight (M×L);
    Section 2.2 (KN becomes L(K+N) in the paper's letters)."""
    return L * (K + M)


def compression(K, M, L):
    """Per-layer inference compression 1 - L(K+M)/(KM)."""
    return 1.0 - inference_params(K, M, L) / dense_params(K, M)


def tp_compression(kind, K, M, L, tp=1):
    """Compression of a tensor-parallel layer with P applied per rank
    (Appendix B.2, Table 2 caption).  A column-parallel layer (QKV, FC1) splits
    the output features; every rank sees the same input, so one K×L projection
    serves all ranks and the ratio is that of the whole layer.  A row-parallel
    layer (Proj, FC2) splits the input features; each rank has its own
    (K/tp)×L projection and an M×L folded weight."""
    if kind == "column":
        return compression(K, M, L)
    if kind == "row":
        if K % tp:
            raise ValueError("K not divisible by tp")
        return compression(K // tp, M, L)
    raise ValueError(kind)


def ideal_speedup(K, M, L):
    """Dense flops over projected flops, KM / (L(K+M)) (also the parameter ratio)."""
    return dense_params(K, M) / inference_params(K, M, L)


def projected_flops(K, M, L, N):
    """2·L·N·(K+M): the projection (2KLN) plus the folded product (2MLN)."""
    return 2 * L * N * (K + M)


def dense_flops(K, M, N):
    return 2 * M * K * N


def projected_bytes(K, M, L, N, elem=2):
    """Algorithmic HBM bytes of one call: X, P and the folded weight read once,
    Y written once."""
    return elem * (K * N + K * L + M * L + M * N)


def dense_bytes(K, M, N, elem=2):
    return elem * (K * N + M * K + M * N)


def gemm_flops(rows, cols, depth):
    return 2 * rows * cols * depth


def gemm_bytes(rows, cols, depth, elem=2):
    return elem * (rows * depth + cols * depth + rows * cols)
