"""Seeded generators: Haar-random rotations, structured activations, weights.

Recipe (all in float64, then rounded once to the workload's storage type):
  Q   Haar-random K×K orthogonal: the QR factor with positive diagonal of R of a
      K×K matrix of iid N(0,1) draws (Mezzadri 2007); computed by two passes of
      Cholesky QR, which yields exactly that factor.
  lam lam_i = 1/i + floor, i = 1..K.
  X   token-major [N][K]; token n is Q·diag(sqrt(lam))·g_n with g_n iid N(0, I),
      so tokens are draws of N(0, Q·diag(lam)·Qᵀ).  A "silu_gated" workload uses
      SiLU(a)*b with a, b independent tokens of that kind.
  P   "leading": the first L columns of Q; "calibrated": the top-L eigenvectors
      of the sample second moment of n_cal separate calibration tokens.
  W   [M][K] iid N(0, 1/K).
Random streams: stream s of key k fills a row-major array in blocks of 2^20
elements, block b drawn by a numpy Generator seeded with
SeedSequence([241005437, k, s, b]) (blocks are independent, so large arrays
are drawn by several threads); s = 0 (Q), 1 (evaluation tokens), 2 (W), 4/5
(a/b evaluation), 6/7 (a/b calibration), 8 (rotation of a symmetric test
matrix with a given spectrum), 9 (upstream gradients of the training view).  Tokens are drawn token by token, so
the first n tokens of a larger draw equal a draw of n tokens.

For K >= 4096 on a machine with a GPU, the dense float64 linear algebra of the
recipe (the Cholesky QR, the token products, the calibration second moment and
its eigendecomposition) runs in float64 through torch on the GPU: the same
recipe, rounded differently in the last bits than the numpy path.  It builds
inputs only; nothing of the projected linear layer is computed here.
"""
import functools
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
from scipy.linalg import lapack

from .bf16 import bf16_bits_from_f64, f64_from_bf16_bits
from .configs import SEED, Workload

_BLOCK = 1 << 20
GPU_MIN_K = 4096


def _workers():
    return max(1, min(16, os.cpu_count() or 1))


class Stream:
    """Normal draws of stream `stream` of seed key `key` (see the recipe)."""

    def __init__(self, key, stream):
        self.key, self.stream = int(key), int(stream)

    def standard_normal(self, shape):
        out = np.empty(shape, dtype=np.float64)
        flat = out.reshape(-1)

        def fill(b):
            g = np.random.default_rng(np.random.SeedSequence([SEED, self.key, self.stream, b]))
            lo = b * _BLOCK
            g.standard_normal(out=flat[lo:lo + _BLOCK])

        nb = (flat.size + _BLOCK - 1) // _BLOCK
        if nb > 1:
            with ThreadPoolExecutor(max_workers=_workers()) as ex:
                list(ex.map(fill, range(nb)))
        elif nb == 1:
            fill(0)
        return out


def rng_for(key, stream):
    return Stream(key, stream)


def _device(K):
    """torch GPU device for the float64 linear algebra of size-K recipes, or None."""
    if K < GPU_MIN_K or os.environ.get("SYNTH_CPU_ONLY"):
        return None
    try:
        import torch
        if torch.cuda.is_available():
            return torch.device("cuda:0")
    except ImportError:
        pass
    return None


def _np(t):
    return t if isinstance(t, np.ndarray) else t.cpu().numpy()


def _cholesky_qr_pass(G):
    A = G.T @ G
    R, info = lapack.dpotrf(A, lower=0, clean=1)
    if info != 0:
        raise np.linalg.LinAlgError("Cholesky QR: Gram matrix not positive definite")
    Ri, info = lapack.dtrtri(R, lower=0)
    if info != 0:
        raise np.linalg.LinAlgError("Cholesky QR: singular triangular factor")
    return G @ Ri


def _orth_err(Q):
    K = Q.shape[0]
    if K <= 2048:
        return float(abs(Q.T @ Q - np.eye(K)).max())
    return float(abs(Q[:, :64].T @ Q - np.eye(K)[:64]).max())


def haar_from_gaussian(G):
    """Q factor (positive diagonal of R) of a square Gaussian matrix, numpy."""
    try:
        Q = _cholesky_qr_pass(_cholesky_qr_pass(G))
        if _orth_err(Q) < 1e-12:
            return Q
    except np.linalg.LinAlgError:
        pass
    Q, R = np.linalg.qr(G)
    return Q * np.sign(np.diag(R))[None, :]


def _haar_torch(Gn, dev):
    import torch
    G0 = torch.from_numpy(Gn).to(dev)
    Q = G0
    ok = True
    for _ in range(2):
        R, info = torch.linalg.cholesky_ex(Q.T @ Q, upper=True)
        if int(info) != 0:
            ok = False
            break
        # Q·R⁻¹ one block of rows at a time: rows are independent, and the
        # BLAS triangular solve's workspace grows with the right-hand side
        Q = torch.cat([torch.linalg.solve_triangular(R, Q[r:r + 1024], upper=True, left=False)
                       for r in range(0, Q.shape[0], 1024)])
    if ok:
        I = torch.eye(64, Q.shape[0], dtype=Q.dtype, device=dev)
        ok = float((Q[:, :64].T @ Q - I).abs().max()) < 1e-12
    if not ok:
        Q, R = torch.linalg.qr(G0)
        Q = Q * torch.sign(torch.diagonal(R))[None, :]
    return Q


def haar_orthogonal(K, rng, device=None):
    """Haar-distributed K×K orthogonal matrix from one seeded Gaussian draw
    (numpy array, or a torch tensor on `device`)."""
    G = rng.standard_normal((K, K))
    if device is not None:
        return _haar_torch(G, device)
    return haar_from_gaussian(G)


def index_pattern(m, k):
    """Deterministic matrix entry for indexing tests: ((73m + 151k) mod 255 -
    127) / 512 for integer row and column indices (numpy arrays or torch
    tensors; m < 2^24, k < 2^16).  Every value is exact in bfloat16, so a
    matrix of any size can be built on the device in pieces and any row of it
    recomputed on the host."""
    return ((m * 73 + k * 151) % 255 - 127) / 512.0


def symmetric_with_spectrum(K, lam, key):
    """K×K symmetric matrix Q·diag(lam)·Qᵀ, Q Haar-random from stream 8 of
    `key` (float64, exactly symmetric): an input with known eigenvalues."""
    Q = haar_orthogonal(K, rng_for(key, 8))
    C = (Q * np.asarray(lam, dtype=np.float64)[None, :]) @ Q.T
    return (C + C.T) / 2


def upstream_gradient(N, M, key):
    """An upstream gradient dY [N][M] for the training-view tests: iid
    N(0, 1/M) entries from stream 9 of `key` (float64)."""
    return rng_for(key, 9).standard_normal((N, M)) / np.sqrt(M)


def spectrum(K, floor=0.0):
    i = np.arange(1, K + 1, dtype=np.float64)
    return 1.0 / i + floor


def gaussian_tokens(Q, lam, N, rng):
    """N tokens (rows) drawn from N(0, Q·diag(lam)·Qᵀ), token-major [N][K]
    (numpy, or a torch tensor when Q is one)."""
    K = Q.shape[0]
    G = rng.standard_normal((N, K))
    if isinstance(Q, np.ndarray):
        return (G * np.sqrt(lam)[None, :]) @ Q.T
    import torch
    Gt = torch.from_numpy(G).to(Q.device) * torch.from_numpy(np.sqrt(lam)).to(Q.device)[None, :]
    return Gt @ Q.T


def structured_tokens(w, N, stream_g=1):
    Q = _haar_cached(w.cov_key, w.K)
    return _np(gaussian_tokens(Q, spectrum(w.K, w.lam_floor), N, rng_for(w.cov_key, stream_g)))


def silu_gated_tokens(Q, lam, N, rng_a, rng_b):
    """SiLU(a)*b with a, b independent structured tokens; SiLU(t) = t/(1+e^-t)."""
    a = gaussian_tokens(Q, lam, N, rng_a)
    b = gaussian_tokens(Q, lam, N, rng_b)
    if isinstance(a, np.ndarray):
        return a / (1.0 + np.exp(-a)) * b
    import torch
    return a / (1.0 + torch.exp(-a)) * b


def principal_subspace(Xc, L):
    """Top-L eigenvectors (as rows, [L][K]) of the sample second moment of the
    calibration tokens Xc [n][K], with the eigenvalues in decreasing order.
    Each eigenvector's largest-magnitude entry is made positive."""
    n = Xc.shape[0]
    if isinstance(Xc, np.ndarray):
        C = (Xc.T @ Xc) / n
        d, V = np.linalg.eigh(C)
    else:
        import torch
        d, V = torch.linalg.eigh((Xc.T @ Xc) / n)
        d, V = _np(d), _np(V)
    order = np.argsort(d)[::-1]
    d = d[order]
    V = V[:, order[:L]]
    idx = np.argmax(np.abs(V), axis=0)
    V = V * np.sign(V[idx, np.arange(L)])[None, :]
    return np.ascontiguousarray(V.T), d


def weights(M, K, rng):
    W = rng.standard_normal((M, K))
    W *= 1.0 / np.sqrt(K)
    return W


@functools.lru_cache(maxsize=2)
def _haar_cached(key, K):
    Q = haar_orthogonal(K, rng_for(key, 0), _device(K))
    if isinstance(Q, np.ndarray):
        Q.setflags(write=False)
    return Q


def _round(a, dtype):
    """Round float64 to the storage type; return (exact float64 values, storage array)."""
    if dtype == "bf16":
        bits = bf16_bits_from_f64(a)
        return f64_from_bf16_bits(bits).reshape(a.shape), bits.reshape(a.shape)
    if dtype == "f32":
        s = np.ascontiguousarray(a, dtype=np.float32)
        return s.astype(np.float64), s
    raise ValueError(dtype)


class Inputs:
    """One workload's inputs.  X, Pt, W are float64 arrays holding exactly the
    rounded values; X_s, Pt_s, W_s are the same values in storage form (uint16
    bfloat16 patterns, or float32).  W may be passed already rounded, as the
    pair (exact values, storage)."""

    def __init__(self, w, X, Pt, W, meta):
        self.w = w
        self.X, self.X_s = _round(X, w.dtype)
        self.Pt, self.Pt_s = _round(Pt, w.dtype)
        self.W, self.W_s = W if isinstance(W, tuple) else _round(W, w.dtype)
        self.meta = meta


@functools.lru_cache(maxsize=2)
def _weights_rounded(key, M, K, dtype):
    """W of one seed key and shape, rounded (shared by the workloads that
    differ only in L or N)."""
    W64, Ws = _round(weights(M, K, rng_for(key, 2)), dtype)
    W64.setflags(write=False)
    Ws.setflags(write=False)
    return W64, Ws


def _make(w: Workload):
    meta = {}
    Q = _haar_cached(w.cov_key, w.K)
    lam = spectrum(w.K, w.lam_floor)
    if w.recipe == "gaussian":
        X = gaussian_tokens(Q, lam, w.N, rng_for(w.cov_key, 1))
    elif w.recipe == "silu_gated":
        X = silu_gated_tokens(Q, lam, w.N, rng_for(w.cov_key, 4), rng_for(w.cov_key, 5))
    else:
        raise ValueError(w.recipe)
    X = _np(X)
    if w.proj == "leading":
        Pt = np.ascontiguousarray(_np(Q[:, :w.L].T))
    elif w.proj == "calibrated":
        if w.recipe != "silu_gated":
            raise ValueError("calibrated P is defined for the silu_gated recipe")
        Xc = silu_gated_tokens(Q, lam, w.n_cal, rng_for(w.cov_key, 6), rng_for(w.cov_key, 7))
        Pt, d = principal_subspace(Xc, w.L)
        meta["eig"] = d
        meta["eig_gap"] = float(d[w.L - 1] - d[w.L]) if w.L < len(d) else float("inf")
    else:
        raise ValueError(w.proj)
    return Inputs(w, X, Pt, _weights_rounded(w.w_key, w.M, w.K, w.dtype), meta)


@functools.lru_cache(maxsize=2)
def _make_cached(key, w):
    return _make(w)


def make_inputs(w: Workload):
    """Inputs of one workload (cached per process for the last two workloads)."""
    return _make_cached(w.key(), w)
