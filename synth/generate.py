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
Random streams: numpy Generator seeded with SeedSequence([241005437, key, s]),
s = 0 (Q), 1 (evaluation tokens), 2 (W), 4/5 (a/b evaluation), 6/7 (a/b
calibration).  Tokens are drawn token by token, so the first n tokens of a
larger draw equal a draw of n tokens.
"""
import functools

import numpy as np
from scipy.linalg import lapack

from .bf16 import bf16_bits_from_f64, f64_from_bf16_bits
from .configs import SEED, Workload


def rng_for(key, stream):
    return np.random.default_rng(np.random.SeedSequence([SEED, int(key), int(stream)]))


def _cholesky_qr_pass(G):
    A = G.T @ G
    R, info = lapack.dpotrf(A, lower=0, clean=1)
    if info != 0:
        raise np.linalg.LinAlgError("Cholesky QR: Gram matrix not positive definite")
    Ri, info = lapack.dtrtri(R, lower=0)
    if info != 0:
        raise np.linalg.LinAlgError("Cholesky QR: singular triangular factor")
    return G @ Ri


def haar_orthogonal(K, rng):
    """Haar-distributed K×K orthogonal matrix from one seeded Gaussian draw."""
    G = rng.standard_normal((K, K))
    try:
        Q = _cholesky_qr_pass(_cholesky_qr_pass(G))
        err = np.abs(Q.T @ Q - np.eye(K)).max() if K <= 2048 else \
            np.abs(Q[:, :64].T @ Q - np.eye(K)[:64]).max()
        if err < 1e-12:
            return Q
    except np.linalg.LinAlgError:
        pass
    Q, R = np.linalg.qr(G)
    return Q * np.sign(np.diag(R))[None, :]


def spectrum(K, floor=0.0):
    i = np.arange(1, K + 1, dtype=np.float64)
    return 1.0 / i + floor


def gaussian_tokens(Q, lam, N, rng):
    """N tokens (rows) drawn from N(0, Q·diag(lam)·Qᵀ), token-major [N][K]."""
    K = Q.shape[0]
    G = rng.standard_normal((N, K))
    return (G * np.sqrt(lam)[None, :]) @ Q.T


def structured_tokens(w, N, stream_g=1):
    Q = _haar_cached(w.cov_key, w.K)
    return gaussian_tokens(Q, spectrum(w.K, w.lam_floor), N, rng_for(w.cov_key, stream_g))


def silu_gated_tokens(Q, lam, N, rng_a, rng_b):
    """SiLU(a)*b with a, b independent structured tokens; SiLU(t) = t/(1+e^-t)."""
    a = gaussian_tokens(Q, lam, N, rng_a)
    b = gaussian_tokens(Q, lam, N, rng_b)
    return a / (1.0 + np.exp(-a)) * b


def principal_subspace(Xc, L):
    """Top-L eigenvectors (as rows, [L][K]) of the sample second moment of the
    calibration tokens Xc [n][K], with the eigenvalues in decreasing order.
    Each eigenvector's largest-magnitude entry is made positive."""
    n = Xc.shape[0]
    C = (Xc.T @ Xc) / n
    d, V = np.linalg.eigh(C)
    order = np.argsort(d)[::-1]
    d = d[order]
    V = V[:, order[:L]]
    idx = np.argmax(np.abs(V), axis=0)
    V = V * np.sign(V[idx, np.arange(L)])[None, :]
    return np.ascontiguousarray(V.T), d


def weights(M, K, rng):
    return rng.standard_normal((M, K)) / np.sqrt(K)


@functools.lru_cache(maxsize=4)
def _haar_cached(key, K):
    Q = haar_orthogonal(K, rng_for(key, 0))
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
    bfloat16 patterns, or float32)."""

    def __init__(self, w, X, Pt, W, meta):
        self.w = w
        self.X, self.X_s = _round(X, w.dtype)
        self.Pt, self.Pt_s = _round(Pt, w.dtype)
        self.W, self.W_s = _round(W, w.dtype)
        self.meta = meta


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
    if w.proj == "leading":
        Pt = np.ascontiguousarray(Q[:, :w.L].T)
    elif w.proj == "calibrated":
        if w.recipe != "silu_gated":
            raise ValueError("calibrated P is defined for the silu_gated recipe")
        Xc = silu_gated_tokens(Q, lam, w.n_cal, rng_for(w.cov_key, 6), rng_for(w.cov_key, 7))
        Pt, d = principal_subspace(Xc, w.L)
        meta["eig"] = d
        meta["eig_gap"] = float(d[w.L - 1] - d[w.L]) if w.L < len(d) else float("inf")
    else:
        raise ValueError(w.proj)
    W = weights(w.M, w.K, rng_for(w.w_key, 2))
    return Inputs(w, X, Pt, W, meta)


@functools.lru_cache(maxsize=2)
def _make_cached(key, w):
    return _make(w)


def make_inputs(w: Workload):
    """Inputs of one workload (cached per process for the last two workloads)."""
    return _make_cached(w.key(), w)
