"""Pure-Python loop versions of the products, for tiny shapes only.

TEST INFRASTRUCTURE ONLY.  Each output entry is one exactly-rounded sum
(math.fsum) of its defining products, written index by index from the same
definitions as the float64 reference (Section 2.2, Eq. 3 and Eq. 6), in the
storage orientation W[M][K], Pt[L][K], X[N][K], Wf[M][L], Z[N][L], Y[N][M].
"""
import math


def _shape(a):
    return len(a), len(a[0])


def bf_fold(W, Pt):
    """Wf[m][l] = Σ_k W[m][k]·P[k][l], with P[k][l] = Pt[l][k]."""
    M, K = _shape(W)
    L, _ = _shape(Pt)
    return [[math.fsum(W[m][k] * Pt[l][k] for k in range(K)) for l in range(L)]
            for m in range(M)]


def bf_project(Pt, X):
    """Z[n][l] = <p_l, x_n> = Σ_k P[k][l]·X[n][k]."""
    L, K = _shape(Pt)
    N, _ = _shape(X)
    return [[math.fsum(Pt[l][k] * X[n][k] for k in range(K)) for l in range(L)]
            for n in range(N)]


def bf_expand(Z, Wf):
    """Y[n][m] = Σ_l Wf[m][l]·Z[n][l]."""
    N, L = _shape(Z)
    M, _ = _shape(Wf)
    return [[math.fsum(Wf[m][l] * Z[n][l] for l in range(L)) for m in range(M)]
            for n in range(N)]


def bf_dense(X, W):
    """Y[n][m] = Σ_k W[m][k]·X[n][k]."""
    N, K = _shape(X)
    M, _ = _shape(W)
    return [[math.fsum(W[m][k] * X[n][k] for k in range(K)) for m in range(M)]
            for n in range(N)]


def bf_reconstruct(Pt, X):
    """x̃_n[k] = Σ_l <p_l, x_n> P[k][l]  (Eq. 6)."""
    L, K = _shape(Pt)
    N, _ = _shape(X)
    out = []
    for n in range(N):
        coef = [math.fsum(Pt[l][k] * X[n][k] for k in range(K)) for l in range(L)]
        out.append([math.fsum(coef[l] * Pt[l][k] for l in range(L)) for k in range(K)])
    return out
