"""Checks that pin the CPU oracle to facts the paper and the mathematics fix.

Each pin takes a namespace `o` exposing the oracle's functions and raises
AssertionError when the oracle disagrees with the fact.  The pins do not
re-type the oracle's formulas: they compare it with brute-force loop sums,
with a different formula for the same quantity (Eq. 6 instead of Eq. 3),
with special cases that reduce to a plain product, with exact results of
permutation matrices, and with the identities of Theorem 1, Proposition 1
and Theorem 2.
"""
import itertools
import math

import numpy as np

from oracle import brute

RTOL = 1e-12


def _rng(seed):
    return np.random.default_rng(np.random.SeedSequence([20241005, seed]))


def _orthonormal(K, L, rng):
    q, r = np.linalg.qr(rng.standard_normal((K, L)))
    return q * np.sign(np.diag(r))[None, :]


def _close(a, b, rtol=RTOL, what=""):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, f"{what}: shape {a.shape} != {b.shape}"
    scale = max(np.abs(b).max(), 1e-300)
    err = np.abs(a - b).max() / scale
    assert err <= rtol, f"{what}: max rel err {err:.3e} > {rtol:.1e}"


def _tiny_case(seed, K=7, M=5, L=3, N=4):
    rng = _rng(seed)
    W = rng.standard_normal((M, K))
    X = rng.standard_normal((N, K))
    Pt = _orthonormal(K, L, rng).T.copy()
    return W, X, Pt


# -- pins --------------------------------------------------------------------

def pin_brute_force(o):
    """Every product equals its entry-by-entry exactly rounded sum (math.fsum)
    on tiny non-square shapes (Section 2.2, Eq. 3; Section 2.1, Eq. 1)."""
    for seed, (K, M, L, N) in enumerate([(7, 5, 3, 4), (6, 9, 6, 2), (8, 3, 1, 5)]):
        W, X, Pt = _tiny_case(seed, K, M, L, N)
        Wf = o.fold(W, Pt)
        Z = o.project(Pt, X)
        _close(Wf, brute.bf_fold(W.tolist(), Pt.tolist()), what="fold")
        _close(Z, brute.bf_project(Pt.tolist(), X.tolist()), what="project")
        _close(o.expand(Z, Wf), brute.bf_expand(Z.tolist(), Wf.tolist()), what="expand")
        _close(o.dense(X, W), brute.bf_dense(X.tolist(), W.tolist()), what="dense")
        _close(o.reconstruct(Pt, X), brute.bf_reconstruct(Pt.tolist(), X.tolist()),
               what="reconstruct")
        # the composed layer against the loops composed by hand
        Yb = brute.bf_expand(brute.bf_project(Pt.tolist(), X.tolist()),
                             brute.bf_fold(W.tolist(), Pt.tolist()))
        _close(o.projected_linear_from_weights(X, Pt, W), Yb, what="projected_linear")
        _close(o.projected_linear(X, Pt, Wf), Yb, what="projected_linear(Wf)")


def pin_associativity(o):
    """(PᵀW)ᵀ(PᵀX) = Wᵀ(PPᵀX) (Eq. 3), with PPᵀX evaluated token by token as
    Σ_i <p_i, x> p_i (Eq. 6) and the outer product as a plain dense layer."""
    rng = _rng(100)
    K, M, L, N = 48, 40, 12, 30
    W = rng.standard_normal((M, K))
    X = rng.standard_normal((N, K))
    Pt = _orthonormal(K, L, rng).T.copy()
    Y = o.projected_linear_from_weights(X, Pt, W)
    Xt = brute.bf_reconstruct(Pt.tolist(), X.tolist())
    Y2 = brute.bf_dense(Xt, W.tolist())
    _close(Y, Y2, rtol=1e-11, what="associativity")


def pin_full_rank_identity(o):
    """L = K with orthonormal P gives PPᵀ = I, so the layer equals WᵀX
    (Section 2.2: PPᵀ differs from the identity only when L < K)."""
    rng = _rng(200)
    K, M, N = 32, 20, 16
    W = rng.standard_normal((M, K))
    X = rng.standard_normal((N, K))
    Pt = _orthonormal(K, K, rng).T.copy()
    _close(o.projected_linear_from_weights(X, Pt, W),
           brute.bf_dense(X.tolist(), W.tolist()), rtol=1e-11, what="L=K identity")


def pin_rotation_invariance(o):
    """Replacing P by P·R with R orthogonal (L×L) leaves the layer unchanged,
    since (PR)(PR)ᵀ = PPᵀ; a mistake that breaks the pairing of the two P
    factors changes the result."""
    rng = _rng(300)
    K, M, L, N = 24, 18, 9, 11
    W = rng.standard_normal((M, K))
    X = rng.standard_normal((N, K))
    P = _orthonormal(K, L, rng)
    R = _orthonormal(L, L, rng)
    Y1 = o.projected_linear_from_weights(X, P.T.copy(), W)
    Y2 = o.projected_linear_from_weights(X, (P @ R).T.copy(), W)
    _close(Y1, Y2, rtol=1e-11, what="rotation invariance")


def pin_selection_matrix(o):
    """P whose columns are distinct signed unit vectors ±e_j: the folded weight
    is exactly ±W[:, j] and the projection exactly ±X[:, j] (products with ±1
    and sums of zeros are exact)."""
    rng = _rng(400)
    K, M, L, N = 16, 7, 5, 6
    W = rng.standard_normal((M, K))
    X = rng.standard_normal((N, K))
    J = rng.permutation(K)[:L]
    s = rng.choice([-1.0, 1.0], size=L)
    Pt = np.zeros((L, K))
    Pt[np.arange(L), J] = s
    Wf = o.fold(W, Pt)
    Z = o.project(Pt, X)
    assert np.array_equal(Wf, W[:, J] * s[None, :]), "fold with selection P"
    assert np.array_equal(Z, X[:, J] * s[None, :]), "project with selection P"
    Y = o.expand(Z, Wf)
    _close(Y, brute.bf_dense((X[:, J]).tolist(), (W[:, J]).tolist()), what="selection expand")


def _hadamard(K):
    H = np.array([[1.0]])
    while H.shape[0] < K:
        H = np.block([[H, H], [H, -H]])
    return H


def pin_hadamard(o):
    """Sylvester-Hadamard/sqrt(K) is orthonormal; with L = K the layer is WᵀX,
    and with L < K it keeps exactly the leading Hadamard directions."""
    rng = _rng(500)
    K, M, N = 64, 10, 9
    W = rng.standard_normal((M, K))
    X = rng.standard_normal((N, K))
    H = _hadamard(K) / np.sqrt(K)
    _close(o.projected_linear_from_weights(X, H.T.copy(), W),
           brute.bf_dense(X.tolist(), W.tolist()), rtol=1e-11, what="Hadamard L=K")


def pin_exact_rank_reconstruction(o):
    """Tokens of exact rank r <= L: the top-L eigenvectors of the calibrated
    autocorrelation span them, so PPᵀX = X and the layer equals WᵀX (consequence
    of Theorem 1: the minimal mean squared error is then zero)."""
    rng = _rng(600)
    K, M, r, L, N = 40, 12, 6, 8, 50
    basis = _orthonormal(K, r, rng)
    X = (rng.standard_normal((N, r)) @ basis.T)
    W = rng.standard_normal((M, K))
    C = o.autocorrelation([X[:25], X[25:]])
    Pt, d = o.principal_components(C, L)
    _close(o.reconstruct(Pt, X), X, rtol=1e-10, what="rank<=L reconstruction")
    _close(o.projected_linear_from_weights(X, Pt, W),
           brute.bf_dense(X.tolist(), W.tolist()), rtol=1e-10, what="rank<=L layer")


def pin_tail_eigenvalue_identity(o):
    """From the proof of Theorem 1: the MSE of the projection equals
    E||x||² − Σ_{i<=L} p_iᵀ C_X p_i, which for the principal eigenvectors is the
    sum of the discarded eigenvalues: (1/N)||X − PPᵀX||² = Σ_{i>L} d_i."""
    rng = _rng(700)
    K, L, N = 20, 7, 300
    A = rng.standard_normal((K, K)) * (1.0 / np.arange(1, K + 1))[None, :]
    X = rng.standard_normal((N, K)) @ A.T
    C = o.autocorrelation([X])
    Pt, d = o.principal_components(C, L)
    mse = np.sum((X - o.reconstruct(Pt, X)) ** 2) / N
    tail = float(np.sum(d[L:]))
    assert abs(mse - tail) <= 1e-10 * max(tail, 1e-300), f"tail identity {mse} vs {tail}"
    # and the eigenvalues are those of the batch second moment, in decreasing order
    assert np.all(np.diff(d) <= 1e-12), "eigenvalues not in decreasing order"
    brute_C = np.array([[sum(X[n, i] * X[n, j] for n in range(N)) / N for j in range(K)]
                        for i in range(K)])
    _close(C, brute_C, rtol=1e-12, what="autocorrelation")


def pin_batch_average(o):
    """Eq. 5: C_X is the average over calibration batches of X_i X_iᵀ / M_i;
    with batches of unequal size that is not the pooled second moment."""
    rng = _rng(750)
    K = 5
    b1 = rng.standard_normal((3, K))
    b2 = rng.standard_normal((9, K)) * 2.0
    C = o.autocorrelation([b1, b2])
    C1 = np.array([[sum(b1[n, i] * b1[n, j] for n in range(3)) / 3 for j in range(K)]
                   for i in range(K)])
    C2 = np.array([[sum(b2[n, i] * b2[n, j] for n in range(9)) / 9 for j in range(K)]
                   for i in range(K)])
    _close(C, (C1 + C2) / 2, rtol=1e-12, what="batch average")


def pin_theorem1_brute_force(o):
    """Theorem 1 on tiny inputs: no random orthonormal P (K <= 6) attains a
    lower empirical MSE than the top-L eigenvectors of C_X; Corollary 1 likewise
    for the normalised MSE with the normalised autocorrelation."""
    rng = _rng(800)
    for K, L in ((4, 2), (6, 3), (5, 1)):
        X = rng.standard_normal((60, K)) @ rng.standard_normal((K, K))
        X[:5] *= 20.0  # a few large outliers, so MSE and NMSE optima differ
        Pt, _ = o.principal_components(o.autocorrelation([X]), L)
        Pn, _ = o.principal_components(o.normalized_autocorrelation([X]), L)

        def mse(Ptr):
            return np.mean(np.sum((X - o.reconstruct(Ptr, X)) ** 2, axis=1))

        def nmse(Ptr):
            e = np.sum((X - o.reconstruct(Ptr, X)) ** 2, axis=1)
            return np.mean(e / np.sum(X ** 2, axis=1))

        best, bestn = mse(Pt), nmse(Pn)
        for _ in range(2000):
            Pr = _orthonormal(K, L, rng).T.copy()
            assert mse(Pr) >= best - 1e-12, "random P beats Theorem 1"
            assert nmse(Pr) >= bestn - 1e-12, "random P beats Corollary 1"
        # coordinate subspaces too (exhaustive over column subsets)
        for J in itertools.combinations(range(K), L):
            Pc = np.zeros((L, K))
            Pc[np.arange(L), list(J)] = 1.0
            assert mse(Pc) >= best - 1e-12


def pin_norm_and_bound(o):
    """Proposition 1 (proof, Appendix A.3): ||x̃|| <= ||x|| for every token, and
    per sample (y − ỹ)² <= 2||w||²||x||² − 2<w,x><w,x̃>, with y from the dense
    layer and ỹ from the projected one."""
    rng = _rng(900)
    K, M, L, N = 12, 6, 4, 25
    W = rng.standard_normal((M, K))
    X = rng.standard_normal((N, K))
    Pt = _orthonormal(K, L, rng).T.copy()
    Xt = o.reconstruct(Pt, X)
    assert np.all(np.sum(Xt ** 2, 1) <= np.sum(X ** 2, 1) * (1 + 1e-12)), "||x~|| > ||x||"
    Y = np.asarray(o.dense(X, W))
    Yt = np.asarray(o.projected_linear_from_weights(X, Pt, W))
    wx = X @ W.T
    wxt = Xt @ W.T
    bound = 2 * np.sum(W ** 2, 1)[None, :] * np.sum(X ** 2, 1)[:, None] - 2 * wx * wxt
    assert np.all((Y - Yt) ** 2 <= bound + 1e-9), "Proposition 1 bound violated"
    # the projected layer is the dense layer applied to x̃
    _close(Yt, wxt, rtol=1e-11, what="projected = dense(x~)")


def pin_sampled(o):
    """Outputs at sampled positions equal the same entries of the whole layer."""
    rng = _rng(1000)
    K, M, L, N = 30, 26, 10, 19
    W = rng.standard_normal((M, K))
    X = rng.standard_normal((N, K))
    Pt = _orthonormal(K, L, rng).T.copy()
    rows = np.array([0, 5, 18, 7])
    cols = np.array([25, 0, 3, 11, 12])
    Yb = np.array(brute.bf_expand(brute.bf_project(Pt.tolist(), X.tolist()),
                                  brute.bf_fold(W.tolist(), Pt.tolist())))
    _close(o.sampled_projected_linear(X, Pt, W, rows, cols), Yb[np.ix_(rows, cols)],
           what="sampled projected")
    _close(o.sampled_dense(X, W, rows, cols),
           np.array(brute.bf_dense(X.tolist(), W.tolist()))[np.ix_(rows, cols)],
           what="sampled dense")


def pin_rel_fro(o):
    """Relative Frobenius error on values with a known answer."""
    ref = np.array([[3.0, 0.0], [0.0, 4.0]])
    a = ref + np.array([[0.0, 0.0], [0.0, 0.5]])
    assert abs(o.rel_fro(a, ref) - 0.1) < 1e-15
    assert o.rel_fro(ref, ref) == 0.0


def pin_gomse_expectation(o):
    """Theorem 2: over independent draws of x (the tokens of X) and w (the rows
    of W) the average of x xᵀ w wᵀ + w wᵀ x xᵀ, summed pair by pair, is the
    oracle's C_X·C_W + C_W·C_X; with unit-norm x and w, its normalised Ĉ."""
    rng = _rng(1100)
    K, N, M = 5, 7, 6
    X = rng.standard_normal((N, K))
    W = rng.standard_normal((M, K))
    acc = np.zeros((K, K))
    accn = np.zeros((K, K))
    for n in range(N):
        x = X[n]
        xn = x / np.sqrt(sum(v * v for v in x))
        for m in range(M):
            w = W[m]
            wn = w / np.sqrt(sum(v * v for v in w))
            for i in range(K):
                for j in range(K):
                    # (x xᵀ w wᵀ)_ij = x_i (x·w) w_j, and its transpose
                    xw = sum(x[k] * w[k] for k in range(K))
                    acc[i, j] += x[i] * xw * w[j] + w[i] * xw * x[j]
                    xwn = sum(xn[k] * wn[k] for k in range(K))
                    accn[i, j] += xn[i] * xwn * wn[j] + wn[i] * xwn * xn[j]
    _close(o.gomse_matrix(o.autocorrelation([X]), o.autocorrelation([W])), acc / (N * M),
           rtol=1e-12, what="GO-MSE matrix")
    _close(o.gomse_matrix(o.normalized_autocorrelation([X]), o.normalized_autocorrelation([W])),
           accn / (N * M), rtol=1e-12, what="normalised GO-MSE matrix")


def pin_nlmse_expectation(o):
    """Theorem 2's NL-MSE matrix as its proof calibrates it: per sequence, the
    average over all (activation, gradient) pairs of the sequence of
    x xᵀ g gᵀ + g gᵀ x xᵀ, summed pair by pair, then the mean over sequences;
    the normalised variant with unit vectors."""
    rng = _rng(1500)
    K = 4
    seqs = [(rng.standard_normal((5, K)), rng.standard_normal((5, K))),
            (rng.standard_normal((3, K)), rng.standard_normal((3, K)))]
    for normalized in (False, True):
        tot = np.zeros((K, K))
        for X, G in seqs:
            acc = np.zeros((K, K))
            for x in X:
                if normalized:
                    x = x / np.sqrt(sum(v * v for v in x))
                for g in G:
                    if normalized:
                        g = g / np.sqrt(sum(v * v for v in g))
                    xg = sum(x[k] * g[k] for k in range(K))
                    for i in range(K):
                        for j in range(K):
                            acc[i, j] += x[i] * xg * g[j] + g[i] * xg * x[j]
            tot += acc / (len(X) * len(G))
        _close(o.nlmse_matrix(seqs, normalized=normalized), tot / len(seqs), rtol=1e-12,
               what="NL-MSE matrix" + (" (normalised)" if normalized else ""))


def pin_gomse_bound_identity(o):
    """Theorem 2's derivation: for any orthonormal P, the mean over pairs of
    2<w,x><w,x̃> (the part of Proposition 1's bound that P controls) equals
    Σ_i p_iᵀ C p_i; and when C's largest eigenvalues are also its largest in
    magnitude, the selected P maximises it (no random orthonormal P does
    better), i.e. minimises the bound."""
    rng = _rng(1200)
    K, N, M, L = 5, 40, 30, 2
    X = rng.standard_normal((N, K)) @ rng.standard_normal((K, K))
    W = rng.standard_normal((M, K)) @ rng.standard_normal((K, K))
    C = o.gomse_matrix(o.autocorrelation([X]), o.autocorrelation([W]))

    def q_pairs(Pt):
        Xt = o.reconstruct(Pt, X)
        return float(np.mean(2 * (X @ W.T) * (Xt @ W.T)))

    def q_form(Pt):
        return float(sum(p @ C @ p for p in np.asarray(Pt)))

    for _ in range(20):
        Pr = _orthonormal(K, L, rng).T.copy()
        _close(q_pairs(Pr), q_form(Pr), rtol=1e-11, what="bound term vs quadratic form")
    d = np.linalg.eigvalsh(C)
    assert abs(d[0]) < d[-1] and abs(d[1]) < d[-2], "test matrix: top eigenvalues not the largest in magnitude"
    Pt, _ = o.principal_components_by_magnitude(C, L)
    best = q_pairs(Pt)
    for _ in range(3000):
        assert q_pairs(_orthonormal(K, L, rng).T.copy()) <= best + 1e-9, "random P beats Theorem 2"


def pin_magnitude_order(o):
    """Selection by absolute eigenvalue on a matrix of known spectrum: a
    rotated diagonal with eigenvalues 3, -5, 1, -0.9, 0.5 gives -5, 3, 1,
    -0.9, 0.5, and the rotated unit vectors."""
    rng = _rng(1300)
    Q = _orthonormal(5, 5, rng)
    lam = np.array([3.0, -5.0, 1.0, -0.9, 0.5])
    C = (Q * lam[None, :]) @ Q.T
    Pt, d = o.principal_components_by_magnitude((C + C.T) / 2, 4)
    _close(d, [-5.0, 3.0, 1.0, -0.9, 0.5], rtol=1e-12, what="order")
    for row, col in zip(Pt, [1, 0, 2, 3]):
        assert abs(abs(row @ Q[:, col]) - 1.0) < 1e-12, "eigenvector"


def pin_training_gradients(o):
    """The training view's gradients against central finite differences of the
    scalar loss ℓ = Σ R ⊙ Y(X, W) (so ∂ℓ/∂Y = R), entry by entry, and its
    forward against the inference form (PᵀW)ᵀ(PᵀX) (associativity)."""
    rng = _rng(1400)
    K, M, L, N = 6, 4, 3, 5
    X = rng.standard_normal((N, K))
    W = rng.standard_normal((M, K))
    Pt = _orthonormal(K, L, rng).T.copy()
    R = rng.standard_normal((N, M))
    Y, _ = o.train_forward(X, Pt, W)
    _close(Y, o.projected_linear_from_weights(X, Pt, W), rtol=1e-12, what="training forward")
    dX, dW = o.train_backward(R, X, Pt, W)

    def loss(Xv, Wv):
        return float(np.sum(R * o.train_forward(Xv, Pt, Wv)[0]))

    # with a full-rank P (PPᵀ = I) the training view is the dense layer
    Pf = _orthonormal(K, K, rng).T.copy()
    for a, b, what in zip(o.train_backward(R, X, Pf, W), o.dense_backward(R, X, W), ("dX", "dW")):
        _close(a, b, rtol=1e-11, what="full-rank training gradient " + what)
    h = 1e-6
    for (n, k) in itertools.product(range(N), range(K)):
        Xp, Xm = X.copy(), X.copy()
        Xp[n, k] += h
        Xm[n, k] -= h
        assert abs((loss(Xp, W) - loss(Xm, W)) / (2 * h) - dX[n, k]) < 1e-7, ("dX", n, k)
    for (m, k) in itertools.product(range(M), range(K)):
        Wp, Wm = W.copy(), W.copy()
        Wp[m, k] += h
        Wm[m, k] -= h
        assert abs((loss(X, Wp) - loss(X, Wm)) / (2 * h) - dW[m, k]) < 1e-7, ("dW", m, k)


# -- MX-FP8 (the low-precision reading of Section 1.1 / Section 5) ------------

def _torch_e4m3_table():
    """float64 values of the 256 E4M3 bit patterns by torch's float8_e4m3fn
    (a library the oracle does not use)."""
    import torch
    return torch.arange(256, dtype=torch.int32).to(torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()


def pin_e4m3_decode_table(o):
    """Every E4M3 bit pattern decodes to torch's value (NaN patterns
    included), and encode inverts decode on all 254 finite patterns."""
    ref = _torch_e4m3_table()
    got = o.e4m3_decode(np.arange(256))
    assert np.array_equal(np.isnan(got), np.isnan(ref)), "e4m3 NaN patterns"
    fin = ~np.isnan(ref)
    assert np.array_equal(got[fin], ref[fin]), "e4m3 decode"
    codes = np.arange(256)[fin]
    back = o.e4m3_encode(ref[fin])
    assert np.array_equal(back.astype(np.int64), codes), "e4m3 encode"
    # closed form: 448 is the largest finite value, 2^-9 the smallest positive one
    assert np.nanmax(ref) == 448.0 and np.min(ref[fin & (ref > 0)]) == 2.0 ** -9


def pin_e4m3_round(o):
    """Rounding to E4M3 agrees with torch's float32 -> float8_e4m3fn cast on
    every in-range value of a random sweep, and takes the ties, the
    saturation and the subnormal steps a reader can check by hand."""
    import torch
    rng = _rng(40)
    v = np.concatenate([rng.standard_normal(20000) * 30, rng.standard_normal(20000) * 1e-2,
                        rng.uniform(-448, 448, 20000)]).astype(np.float32).astype(np.float64)
    ref = torch.from_numpy(v.astype(np.float32)).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(o.e4m3_round(v), ref), "e4m3 rounding vs torch"
    cases = {1.0625: 1.0, 1.1875: 1.25, 17.0: 16.0, 19.0: 20.0, 2.0 ** -10: 0.0, 3 * 2.0 ** -10: 2.0 ** -8,
             5 * 2.0 ** -10: 2.0 ** -8, 448.0: 448.0, 460.0: 448.0, 500.0: 448.0, 1e30: 448.0, -1e30: -448.0,
             0.3: 0.3125, -0.3: -0.3125}
    for x, want in cases.items():
        got = float(o.e4m3_round(np.array([x]))[0])
        assert got == want, f"e4m3_round({x}) = {got}, expected {want}"


def _mx_blocks_case(seed):
    rng = _rng(seed)
    A = rng.standard_normal((6, 75)) * np.exp(rng.uniform(-12, 12, (6, 1)))
    A[1, 32:64] = 0.0                         # an all-zero block
    A[2, :32] *= 1e-30                        # tiny magnitudes
    A[3, 5] = 2.0 ** 20                       # one large entry dominating its block
    A[4, 64:] = [2.0 ** k for k in range(-5, 6)]    # powers of two in the ragged tail block
    return A


def pin_mx_quantize(o):
    """MX-FP8 blocks (32 along the row, ragged tail): the scale byte is the
    brute-force smallest S with max|v| < 2^(S + 9) (zero blocks: byte 0), every
    nonzero block's largest element lies in [256, 448], every element is
    within half an E4M3 step of v / 2^S, and values already on the MX grid
    come back unchanged."""
    for seed in (41, 42, 43):
        A = _mx_blocks_case(seed)
        q, sb = o.mx_quantize(A)
        rows, cols = A.shape
        nb = -(-cols // 32)
        assert q.shape == A.shape and sb.shape == (rows, nb)
        for r in range(rows):
            for b in range(nb):
                blk = A[r, 32 * b:32 * b + 32]
                amax = float(np.abs(blk).max())
                if amax == 0.0:
                    assert sb[r, b] == 0, "zero block scale"
                    assert np.all(q[r, 32 * b:32 * b + 32] == 0)
                    continue
                S = next(S for S in range(-400, 400) if amax < 2.0 ** (S + 9))
                assert int(sb[r, b]) == min(max(S + 127, 0), 254), (r, b, int(sb[r, b]), S)
                Se = int(sb[r, b]) - 127
                qb = q[r, 32 * b:32 * b + 32]
                if S + 127 >= 0:
                    assert 256.0 <= np.abs(qb).max() <= 448.0, (r, b, np.abs(qb).max())
                for x, y in zip(blk / 2.0 ** Se, qb):
                    a = abs(x)
                    step = 2.0 ** -9 if a < 2.0 ** -6 else 2.0 ** (math.floor(math.log2(a)) - 3)
                    assert abs(min(a, 448.0) - abs(y)) <= step / 2 * (1 + 1e-12), (x, y)
        deq = o.mx_dequantize(q, sb)
        q2, sb2 = o.mx_quantize(deq)
        assert np.array_equal(q2, q) and np.array_equal(sb2, sb), "MX round trip"


def _mx_inputs(seed, N, K, L, M):
    rng = _rng(seed)
    X = rng.standard_normal((N, K)) * np.exp(rng.uniform(-2, 2, (N, 1)))
    Pt = _orthonormal(K, L, rng).T.copy()
    Wf = rng.standard_normal((M, L)) / np.sqrt(L)
    return o_q(X), o_q(Pt), o_q(Wf)


def o_q(A):
    from oracle import mxfp8_ref
    return mxfp8_ref.mx_quantize(A)


def pin_mx_layer_brute_force(o):
    """The MX-FP8 layer on tiny shapes: Z and Y equal entry-by-entry exactly
    rounded loop sums (math.fsum) over the decoded operands, with Z
    re-quantised in between (Section 2.2, Eq. 3)."""
    for seed, (N, K, L, M) in enumerate([(3, 40, 33, 5), (2, 64, 7, 3), (4, 70, 64, 9)]):
        (Xq, Xs), (Pq, Ps), (Wq, Ws) = _mx_inputs(50 + seed, N, K, L, M)
        Xd, Pd, Wd = o.mx_dequantize(Xq, Xs), o.mx_dequantize(Pq, Ps), o.mx_dequantize(Wq, Ws)
        Z = o.mx_project(Xq, Xs, Pq, Ps)
        _close(Z, brute.bf_project(Pd.tolist(), Xd.tolist()), what="mx project")
        Y, Zq, Zs = o.mx_projected_linear(Xq, Xs, Pq, Ps, Wq, Ws)
        Zq2, Zs2 = o.mx_quantize(Z)
        assert np.array_equal(Zq, Zq2) and np.array_equal(Zs, Zs2), "layer re-quantises Z"
        Zd = o.mx_dequantize(Zq, Zs)
        _close(Y, brute.bf_expand(Zd.tolist(), Wd.tolist()), what="mx layer")
        _close(o.mx_expand(Zq, Zs, Wq, Ws), Y, what="mx expand")


def pin_mx_block_selection(o):
    """With P selecting whole 32-blocks of coordinates, Z is exactly the
    selected decoded columns of X, its re-quantisation returns X's codes and
    scales for those blocks, and Y is the plain product of those columns with
    the decoded folded weight."""
    rng = _rng(60)
    N, K, M = 5, 128, 7
    X = rng.standard_normal((N, K)) * np.exp(rng.uniform(-3, 3, (N, K // 32))).repeat(32, axis=1)
    Xq, Xs = o.mx_quantize(X)
    sel_blocks = [2, 0]
    sel = np.concatenate([np.arange(32 * b, 32 * b + 32) for b in sel_blocks])
    Pt = np.zeros((len(sel), K))
    Pt[np.arange(len(sel)), sel] = 1.0
    Pq, Ps = o.mx_quantize(Pt)
    Wq, Ws = o.mx_quantize(rng.standard_normal((M, len(sel))))
    Y, Zq, Zs = o.mx_projected_linear(Xq, Xs, Pq, Ps, Wq, Ws)
    assert np.array_equal(Zq, Xq[:, sel]), "selected codes"
    assert np.array_equal(Zs, Xs[:, sel_blocks]), "selected scales"
    ref = o.mx_dequantize(Xq, Xs)[:, sel] @ o.mx_dequantize(Wq, Ws).T
    assert np.array_equal(Y, ref), "selected product"


ALL_PINS = [
    pin_brute_force,
    pin_associativity,
    pin_full_rank_identity,
    pin_rotation_invariance,
    pin_selection_matrix,
    pin_hadamard,
    pin_exact_rank_reconstruction,
    pin_tail_eigenvalue_identity,
    pin_batch_average,
    pin_theorem1_brute_force,
    pin_norm_and_bound,
    pin_sampled,
    pin_rel_fro,
    pin_gomse_expectation,
    pin_nlmse_expectation,
    pin_gomse_bound_identity,
    pin_magnitude_order,
    pin_training_gradients,
    pin_e4m3_decode_table,
    pin_e4m3_round,
    pin_mx_quantize,
    pin_mx_layer_brute_force,
    pin_mx_block_selection,
]
