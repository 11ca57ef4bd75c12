"""Plain float64 reference of the ESPACE projected linear layer.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What the method computes (paper, Section 2.2, Eq. 3): a linear layer
Y = WᵀX (Section 2.1, Eq. 1) is replaced at inference by
    Y ≈ (PᵀW)ᵀ (PᵀX)
with a static K×L matrix P of orthonormal columns; the folded weight PᵀW is
computed once before deployment ("inference view", Section 2.2), and each call
computes the projection PᵀX followed by the product with the folded weight.
The result of the method for a given P is exactly (PᵀW)ᵀ(PᵀX); it is written
out here with plain matrix products in float64.

Paper orientation vs storage.  The paper writes W as K×N_p (used transposed),
X as K×M_p (tokens as columns) and P as K×L.  Arrays here are stored
row-major as
    W[M][K]   = the paper's Wᵀ            (M output features)
    X[N][K]   = the paper's Xᵀ            (N tokens, token-major)
    Pt[L][K]  = the paper's Pᵀ
    Wf[M][L]  = the paper's (PᵀW)ᵀ        (folded weight)
    Z[N][L]   = the paper's (PᵀX)ᵀ        (projected activations)
    Y[N][M]   = the paper's Yᵀ
Every function below converts its arguments to the paper's orientation,
evaluates the paper's expression, and converts the result back.
"""
import numpy as np


def _f64(a):
    return np.asarray(a, dtype=np.float64)


# -- the inference path (Section 2.2, Eq. 3) ---------------------------------

def fold(W, Pt):
    """Folded weight, stored as Wf[M][L]: the paper's PᵀW (L×M), transposed.
    Section 2.2 (inference view: PᵀW is pre-computed before deployment)."""
    Wp = _f64(W).T            # K×M
    P = _f64(Pt).T            # K×L
    PtW = P.T @ Wp            # L×M
    return np.ascontiguousarray(PtW.T)


def project(Pt, X):
    """Projected activations, stored as Z[N][L]: the paper's PᵀX (L×N),
    transposed.  Section 2.2, Eq. 3 (right factor); Eq. 6 gives its entries as
    the inner products <p_i, x>."""
    Xp = _f64(X).T            # K×N
    P = _f64(Pt).T            # K×L
    PtX = P.T @ Xp            # L×N
    return np.ascontiguousarray(PtX.T)


def expand(Z, Wf):
    """Y[N][M] from the projected activations and the folded weight: the
    paper's (PᵀW)ᵀ(PᵀX), transposed.  Section 2.2, Eq. 3."""
    PtX = _f64(Z).T           # L×N
    PtW = _f64(Wf).T          # L×M
    Yp = PtW.T @ PtX          # M×N
    return np.ascontiguousarray(Yp.T)


def projected_linear(X, Pt, Wf):
    """One call of the layer given its folded weight: expand(project(X))."""
    return expand(project(Pt, X), Wf)


def projected_linear_from_weights(X, Pt, W):
    """The method's result for weight W: (PᵀW)ᵀ(PᵀX), Eq. 3, folding included."""
    return expand(project(Pt, X), fold(W, Pt))


def dense(X, W):
    """The layer without projection, Y = WᵀX (Section 2.1, Eq. 1), as Y[N][M]."""
    Wp = _f64(W).T            # K×M
    Xp = _f64(X).T            # K×N
    return np.ascontiguousarray((Wp.T @ Xp).T)


def reconstruct(Pt, X):
    """X̃ = PPᵀX written as Eq. 6: x̃ = Σ_i <p_i, x> p_i for each token x,
    returned token-major [N][K]."""
    P = _f64(Pt).T            # K×L
    Xp = _f64(X).T            # K×N
    Xt = np.zeros_like(Xp)
    for i in range(P.shape[1]):
        p = P[:, i]
        Xt += np.outer(p, p @ Xp)
    return np.ascontiguousarray(Xt.T)


def rel_fro(a, ref):
    """Relative Frobenius error ||a - ref||_F / ||ref||_F in float64."""
    a = _f64(a)
    ref = _f64(ref)
    den = np.linalg.norm(ref)
    num = np.linalg.norm(a - ref)
    return float(num / den) if den > 0 else float(num)


# -- outputs at sampled positions (for layers too large to evaluate whole) ---

def sampled_projected_linear(X, Pt, W, rows, cols):
    """Y[rows][:, cols] of (PᵀW)ᵀ(PᵀX), computing only what those outputs need:
    the folded-weight rows of the selected output features and the projections
    of the selected tokens."""
    rows = np.asarray(rows)
    cols = np.asarray(cols)
    Wf_sel = fold(_f64(W)[cols], Pt)          # [|cols|][L]
    Z_sel = project(Pt, _f64(X)[rows])        # [|rows|][L]
    return expand(Z_sel, Wf_sel)              # [|rows|][|cols|]


def sampled_dense(X, W, rows, cols):
    return dense(_f64(X)[np.asarray(rows)], _f64(W)[np.asarray(cols)])


# -- calibration (Section 3.1, Eq. 5; Theorem 1; Corollary 1) -----------------

def autocorrelation(batches):
    """C_X averaged over calibration batches, Eq. 5: for each batch X_i (tokens
    as rows here, K-vectors x), C_i = (Σ x xᵀ)/M_i, and C_X = (Σ_i C_i)/B."""
    C = None
    for Xi in batches:
        Xp = _f64(Xi).T                       # K×M_i, tokens as columns
        Ci = (Xp @ Xp.T) / Xp.shape[1]
        C = Ci if C is None else C + Ci
    return C / len(batches)


def normalized_autocorrelation(batches):
    """Ĉ_X of Corollary 1: the autocorrelation of L2-normalised tokens."""
    normed = []
    for Xi in batches:
        Xi = _f64(Xi)
        normed.append(Xi / np.linalg.norm(Xi, axis=1, keepdims=True))
    return autocorrelation(normed)


def principal_components(C, L):
    """Theorem 1: P is the L principal eigenvectors of C (eigenvalues sorted in
    decreasing order).  Returns (Pt[L][K], all eigenvalues descending)."""
    d, V = np.linalg.eigh(_f64(C))
    order = np.argsort(d)[::-1]
    return np.ascontiguousarray(V[:, order[:L]].T), d[order]


# -- GO-MSE candidates (Section 3.3: Proposition 1, Theorem 2) -------------------

def gomse_matrix(CX, CW):
    """Theorem 2, GO-MSE bound: C = E[x xᵀ w wᵀ + w wᵀ x xᵀ].  For weights and
    activations drawn independently the expectation factors into
    C_X·C_W + C_W·C_X (proof of Theorem 2, Appendix), with C_X the activation
    autocorrelation and C_W = E[w wᵀ] the weight autocorrelation (rows of the
    stored W as the vectors w).  With the L2-normalised autocorrelations of
    both it is the normalised variant Ĉ of the same section."""
    CX = _f64(CX)
    CW = _f64(CW)
    return CX @ CW + CW @ CX


def principal_components_by_magnitude(C, L):
    """Theorem 2's selection for a C that need not be positive semi-definite:
    the L eigenvectors whose eigenvalues are largest in absolute value (proof
    of Theorem 2, Appendix); equal magnitudes: the positive eigenvalue first.
    Returns (Pt[L][K], all eigenvalues in that order)."""
    d, V = np.linalg.eigh(_f64(C))
    order = np.lexsort((-d, -np.abs(d)))
    return np.ascontiguousarray(V[:, order[:L]].T), d[order]


# -- training view (Section 2.2, "during training/finetuning") -----------------

def train_forward(X, Pt, W):
    """The training view of the layer: W acts on the reconstructed activations,
    Y = Wᵀ(PPᵀX) (Section 2.2, Eq. 3 read left to right), with P static and W
    trainable.  Returns Y[N][M] and X̃[N][K] = (PPᵀX)ᵀ."""
    Xt = reconstruct(Pt, X)
    return Xt @ _f64(W).T, Xt


def train_backward(dY, X, Pt, W):
    """Gradients of the training view for an upstream gradient dY[N][M] = ∂ℓ/∂Y:
    with X̃ = PPᵀX (P fixed), ∂ℓ/∂W = dYᵀ·X̃ (paper orientation: X̃·dYᵀ) and
    ∂ℓ/∂X = PPᵀ·(W·dY) (PPᵀ is symmetric).  Returns (dX[N][K], dW[M][K])."""
    dY = _f64(dY)
    W = _f64(W)
    Xt = reconstruct(Pt, X)
    dW = dY.T @ Xt
    dX = reconstruct(Pt, dY @ W)
    return dX, dW


def dense_backward(dY, X, W):
    """Gradients of the dense layer Y = WᵀX (Section 2.1, Eq. 1) for an
    upstream gradient dY[N][M]: ∂ℓ/∂X = dY·W, ∂ℓ/∂W = dYᵀ·X (storage
    orientation).  Returns (dX[N][K], dW[M][K])."""
    dY = _f64(dY)
    return dY @ _f64(W), dY.T @ _f64(X)


def nlmse_matrix(pairs, normalized=False):
    """Theorem 2, NL-MSE bound: C = E[x xᵀ ∇ ∇ᵀ + ∇ ∇ᵀ x xᵀ] with ∇ the loss
    gradient with respect to the activation vector, calibrated as the proof of
    Theorem 2 describes (Appendix): per sequence i, with its activations X^(i)
    and gradients G^(i) (M_i vectors each, as rows here),
    C^(i) = (X Xᵀ G Gᵀ + G Gᵀ X Xᵀ)/M_i², averaged over the B sequences.
    normalized: the L2-normalised variant Ĉ, each activation and each gradient
    vector scaled to unit norm (Section 3.3)."""
    C = None
    for X, G in pairs:
        X = _f64(X)
        G = _f64(G)
        if normalized:
            X = X / np.linalg.norm(X, axis=1, keepdims=True)
            G = G / np.linalg.norm(G, axis=1, keepdims=True)
        M = X.shape[0]
        Xp, Gp = X.T, G.T                          # K×M: vectors as columns
        Ci = (Xp @ Xp.T @ Gp @ Gp.T + Gp @ Gp.T @ Xp @ Xp.T) / (M * M)
        C = Ci if C is None else C + Ci
    return C / len(pairs)
