"""Calibration of P on the GPU (Section 3.1, Eq. 5; Theorem 1; Corollary 1)
against the fp64 CPU oracle, through the C ABI.

Autocorrelation: compared element by element with a bound on the rounding
the GPU path performs, |C_gpu - C| <= tol_ij, where with S_ij = alpha·Σ_n
|x̂_ni·x̂_nj| (exact, from the oracle's inputs):
  * bf16 tokens: products of bf16 values are exact in fp32, and the fp32 sum
    of N terms plus the update of C err by at most (N + 4)·2^-24·S_ij (the
    usual γ_n bound of recursive summation, a few terms for the depth ranges,
    the alpha scaling and the final addition);
  * normalised tokens are scaled by 1/||x|| (fp32) and rounded to bf16, so
    each factor carries a relative error below 2^-8 + 2^-23: tol_ij adds
    2·(2^-8 + 2^-23)·S_ij;
  * f32 tokens: the products round too: (N + 6)·2^-24·S_ij (plus 2·2^-23
    when normalising).
Principal components: on matrices with a known, well-separated spectrum
(synth.symmetric_with_spectrum, rounded to float32 and given to both sides)
the eigenvalues match the oracle's fp64 decomposition of the same matrix to
fp32 rounding and the eigenvectors, after the documented sign convention,
match element by element.  At the Llama2-7B calibration size the checks are
properties that hold at any size: sampled autocorrelation entries within the
bound above, orthonormal rows of Pt, eigenvalues in decreasing order, and
Theorem 1's minimum-MSE identity.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import dev_mat, host64, need_gpu

pytestmark = pytest.mark.gpu

U32 = 2.0 ** -24


@pytest.fixture(scope="module")
def E():
    need_gpu()
    import paper_2410_05437_amd as e
    return e


def _tokens(K, N, dtype, seed, recipe="gaussian"):
    w = synth.Workload(cfg=-1, name="calib", K=K, M=8, L=1, N=N, dtype=dtype, recipe=recipe,
                       lam_floor=1e-4, proj="leading", cov_key=3000 + seed, w_key=4000 + seed)
    inp = synth.make_inputs(w)
    return inp.X, inp.X_s


def _bound(Xh, alpha, N, dtype, normalize):
    """tol_ij of the module docstring for tokens Xh (already normalised when
    `normalize`)."""
    A = np.abs(Xh)
    S = alpha * (A.T @ A)
    if dtype == "bf16":
        rel = (N + 4) * U32 + (2 * (2.0 ** -8 + 2.0 ** -23) if normalize else 0.0)
    else:
        rel = (N + 6) * U32 + (2 * 2.0 ** -23 if normalize else 0.0)
    return rel * S + 1e-30


def _normalised(X):
    n = np.linalg.norm(X, axis=1, keepdims=True)
    return np.where(n > 0, X / np.where(n > 0, n, 1.0), 0.0)


def _gpu_autocorr(E, Xs, dtype, dev, C0, alpha, normalize):
    C = torch.from_numpy(np.ascontiguousarray(C0, dtype=np.float32)).to(dev)
    Cp = torch.full((C.shape[0], (C.shape[0] + 3) // 4 * 4), float("nan"), dtype=torch.float32, device=dev)
    Cv = Cp[:, :C.shape[0]]
    Cv.copy_(C)
    E.espace_autocorrelation_update(dev_mat(Xs, dtype, dev), Cv, alpha, normalize=normalize)
    torch.cuda.synchronize()
    pad = Cp[:, C.shape[0]:].cpu().numpy()
    assert np.isnan(pad).all(), "padding of C written"
    return host64(Cv)


AC_SHAPES = [(64, 100), (300, 1000), (517, 333), (1000, 2048), (256, 1), (130, 4000)]


@pytest.mark.parametrize("normalize", [False, True], ids=["C_X", "C_hat"])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("shape", AC_SHAPES, ids=lambda s: "K%d_N%d" % s)
def test_autocorrelation_update(E, shape, dtype, normalize):
    dev = need_gpu()
    K, N = shape
    X, Xs = _tokens(K, N, dtype, seed=K + N)
    got = _gpu_autocorr(E, Xs, dtype, dev, np.zeros((K, K)), 1.0 / N, normalize)
    ref = (oracle.normalized_autocorrelation if normalize else oracle.autocorrelation)([X])
    tol = _bound(_normalised(X) if normalize else X, 1.0 / N, N, dtype, normalize)
    err = np.abs(got - ref)
    assert (err <= tol).all(), float((err / tol).max())


def test_batches_accumulate_to_the_batch_average(E):
    """Eq. 5: C_X is the average of the per-batch estimates; two updates with
    alpha = 1/(N_i·B), on top of an existing C, add exactly that."""
    dev = need_gpu()
    K = 200
    X1, X1s = _tokens(K, 700, "bf16", seed=11)
    X2, X2s = _tokens(K, 300, "bf16", seed=12)
    C0 = synth.symmetric_with_spectrum(K, np.linspace(1.0, 0.1, K), 5).astype(np.float32).astype(np.float64)
    C = torch.from_numpy(C0.astype(np.float32)).to(dev)
    E.espace_autocorrelation_update(dev_mat(X1s, "bf16", dev), C, 1.0 / (700 * 2))
    E.espace_autocorrelation_update(dev_mat(X2s, "bf16", dev), C, 1.0 / (300 * 2))
    torch.cuda.synchronize()
    got = host64(C)
    ref = C0 + oracle.autocorrelation([X1, X2])
    tol = _bound(X1, 1.0 / 1400, 700, "bf16", False) + _bound(X2, 1.0 / 600, 300, "bf16", False) \
        + 4 * U32 * np.abs(ref)
    assert (np.abs(got - ref) <= tol).all()


def test_zero_token_contributes_nothing_when_normalised(E):
    dev = need_gpu()
    K, N = 96, 500
    X, Xs = _tokens(K, N, "bf16", seed=21)
    Xs = Xs.copy()
    Xs[7] = 0
    X = X.copy()
    X[7] = 0
    got = _gpu_autocorr(E, Xs, "bf16", dev, np.zeros((K, K)), 1.0 / N, True)
    keep = np.r_[0:7, 8:N]
    ref = oracle.normalized_autocorrelation([X[keep]]) * (N - 1) / N
    tol = _bound(_normalised(X), 1.0 / N, N, "bf16", True)
    assert (np.abs(got - ref) <= tol).all()


def _sign_fixed(Pt):
    """The documented convention: each row's entry of largest magnitude
    (the first such) is positive."""
    idx = np.argmax(np.abs(Pt), axis=1)
    s = np.sign(Pt[np.arange(Pt.shape[0]), idx])
    s[s == 0] = 1
    return Pt * s[:, None]


def _gapped_spectrum(K, L):
    lam = np.empty(K)
    lam[:L] = 1.0 / (1.0 + np.arange(L))            # distinct leading eigenvalues
    lam[L:] = 1e-3 / (1.0 + np.arange(K - L))       # far below them
    return lam


PCA_CASES = [(64, 16), (300, 1), (300, 300), (1000, 100), (517, 200)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", PCA_CASES, ids=lambda c: "K%d_L%d" % c)
def test_principal_components(E, case, dtype):
    dev = need_gpu()
    K, L = case
    C32 = synth.symmetric_with_spectrum(K, _gapped_spectrum(K, L), 100 + K + L).astype(np.float32)
    C = dev_mat(C32, "f32", dev)          # NaN in the padding columns
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    Pt, ev, info = E.espace_principal_components(C, L, dtype=tdt)
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    Pt_ref, d_ref = oracle.principal_components(C32.astype(np.float64), L)
    Pt_ref = _sign_fixed(Pt_ref)
    got_ev = ev.cpu().numpy().astype(np.float64)
    assert np.all(np.diff(got_ev) <= 0)
    assert np.allclose(got_ev, d_ref, rtol=2 * U32, atol=1e-12 * abs(d_ref).max())
    got = host64(Pt)
    if dtype == "f32":
        assert np.abs(got - Pt_ref).max() <= 1e-6
        assert np.abs(got @ got.T - np.eye(L)).max() <= 1e-5
    else:
        assert (np.abs(got - Pt_ref) <= 2.0 ** -8 * np.abs(Pt_ref) + 1e-9).all()


def test_principal_components_degenerate_spectrum(E):
    """Degenerate spectrum (C = I): every orthonormal set is optimal, so the
    check is what holds for any choice: Pt Ptᵀ = I and all eigenvalues 1."""
    dev = need_gpu()
    K, L = 40, 10
    C = torch.eye(K, dtype=torch.float32, device=dev)
    Pt, ev, info = E.espace_principal_components(C, L, dtype=torch.float32)
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    got = host64(Pt)
    assert np.abs(got @ got.T - np.eye(L)).max() <= 1e-6
    assert np.allclose(ev.cpu().numpy(), 1.0, atol=1e-6)


@pytest.mark.parametrize("normalize", [False, True], ids=["Thm1_MSE", "Cor1_NMSE"])
def test_calibrated_projection_attains_the_minimum(E, normalize):
    """Theorem 1 / Corollary 1 end to end: C (or Ĉ) from the GPU's update, P
    from the GPU's decomposition; the oracle measures the (normalised) MSE of
    that P on the calibration tokens, which must equal the sum of the
    discarded eigenvalues of the oracle's own autocorrelation (the minimum)
    up to the effect of the GPU's rounding of C."""
    dev = need_gpu()
    K, N, L = 512, 3000, 128
    X, Xs = _tokens(K, N, "bf16", seed=31)
    C = torch.zeros(K, K, dtype=torch.float32, device=dev)
    E.espace_autocorrelation_update(dev_mat(Xs, "bf16", dev), C, 1.0 / N, normalize=normalize)
    Pt, ev, info = E.espace_principal_components(C, L, dtype=torch.float32)
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    P = host64(Pt)
    Xr = _normalised(X) if normalize else X
    resid = Xr - oracle.reconstruct(P, Xr)
    mse = float((resid ** 2).sum(axis=1).mean())
    Cref = (oracle.normalized_autocorrelation if normalize else oracle.autocorrelation)([X])
    _, d = oracle.principal_components(Cref, L)
    tail = float(d[L:].sum())
    assert mse >= tail * (1 - 1e-6)
    assert mse <= tail * (1 + 1e-4)


def test_llama2_7b_calibration_size(E):
    """K = 4096 (Llama2-7B hidden size), 16384 calibration tokens, L = 1536:
    sampled autocorrelation entries within the rounding bound; orthonormal
    principal components with decreasing eigenvalues; each sampled eigenpair
    satisfies the eigen-equation of the matrix it was computed from."""
    dev = need_gpu()
    K, N, L = 4096, 16384, 1536
    X, Xs = _tokens(K, N, "bf16", seed=41)
    Xd = dev_mat(Xs, "bf16", dev)
    C = torch.zeros(K, K, dtype=torch.float32, device=dev)
    E.espace_autocorrelation_update(Xd, C, 1.0 / N)
    torch.cuda.synchronize()
    rng = np.random.default_rng(5)
    rows = np.unique(np.concatenate([rng.choice(K, 48, replace=False), [0, K - 1]]))
    cols = np.unique(np.concatenate([rng.choice(K, 48, replace=False), [0, K - 1]]))
    Ch = C[torch.as_tensor(rows, device=dev)][:, torch.as_tensor(cols, device=dev)].double().cpu().numpy()
    ref = (X[:, rows].T @ X[:, cols]) / N
    tol = (N + 4) * U32 * (np.abs(X[:, rows]).T @ np.abs(X[:, cols])) / N
    assert (np.abs(Ch - ref) <= tol).all()
    Pt, ev, info = E.espace_principal_components(C, L, dtype=torch.float32)
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    P = host64(Pt)
    assert np.abs(P @ P.T - np.eye(L)).max() <= 1e-5
    e = ev.cpu().numpy().astype(np.float64)
    assert np.all(np.diff(e) <= 0) and e[-1] > -1e-6
    C64 = host64(C)
    for l in [0, 1, 10, 100, 1000, L - 1]:
        r = C64 @ P[l] - e[l] * P[l]
        assert np.linalg.norm(r) <= 1e-5 * e[0], (l, float(np.linalg.norm(r)))


# ---- GO-MSE candidates (Theorem 2) ------------------------------------------

SYM_SIZES = [64, 300, 517, 1000]


@pytest.mark.parametrize("K", SYM_SIZES)
def test_symmetrized_product(E, K):
    """C = A·Bᵀ + B·Aᵀ on symmetric A, B (float32 inputs given to both sides)
    against the oracle's C_X·C_W + C_W·C_X, entry by entry within the fp32
    rounding bound (K + 1)·2^-24·(S_ij + S_ji) + 2^-24·|C_ij|, S = |A|·|B|ᵀ
    (the product's K fused multiply-adds, then one addition); the result is
    exactly symmetric."""
    dev = need_gpu()
    A32 = synth.symmetric_with_spectrum(K, np.linspace(2.0, 0.01, K), 200 + K).astype(np.float32)
    B32 = synth.symmetric_with_spectrum(K, 1.0 / (1.0 + np.arange(K)), 300 + K).astype(np.float32)
    C = E.espace_symmetrized_product(dev_mat(A32, "f32", dev), dev_mat(B32, "f32", dev))
    torch.cuda.synchronize()
    got = host64(C)
    A, B = A32.astype(np.float64), B32.astype(np.float64)
    ref = oracle.gomse_matrix(A, B)
    S = np.abs(A) @ np.abs(B).T
    tol = (K + 1) * U32 * (S + S.T) + U32 * np.abs(ref)
    assert (np.abs(got - ref) <= tol).all()
    assert (got == got.T).all()


def _mixed_spectrum(K, L):
    lam = np.empty(K)
    i = np.arange(L)
    lam[:L] = (1.0 / (1.0 + i)) * np.where(i % 3 == 1, -1.0, 1.0)     # distinct magnitudes, mixed signs
    lam[L:] = 1e-3 / (1.0 + np.arange(K - L)) * np.where(np.arange(K - L) % 2, -1.0, 1.0)
    return lam


@pytest.mark.parametrize("case", [(64, 16), (300, 40), (517, 100)], ids=lambda c: "K%d_L%d" % c)
def test_principal_components_by_magnitude(E, case):
    dev = need_gpu()
    K, L = case
    C32 = synth.symmetric_with_spectrum(K, _mixed_spectrum(K, L), 400 + K).astype(np.float32)
    Pt, ev, info = E.espace_principal_components(dev_mat(C32, "f32", dev), L, dtype=torch.float32,
                                                 by_magnitude=True)
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    Pt_ref, d_ref = oracle.principal_components_by_magnitude(C32.astype(np.float64), L)
    got_ev = ev.cpu().numpy().astype(np.float64)
    assert np.allclose(got_ev[:L], d_ref[:L], rtol=2 * U32, atol=1e-12)
    assert np.all(np.diff(np.abs(got_ev[:L])) <= 0)
    assert np.abs(host64(Pt) - _sign_fixed(Pt_ref)).max() <= 1e-6


@pytest.mark.parametrize("normalize", [False, True], ids=["GO-MSE", "GO-MSE_hat"])
def test_gomse_projection_end_to_end(E, normalize):
    """Theorem 2 end to end on the GPU: C_X from the tokens, C_W from the rows
    of W, C = C_X·C_W + C_W·C_X, P its L components of largest |eigenvalue|.
    The oracle evaluates the part of Proposition 1's bound that P controls,
    Σ_i p_iᵀ C p_i with its own C, for that P and for its own selection."""
    dev = need_gpu()
    K, M, N, L = 256, 512, 2000, 48
    w = synth.Workload(cfg=-1, name="gomse", K=K, M=M, L=1, N=N, dtype="bf16", recipe="gaussian",
                       lam_floor=1e-4, proj="leading", cov_key=5001, w_key=5002)
    inp = synth.make_inputs(w)
    CX = torch.zeros(K, K, dtype=torch.float32, device=dev)
    CW = torch.zeros(K, K, dtype=torch.float32, device=dev)
    E.espace_autocorrelation_update(dev_mat(inp.X_s, "bf16", dev), CX, 1.0 / N, normalize=normalize)
    E.espace_autocorrelation_update(dev_mat(inp.W_s, "bf16", dev), CW, 1.0 / M, normalize=normalize)
    C = E.espace_symmetrized_product(CX, CW)
    Pt, ev, info = E.espace_principal_components(C, L, dtype=torch.float32, by_magnitude=True)
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    ac = oracle.normalized_autocorrelation if normalize else oracle.autocorrelation
    Cref = oracle.gomse_matrix(ac([inp.X]), ac([inp.W]))
    Pref, _ = oracle.principal_components_by_magnitude(Cref, L)
    P = host64(Pt)
    q = float(np.einsum("lk,kj,lj->", P, Cref, P))
    qref = float(np.einsum("lk,kj,lj->", Pref, Cref, Pref))
    assert abs(q - qref) <= 1e-4 * abs(qref), (q, qref)


@pytest.mark.parametrize("normalize", [False, True], ids=["NL-MSE", "NL-MSE_hat"])
def test_nlmse_matrix_over_sequences(E, normalize):
    """Theorem 2's NL-MSE matrix, calibrated per sequence as its proof
    describes: for each of three sequences the autocorrelations of the
    activations and of their gradients (alpha = 1/M_i), then accumulated with
    alpha = 1/B, beta = 1.  Against the oracle: relative Frobenius error below
    (N + K)·2^-24 ≈ 1e-4 (fp32 sums of the exact bf16 products, then an fp32
    K-term product), or 2·2^-8 when the normalised vectors are rounded to
    bf16."""
    dev = need_gpu()
    K = 200
    seqs = []
    for i, M in enumerate((300, 500, 250)):
        X, Xs = _tokens(K, M, "bf16", seed=60 + i)
        g = synth.upstream_gradient(M, K, 9000 + i)
        bits = synth.bf16_bits_from_f64(g)
        seqs.append((X, Xs, synth.f64_from_bf16_bits(bits).reshape(M, K), bits.reshape(M, K)))
    C = torch.zeros(K, K, dtype=torch.float32, device=dev)
    for i, (X, Xs, G, Gs) in enumerate(seqs):
        M = X.shape[0]
        A = torch.zeros(K, K, dtype=torch.float32, device=dev)
        B = torch.zeros(K, K, dtype=torch.float32, device=dev)
        E.espace_autocorrelation_update(dev_mat(Xs, "bf16", dev), A, 1.0 / M, normalize=normalize)
        E.espace_autocorrelation_update(dev_mat(Gs, "bf16", dev), B, 1.0 / M, normalize=normalize)
        E.espace_symmetrized_product(A, B, C, alpha=1.0 / len(seqs), beta=0.0 if i == 0 else 1.0)
    torch.cuda.synchronize()
    ref = oracle.nlmse_matrix([(X, G) for X, _, G, _ in seqs], normalized=normalize)
    tol = 2 * 2.0 ** -8 if normalize else (1000 + K) * U32
    assert oracle.rel_fro(host64(C), ref) <= tol
    got = host64(C)
    assert (got == got.T).all()
