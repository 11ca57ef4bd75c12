"""The seeded input generators: encoding, reproducibility, distributions."""
import numpy as np
import pytest
import torch

import oracle
import synth
from synth import generate as G


def test_bf16_rne_matches_torch_on_float32_values():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(100000).astype(np.float32).astype(np.float64) * 3.0
    ours = synth.bf16_bits_from_f64(x)
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy()
    assert np.array_equal(ours.view(np.int16), ref)


def test_bf16_ties_to_even_and_zero():
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties to even -> 1.0
    # 1 + 3*2^-8 is halfway between 1 + 2^-7 and 1 + 2^-6: ties to even -> 1 + 2^-6
    x = np.array([1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, 0.0, -0.0, -1.5, 1 + 2.0 ** -8 + 2.0 ** -40])
    back = synth.f64_from_bf16_bits(synth.bf16_bits_from_f64(x))
    assert back[0] == 1.0
    assert back[1] == 1 + 2.0 ** -6
    assert back[2] == 0.0 and back[3] == 0.0 and np.signbit(back[3])
    assert back[4] == -1.5
    assert back[5] == 1 + 2.0 ** -7   # just above the tie rounds up


def test_haar_is_orthogonal_and_sign_corrected():
    Q = G.haar_orthogonal(200, G.rng_for(99, 0))
    assert np.abs(Q.T @ Q - np.eye(200)).max() < 1e-12
    # Haar measure: E[Q_11] = 0; the sign correction removes LAPACK's bias
    vals = [G.haar_orthogonal(3, np.random.default_rng(s))[0, 0] for s in range(3000)]
    assert abs(np.mean(vals)) < 0.04


def test_seeds_reproduce_and_prefix_property():
    w = synth.workload(0).scaled(N=64)
    a = G._make(w)
    b = G._make(w)
    assert np.array_equal(a.X_s, b.X_s) and np.array_equal(a.W_s, b.W_s)
    w8 = w.scaled(N=8)
    c = G._make(w8)
    assert np.array_equal(c.X_s, a.X_s[:8])


def test_tail_energy_matches_spectrum():
    """tokens ~ N(0, Q diag(lam) Qᵀ) and P = Q[:, :L]: the relative energy outside
    span(P) is Σ_{i>L} lam_i / Σ lam_i (0.2254 for K=256, L=64, lam_i = 1/i)."""
    w = synth.workload(0).scaled(N=16384)
    inp = G._make(w)
    X, Pt = inp.X, inp.Pt
    resid = X - (X @ Pt.T) @ Pt
    frac = np.sum(resid ** 2) / np.sum(X ** 2)
    lam = G.spectrum(w.K, w.lam_floor)
    expect = lam[w.L:].sum() / lam.sum()
    assert abs(expect - 0.2254) < 1e-3
    assert abs(frac - expect) / expect < 0.05


def test_calibrated_projection_matches_theorem1():
    """The silu-gated workload's calibrated P spans the same subspace as the
    oracle's Theorem 1 construction on the same calibration tokens."""
    K, L, n = 96, 24, 4096
    Q = G.haar_orthogonal(K, G.rng_for(7, 0))
    lam = G.spectrum(K)
    Xc = G.silu_gated_tokens(Q, lam, n, G.rng_for(7, 6), G.rng_for(7, 7))
    Pt, d = G.principal_subspace(Xc, L)
    Po, do = oracle.principal_components(oracle.autocorrelation([Xc]), L)
    assert d[L - 1] - d[L] > 0
    assert np.abs(Pt.T @ Pt - Po.T @ Po).max() < 1e-8
    assert np.allclose(d, do, rtol=1e-10, atol=1e-14)


def test_workload_table():
    assert len(synth.workloads(2)) == 4
    assert len(synth.workloads(4)) == 18
    w = synth.workload(1)
    assert (w.K, w.M, w.L, w.N) == (4096, 12288, 1536, 4096)
    assert abs(w.compression - 0.5) < 1e-12
    assert abs(synth.workload(4, layer="down", L=2458, N=8192).compression - 0.5) < 1e-3
