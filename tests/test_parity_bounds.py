"""The element-wise parity criteria (tests/parity.py) on the CPU: a float32
emulation of the GPU's arithmetic (bfloat16 operands, exact products, fp32
accumulation, round-to-nearest-even to bfloat16 after each product) stays
inside the derived bounds on several shapes and input distributions, and each
of a set of planted kernel-style mistakes in that emulation is caught."""
import numpy as np
import pytest

import oracle
import synth
from tests import parity


def _rb(a):
    """Round float64 values to bfloat16 (round to nearest even), as float64."""
    a = np.asarray(a, dtype=np.float64)
    return synth.f64_from_bf16_bits(synth.bf16_bits_from_f64(a)).reshape(a.shape)


def _gemm32(A, B):
    """A·Bᵀ with float32 accumulation of exact products."""
    return (A.astype(np.float32) @ B.astype(np.float32).T).astype(np.float64)


def _inputs(K, M, L, N, seed, recipe="gaussian"):
    w = synth.Workload(cfg=-1, name="bounds", K=K, M=M, L=L, N=N, dtype="bf16", recipe=recipe,
                       lam_floor=1e-4, proj="leading", cov_key=3000 + seed, w_key=4000 + seed)
    return synth.make_inputs(w)


def _emulated_layer(inp):
    Wf = _rb(_gemm32(inp.W, inp.Pt))
    Z = _rb(_gemm32(inp.X, inp.Pt))
    return _rb(_gemm32(Z, Wf)), Z, Wf


def _reference(inp):
    Z64 = oracle.project(inp.Pt, inp.X)
    Wf64 = oracle.fold(inp.W, inp.Pt)
    Y64 = oracle.expand(Z64, Wf64)
    K, L = inp.w.K, inp.w.L
    xn, pn, wn = parity.row_norms(inp.X), parity.row_norms(inp.Pt), parity.row_norms(inp.W)
    B = parity.layer_bound(Y64, Z64, Wf64, xn, pn, wn, K, L, parity.U_BF16)
    return Y64, B


SHAPES = [(512, 384, 96, 130), (1000, 700, 136, 65), (256, 300, 256, 7), (2048, 256, 64, 200)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "K%d_M%d_L%d_N%d" % s)
def test_emulation_within_bounds(shape):
    inp = _inputs(*shape, seed=shape[0] % 97)
    Y, Z, Wf = _emulated_layer(inp)
    Y64, B = _reference(inp)
    rel, blk, ratio = parity.check(Y, Y64, B, parity.TOL["bf16"], "emulated layer")
    assert rel < 5e-3 and ratio < 1.0
    # the single products against their own bounds
    u = parity.U_BF16
    K = inp.w.K
    Z64 = oracle.project(inp.Pt, inp.X)
    parity.check(Z, Z64, parity.product_bound(Z64, parity.row_norms(inp.X), parity.row_norms(inp.Pt), K, u),
                 parity.TOL["bf16"], "emulated projection")
    Wf64 = oracle.fold(inp.W, inp.Pt)
    parity.check(Wf, Wf64, parity.product_bound(Wf64, parity.row_norms(inp.W), parity.row_norms(inp.Pt), K, u),
                 parity.TOL["bf16"], "emulated fold")


def test_silu_gated_tokens_within_bounds():
    w = synth.Workload(cfg=-1, name="bounds", K=768, M=256, L=96, N=160, dtype="bf16", recipe="silu_gated",
                       lam_floor=0.0, proj="leading", cov_key=3900, w_key=3901)
    inp = synth.make_inputs(w)
    Y, _, _ = _emulated_layer(inp)
    Y64, B = _reference(inp)
    parity.check(Y, Y64, B, parity.TOL["bf16"], "emulated layer, SiLU-gated tokens")


def _planted(name, Y, Z, Wf, inp):
    Y = Y.copy()
    L = inp.w.L
    if name == "unwritten tile":
        Y[64:128, 64:128] = np.nan
    elif name == "one depth half of a tile lost":
        h = L // 2
        Y[64:128, 0:64] = _rb(_gemm32(Z[64:128, :h], Wf[0:64, :h]))
    elif name == "row index off by one in a tile":
        Y[0:64, 64:128] = Y[1:65, 64:128]
    elif name == "column index off by one in a tile":
        Y[64:128, 64:128] = Y[64:128, 65:129]
    elif name == "tile written transposed":
        Y[0:64, 0:64] = Y[0:64, 0:64].T.copy()
    elif name == "partial sums added twice":
        Y[0:64, 128:192] = _rb(2 * _gemm32(Z[0:64], Wf[128:192]))
    elif name == "last feature not written":
        Y[:, -1] = 0.0
    elif name == "one token's projection zero":
        Zb = Z.copy()
        Zb[5] = 0.0
        Y = _rb(_gemm32(Zb, Wf))
    elif name == "projection depth tail dropped":
        K = inp.w.K
        Zb = _rb(_gemm32(inp.X[:, :K - 64], inp.Pt[:, :K - 64]))
        Y = _rb(_gemm32(Zb, Wf))
    else:
        raise KeyError(name)
    return Y


PLANTED = ["unwritten tile", "one depth half of a tile lost", "row index off by one in a tile",
           "column index off by one in a tile", "tile written transposed", "partial sums added twice",
           "last feature not written", "one token's projection zero", "projection depth tail dropped"]


@pytest.mark.parametrize("name", PLANTED)
def test_planted_mistakes_are_caught(name):
    inp = _inputs(512, 384, 96, 130, seed=11)
    Y, Z, Wf = _emulated_layer(inp)
    Y64, B = _reference(inp)
    bad = _planted(name, Y, Z, Wf, inp)
    with pytest.raises(AssertionError):
        parity.check(bad, Y64, B, parity.TOL["bf16"], name)
    # a global norm alone would miss a lost depth half at a realistic size:
    # one 64 x 64 tile of a 4096 x 12288 output moves it by
    # sqrt(0.5 · 4096 / 5.0e7) ≈ 0.0064, under 1e-2


def test_float32_bounds_are_tight_enough():
    """For float32 storage the bound holds for a float32 emulation and is not
    vacuous: about 1e-3 of the largest output (a worst case of the depth-K
    accumulation of the inputs, K·2^-23 relative), while the Frobenius
    criterion keeps the whole output within 1e-5."""
    w = synth.Workload(cfg=-1, name="bounds", K=256, M=256, L=64, N=128, dtype="f32", recipe="gaussian",
                       lam_floor=0.0, proj="leading", cov_key=3950, w_key=3951)
    inp = synth.make_inputs(w)
    Wf = _gemm32(inp.W, inp.Pt).astype(np.float32).astype(np.float64)
    Z = _gemm32(inp.X, inp.Pt).astype(np.float32).astype(np.float64)
    Y = _gemm32(Z, Wf)
    Z64 = oracle.project(inp.Pt, inp.X)
    Wf64 = oracle.fold(inp.W, inp.Pt)
    Y64 = oracle.expand(Z64, Wf64)
    B = parity.layer_bound(Y64, Z64, Wf64, parity.row_norms(inp.X), parity.row_norms(inp.Pt),
                           parity.row_norms(inp.W), 256, 64, parity.U_F32)
    parity.check(Y, Y64, B, parity.TOL["f32"], "float32 emulation")
    assert float(np.median(B / np.abs(Y64).max())) < 2e-3
