"""Training view of the layer (Section 2.2): gradients on the GPU against the
fp64 oracle, through the C ABI.

The GPU pass is the one a training step runs: Wf = fold(W, P) and Z =
project(P, X) from the forward pass, then the backward entry point.  The
oracle differentiates Y = W·(P·Pᵀ·X) directly from X, P, W and dY (it never
sees the GPU's Wf or Z).  Tolerances: relative Frobenius error 1e-2 (bf16;
Wf, Z and the two intermediate products are rounded to bf16) and 1e-5 (f32).
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import dev_mat, host64, need_gpu, out_mat, padding

pytestmark = pytest.mark.gpu

TOL = {"bf16": 1e-2, "f32": 1e-5}


@pytest.fixture(scope="module")
def E():
    need_gpu()
    import paper_2410_05437_amd as e
    return e


def _case(K, M, L, N, dtype, seed):
    w = synth.Workload(cfg=-1, name="train", K=K, M=M, L=L, N=N, dtype=dtype, recipe="gaussian",
                       lam_floor=1e-4, proj="leading", cov_key=6000 + seed, w_key=7000 + seed)
    inp = synth.make_inputs(w)
    dY64 = synth.upstream_gradient(N, M, 8000 + seed)
    if dtype == "bf16":
        bits = synth.bf16_bits_from_f64(dY64)
        dY = synth.f64_from_bf16_bits(bits).reshape(N, M)
        dYs = bits.reshape(N, M)
    else:
        dYs = dY64.astype(np.float32)
        dY = dYs.astype(np.float64)
    return inp, dY, dYs


SHAPES = [
    (256, 256, 64, 128),
    (1000, 600, 136, 300),
    (1003, 517, 131, 301),
    (520, 390, 72, 33),
    (640, 1100, 200, 8),
    (64, 100, 64, 1),
]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "K%d_M%d_L%d_N%d" % s)
def test_projected_linear_backward(E, shape, dtype):
    dev = need_gpu()
    K, M, L, N = shape
    inp, dY, dYs = _case(K, M, L, N, dtype, seed=K + N)
    X, Pt, W = (dev_mat(a, dtype, dev) for a in (inp.X_s, inp.Pt_s, inp.W_s))
    dYd = dev_mat(dYs, dtype, dev)
    Wf = E.espace_fold_weights(W, Pt)
    Z = E.espace_project(Pt, X)
    dX, dW = E.espace_projected_linear_backward(dYd, Z, Pt, Wf, dX=out_mat(N, K, dtype, dev),
                                                dW=out_mat(M, K, dtype, dev))
    dX1, _ = E.espace_projected_linear_backward(dYd, Z, Pt, Wf, want_dw=False)
    _, dW1 = E.espace_projected_linear_backward(dYd, Z, Pt, Wf, want_dx=False)
    torch.cuda.synchronize()
    dX_ref, dW_ref = oracle.train_backward(dY, inp.X, inp.Pt, inp.W)
    assert oracle.rel_fro(host64(dX), dX_ref) <= TOL[dtype]
    assert oracle.rel_fro(host64(dW), dW_ref) <= TOL[dtype]
    assert torch.equal(dX, dX1) and torch.equal(dW, dW1)
    assert np.isnan(padding(dX)).all() and np.isnan(padding(dW)).all()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("shape", SHAPES[:4], ids=lambda s: "K%d_M%d_L%d_N%d" % s)
def test_dense_linear_backward(E, shape, dtype):
    dev = need_gpu()
    K, M, L, N = shape
    inp, dY, dYs = _case(K, M, L, N, dtype, seed=K + N + 1)
    X, W = dev_mat(inp.X_s, dtype, dev), dev_mat(inp.W_s, dtype, dev)
    dX, dW = E.espace_dense_linear_backward(dev_mat(dYs, dtype, dev), X, W, dX=out_mat(N, K, dtype, dev),
                                            dW=out_mat(M, K, dtype, dev))
    torch.cuda.synchronize()
    dX_ref, dW_ref = oracle.dense_backward(dY, inp.X, inp.W)
    assert oracle.rel_fro(host64(dX), dX_ref) <= TOL[dtype]
    assert oracle.rel_fro(host64(dW), dW_ref) <= TOL[dtype]
    assert np.isnan(padding(dX)).all() and np.isnan(padding(dW)).all()


def test_full_rank_training_gradients_equal_dense(E):
    """L = K with an orthonormal P (a Hadamard matrix: PPᵀ = I exactly in
    binary floating point) makes the training view the dense layer."""
    dev = need_gpu()
    K, M, N = 256, 300, 200
    H = np.array([[1.0]])
    while H.shape[0] < K:
        H = np.block([[H, H], [H, -H]])
    Pt64 = H / np.sqrt(K)                      # 1/16: exact in bf16
    inp, dY, dYs = _case(K, M, 8, N, "bf16", seed=9)
    X, W = dev_mat(inp.X_s, "bf16", dev), dev_mat(inp.W_s, "bf16", dev)
    Pt = dev_mat(synth.bf16_bits_from_f64(Pt64).reshape(K, K), "bf16", dev)
    dYd = dev_mat(dYs, "bf16", dev)
    dX, dW = E.espace_projected_linear_backward(dYd, E.espace_project(Pt, X), Pt, E.espace_fold_weights(W, Pt))
    torch.cuda.synchronize()
    dX_ref, dW_ref = oracle.dense_backward(dY, inp.X, inp.W)
    assert oracle.rel_fro(host64(dX), dX_ref) <= TOL["bf16"]
    assert oracle.rel_fro(host64(dW), dW_ref) <= TOL["bf16"]


def test_llama2_7b_qkv_backward_sampled(E):
    """The Llama2-7B QKV shape (K=4096, M=12288, L=1536, N=4096): sampled rows
    of dX and dW against the oracle, which computes just those rows."""
    dev = need_gpu()
    w = synth.workload(1)
    inp = synth.make_inputs(w)
    K, M, L, N = w.K, w.M, w.L, w.N
    dY64 = synth.upstream_gradient(N, M, 8101)
    bits = synth.bf16_bits_from_f64(dY64)
    dY = synth.f64_from_bf16_bits(bits).reshape(N, M)
    X, Pt, W = (dev_mat(a, "bf16", dev) for a in (inp.X_s, inp.Pt_s, inp.W_s))
    dX, dW = E.espace_projected_linear_backward(dev_mat(bits.reshape(N, M), "bf16", dev),
                                                E.espace_project(Pt, X), Pt, E.espace_fold_weights(W, Pt))
    torch.cuda.synchronize()
    rng = np.random.default_rng(11)
    rn = np.unique(np.concatenate([rng.choice(N, 12, replace=False), [0, N - 1]]))
    rm = np.unique(np.concatenate([rng.choice(M, 12, replace=False), [0, M - 1]]))
    Pt64 = inp.Pt
    # dX rows: P·Pᵀ·(Wᵀ dy_n) for the sampled tokens
    dX_ref = oracle.reconstruct(Pt64, dY[rn] @ inp.W)
    # dW rows: dY[:, m]ᵀ X̃ = (dY[:, m]ᵀ Z) Pt with Z = X·Ptᵀ
    Zr = inp.X @ Pt64.T
    dW_ref = (dY[:, rm].T @ Zr) @ Pt64
    gx = dX[torch.as_tensor(rn, device=dev)].double().cpu().numpy()
    gw = dW[torch.as_tensor(rm, device=dev)].double().cpu().numpy()
    assert oracle.rel_fro(gx, dX_ref) <= TOL["bf16"]
    assert oracle.rel_fro(gw, dW_ref) <= TOL["bf16"]
