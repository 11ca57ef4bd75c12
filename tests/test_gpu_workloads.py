"""The GPU path on the full-size workloads, against the fp64 oracle.

Full outputs are compared where the oracle evaluates them in seconds; larger
layers compare sampled outputs, each computed by the oracle one by one."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import dev_mat, host64, need_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def E():
    need_gpu()
    import paper_2410_05437_amd as e
    return e


def _run(E, inp, dev):
    X = dev_mat(inp.X_s, inp.w.dtype, dev)
    Pt = dev_mat(inp.Pt_s, inp.w.dtype, dev)
    W = dev_mat(inp.W_s, inp.w.dtype, dev)
    Wf = E.espace_fold_weights(W, Pt)
    Y = E.espace_projected_linear(X, Pt, Wf)
    Yd = E.espace_dense_linear(X, W)
    torch.cuda.synchronize()
    return Y, Yd


def test_llama2_7b_qkv_full(E):
    """Llama2-7B fused QKV (K=4096, M=12288, L=1536, N=4096), the benchmark's
    launch configuration, every output against the oracle."""
    dev = need_gpu()
    inp = synth.make_inputs(synth.workload(1))
    Y, Yd = _run(E, inp, dev)
    Y64 = oracle.projected_linear_from_weights(inp.X, inp.Pt, inp.W)
    err = oracle.rel_fro(host64(Y), Y64)
    print(f"llama2-7b qkv: rel_fro {err:.3e}")
    assert err <= 1e-2
    rng = np.random.default_rng(0)
    rows = rng.choice(inp.w.N, 64, replace=False)
    cols = rng.choice(inp.w.M, 64, replace=False)
    Yd_s = host64(Yd)[np.ix_(rows, cols)]
    assert oracle.rel_fro(Yd_s, oracle.sampled_dense(inp.X, inp.W, rows, cols)) <= 1e-2


@pytest.mark.parametrize("N", [1, 8, 16, 4096])
def test_llama2_7b_ffn_upgate(E, N):
    dev = need_gpu()
    inp = synth.make_inputs(synth.workload(2, N=N))
    Y, Yd = _run(E, inp, dev)
    if N <= 16:
        Y64 = oracle.projected_linear_from_weights(inp.X, inp.Pt, inp.W)
        assert oracle.rel_fro(host64(Y), Y64) <= 1e-2
        assert oracle.rel_fro(host64(Yd), oracle.dense(inp.X, inp.W)) <= 1e-2
    else:
        rng = np.random.default_rng(1)
        rows = rng.choice(N, 96, replace=False)
        cols = rng.choice(inp.w.M, 96, replace=False)
        ref = oracle.sampled_projected_linear(inp.X, inp.Pt, inp.W, rows, cols)
        assert oracle.rel_fro(host64(Y)[np.ix_(rows, cols)], ref) <= 1e-2


def _sampled(E, inp, dev, n_rows=96, n_cols=192, seed=2):
    """GPU projected linear and dense outputs at sampled (token, feature)
    positions, each against the oracle computed for exactly those positions;
    the last token and the last feature (ragged tiles) are always included."""
    w = inp.w
    Y, Yd = _run(E, inp, dev)
    rng = np.random.default_rng(seed)
    rows = np.arange(w.N) if w.N <= n_rows else rng.choice(w.N, n_rows, replace=False)
    cols = rng.choice(w.M, n_cols, replace=False)
    rows = np.unique(np.append(rows, w.N - 1))
    cols = np.unique(np.append(cols, w.M - 1))
    ri = torch.as_tensor(rows, device=dev)
    ci = torch.as_tensor(cols, device=dev)
    err = oracle.rel_fro(host64(Y[ri][:, ci]), oracle.sampled_projected_linear(inp.X, inp.Pt, inp.W, rows, cols))
    errd = oracle.rel_fro(host64(Yd[ri][:, ci]), oracle.sampled_dense(inp.X, inp.W, rows, cols))
    print(f"{w.name} K={w.K} M={w.M} L={w.L} N={w.N}: rel_fro {err:.3e} (dense {errd:.3e})")
    assert err <= 1e-2
    assert errd <= 1e-2


def test_llama2_7b_ffn_down_full(E):
    """Llama2-7B FFN down (K=11008, M=4096, L=1536, N=4096): SiLU-gated tokens,
    P calibrated on 16384 separate tokens."""
    dev = need_gpu()
    _sampled(E, synth.make_inputs(synth.workload(3)), dev)


@pytest.mark.parametrize("w", synth.workloads(4), ids=lambda w: f"{w.layer}_L{w.L}_N{w.N}")
def test_gpt3_22b_ffn_full(E, w):
    """GPT3-22B FFN up (K=6144, M=24576) and down (K=24576, M=6144), the
    compression sweep L in {3686, 2458, 1966}, N in {8192, 1, 16}."""
    dev = need_gpu()
    _sampled(E, synth.make_inputs(w), dev)
