"""The allocation-free projected linear call (static device scratch) against
the call with a workspace, through the C ABI: two calls in a row on one
device, the second with smaller sizes, each bitwise equal to the workspace
call and within the parity criteria against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests import parity
from tests.gpu_util import dev_mat, host64, need_gpu, out_mat

pytestmark = pytest.mark.gpu


def _case(E, dev, K, M, L, N, seed):
    w = synth.Workload(cfg=-1, name="noalloc", K=K, M=M, L=L, N=N, dtype="bf16", recipe="gaussian",
                       lam_floor=1e-4, proj="leading", cov_key=5000 + seed, w_key=6000 + seed)
    inp = synth.make_inputs(w)
    X = dev_mat(inp.X_s, "bf16", dev)
    Pt = dev_mat(inp.Pt_s, "bf16", dev)
    W = dev_mat(inp.W_s, "bf16", dev)
    Wf = E.espace_fold_weights(W, Pt)
    return inp, X, Pt, Wf


def test_noalloc_matches_workspace_call():
    dev = need_gpu()
    import paper_2410_05437_amd as E
    # a prefill layer whose Z sits in the scratch in row pairs (an odd token
    # count, components not a multiple of 64), then smaller ones: tiled GEMMs,
    # a pair-combined projection, then a decode call
    cases = [(4096, 6000, 1500, 4095, 4), (2048, 3000, 512, 1500, 1), (1100, 600, 700, 1000, 2),
             (1003, 1500, 200, 16, 3)]
    for K, M, L, N, seed in cases:
        inp, X, Pt, Wf = _case(E, dev, K, M, L, N, seed)
        Y_na = E.espace_projected_linear_noalloc(X, Pt, Wf, out_mat(N, M, "bf16", dev))
        torch.cuda.synchronize()
        Y_ws = E.espace_projected_linear(X, Pt, Wf, out_mat(N, M, "bf16", dev))
        torch.cuda.synchronize()
        assert torch.equal(Y_na, Y_ws), (K, M, L, N)
        Z64 = oracle.project(inp.Pt, inp.X)
        Wf64 = oracle.fold(inp.W, inp.Pt)
        Y64 = oracle.expand(Z64, Wf64)
        B = parity.layer_bound(Y64, Z64, Wf64, parity.row_norms(inp.X), parity.row_norms(inp.Pt),
                               parity.row_norms(inp.W), K, L, parity.U_BF16)
        parity.check(host64(Y_na), Y64, B, parity.TOL["bf16"], f"noalloc K={K} M={M} L={L} N={N}")


def test_noalloc_rejects_oversized_call_on_gpu():
    dev = need_gpu()
    import paper_2410_05437_amd as E
    N, K, L, M = 1 << 16, 4096, 1536, 64
    X = torch.zeros(N, K, dtype=torch.bfloat16, device=dev)
    Pt = torch.zeros(L, K, dtype=torch.bfloat16, device=dev)
    Wf = torch.zeros(M, L, dtype=torch.bfloat16, device=dev)
    Y = torch.full((N, M), 7.0, dtype=torch.bfloat16, device=dev)
    with pytest.raises(E.EspaceError) as ei:
        E.espace_projected_linear_noalloc(X, Pt, Wf, Y)
    assert ei.value.status == 6
    torch.cuda.synchronize()
    assert bool((Y == 7.0).all())
