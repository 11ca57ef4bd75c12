"""GPU path vs the fp64 CPU oracle, through the C ABI.

Tolerances (relative Frobenius error of the GPU output against the oracle's
float64 result on the same rounded inputs): 1e-2 for bfloat16 storage, 1e-5
for float32.  Parity is against the method's result (W·P)(Pᵀ·X), never W·X.
Inputs carry NaN in their row padding, so any read of padding values would
poison the result.
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


def _inputs(K, M, L, N, dtype, seed=0, recipe="gaussian"):
    w = synth.Workload(cfg=-1, name="test", K=K, M=M, L=L, N=N, dtype=dtype, recipe=recipe,
                       lam_floor=1e-4, proj="leading", cov_key=1000 + seed, w_key=2000 + seed)
    return synth.make_inputs(w)


def _dev_inputs(inp, dev):
    dt = inp.w.dtype
    return (dev_mat(inp.X_s, dt, dev), dev_mat(inp.Pt_s, dt, dev), dev_mat(inp.W_s, dt, dev))


# (K, M, L, N): several tiles plus ragged tails in every dimension; N <= 32
# takes the decode path, N > 32 the tiled path
SHAPES = [
    (256, 256, 64, 128),
    (1000, 600, 136, 300),
    (1003, 517, 131, 301),
    (640, 1100, 200, 64),
    (520, 390, 72, 33),
    (1024, 2000, 256, 1),
    (1000, 777, 131, 5),
    (1003, 1500, 200, 16),
    (768, 1000, 96, 17),
    (2048, 3000, 320, 32),
]


# degenerate sizes: depth 1 (every step a masked tail), one output feature,
# one token, L = K, a single partial tile
DEGENERATE = [
    (1, 1, 1, 1),
    (1, 7, 1, 40),
    (8, 3, 8, 33),
    (64, 1, 1, 100),
    (7, 100, 3, 1),
    (32, 40, 32, 64),
]


# bfloat16 decode plans at N <= 8 (the sizes of the Llama2-7B projection and
# beyond): whole-row streaming for one and two tokens (tokens in LDS: depth
# 4500, nine 512-element passes, a full block of eight and a partial one, and
# depth 3000, six passes with a partial last; tokens in registers: depths
# 1003, 1536, 131 and 136), two depth segments per MFMA operand with 16 waves (the
# projection at 8 tokens, 9 row groups over 141 steps) and with 8 waves (its
# expansion, 57 row groups over 5 steps); one depth range of 132 steps for 132
# row groups (3 and 5 tokens).
DECODE_PLANS = [
    (4500, 900, 136, 8),
    (4500, 900, 136, 1),
    (4500, 700, 1536, 2),
    (4500, 2100, 4200, 3),
    (4500, 2100, 4200, 5),
    (1003, 517, 131, 2),
    (3000, 700, 136, 1),
]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("shape", SHAPES + DEGENERATE, ids=lambda s: "K%d_M%d_L%d_N%d" % s)
def test_each_entry_point(E, dtype, shape):
    _check_entry_points(E, dtype, shape)


@pytest.mark.parametrize("shape", DECODE_PLANS, ids=lambda s: "K%d_M%d_L%d_N%d" % s)
def test_decode_plans(E, shape):
    _check_entry_points(E, "bf16", shape, seed=45)


def _check_entry_points(E, dtype, shape, seed=0):
    dev = need_gpu()
    K, M, L, N = shape
    inp = _inputs(K, M, L, N, dtype, seed=seed)
    X, Pt, W = _dev_inputs(inp, dev)
    tol = TOL[dtype]

    Wf64 = oracle.fold(inp.W, inp.Pt)
    Z64 = oracle.project(inp.Pt, inp.X)
    Y64 = oracle.projected_linear_from_weights(inp.X, inp.Pt, inp.W)
    Yd64 = oracle.dense(inp.X, inp.W)

    Wf = E.espace_fold_weights(W, Pt, out_mat(M, L, dtype, dev))
    Z = E.espace_project(Pt, X, out_mat(N, L, dtype, dev))
    Y = E.espace_projected_linear(X, Pt, Wf, out_mat(N, M, dtype, dev))
    Ye = E.espace_expand(Z, Wf, out_mat(N, M, dtype, dev))
    Yd = E.espace_dense_linear(X, W, out_mat(N, M, dtype, dev))
    torch.cuda.synchronize()

    assert oracle.rel_fro(host64(Wf), Wf64) <= tol
    assert oracle.rel_fro(host64(Z), Z64) <= tol
    assert oracle.rel_fro(host64(Y), Y64) <= tol
    assert oracle.rel_fro(host64(Ye), Y64) <= tol
    assert oracle.rel_fro(host64(Yd), Yd64) <= tol
    # the fused call computes exactly what project followed by expand computes
    assert torch.equal(Y, Ye)
    # outputs keep their padding untouched (prefilled with NaN)
    for t in (Wf, Z, Y, Yd):
        assert np.isnan(padding(t)).all()


def test_projected_linear_given_oracle_folded_weight(E):
    """The per-call path alone, with the folded weight rounded from the
    oracle's float64 fold (an input, not a result of the GPU)."""
    dev = need_gpu()
    K, M, L, N = 1000, 900, 136, 257
    inp = _inputs(K, M, L, N, "bf16", seed=3)
    X, Pt, _ = _dev_inputs(inp, dev)
    Wf_bits = synth.bf16_bits_from_f64(oracle.fold(inp.W, inp.Pt))
    Wf_exact = synth.f64_from_bf16_bits(Wf_bits).reshape(M, L)
    Wf = dev_mat(Wf_bits, "bf16", dev)
    Y = E.espace_projected_linear(X, Pt, Wf)
    torch.cuda.synchronize()
    assert oracle.rel_fro(host64(Y), oracle.projected_linear(inp.X, inp.Pt, Wf_exact)) <= 1e-2


@pytest.mark.parametrize("N", [1, 16, 200])
def test_selection_matrix_is_bitwise(E, N):
    """P with distinct signed unit columns: the folded weight is exactly ±W[:, J]
    and the projection exactly ±X[:, J] (one nonzero product per sum)."""
    dev = need_gpu()
    rng = np.random.default_rng(5)
    K, M, L = 1000, 700, 136
    J = rng.permutation(K)[:L]
    s = rng.choice([-1.0, 1.0], size=L)
    Pt = np.zeros((L, K))
    Pt[np.arange(L), J] = s
    inp = _inputs(K, M, L, N, "bf16", seed=4)
    Xd = dev_mat(inp.X_s, "bf16", dev)
    Wd = dev_mat(inp.W_s, "bf16", dev)
    Pd = dev_mat(synth.bf16_bits_from_f64(Pt), "bf16", dev)
    Wf = E.espace_fold_weights(Wd, Pd)
    Z = E.espace_project(Pd, Xd)
    torch.cuda.synchronize()
    assert np.array_equal(host64(Wf), inp.W[:, J] * s[None, :])
    assert np.array_equal(host64(Z), inp.X[:, J] * s[None, :])


def _hadamard(K):
    H = np.array([[1.0]])
    while H.shape[0] < K:
        H = np.block([[H, H], [H, -H]])
    return H / np.sqrt(K)


@pytest.mark.parametrize("N", [4, 300])
def test_full_rank_hadamard_equals_dense(E, N):
    """L = K with an orthonormal P exactly representable in bf16 (Hadamard/16):
    PPᵀ = I, so the layer reproduces W·X within the bf16 tolerance."""
    dev = need_gpu()
    K, M = 256, 640
    inp = _inputs(K, M, 8, N, "bf16", seed=6)
    H = _hadamard(K)
    Pd = dev_mat(synth.bf16_bits_from_f64(H.T.copy()), "bf16", dev)
    Xd = dev_mat(inp.X_s, "bf16", dev)
    Wd = dev_mat(inp.W_s, "bf16", dev)
    Y = E.espace_projected_linear(Xd, Pd, E.espace_fold_weights(Wd, Pd))
    torch.cuda.synchronize()
    assert oracle.rel_fro(host64(Y), oracle.dense(inp.X, inp.W)) <= 1e-2


def test_exact_rank_tokens_reproduce_dense(E):
    """Tokens of exact rank <= L projected on the top-L eigenvectors of their
    autocorrelation: PPᵀX = X (Theorem 1), so the layer reproduces W·X."""
    dev = need_gpu()
    rng = np.random.default_rng(8)
    K, M, r, L, N = 512, 384, 40, 64, 200
    B = np.linalg.qr(rng.standard_normal((K, r)))[0]
    X = rng.standard_normal((N, r)) @ B.T
    Pt, _ = oracle.principal_components(oracle.autocorrelation([X]), L)
    W = rng.standard_normal((M, K)) / np.sqrt(K)
    Xd = dev_mat(X.astype(np.float32), "f32", dev)
    Pd = dev_mat(Pt.astype(np.float32), "f32", dev)
    Wd = dev_mat(W.astype(np.float32), "f32", dev)
    Y = E.espace_projected_linear(Xd, Pd, E.espace_fold_weights(Wd, Pd))
    torch.cuda.synchronize()
    assert oracle.rel_fro(host64(Y), oracle.dense(X, W)) <= 1e-5


def test_tiny_fp32_workload(E):
    """Workload 0 (K=M=256, L=64, N=128, float32) end to end."""
    dev = need_gpu()
    w = synth.workload(0)
    inp = synth.make_inputs(w)
    X, Pt, W = _dev_inputs(inp, dev)
    Y = E.espace_projected_linear(X, Pt, E.espace_fold_weights(W, Pt))
    torch.cuda.synchronize()
    Y64 = oracle.projected_linear_from_weights(inp.X, inp.Pt, inp.W)
    assert oracle.rel_fro(host64(Y), Y64) <= 1e-5
    # information: the projection error against the dense layer is large by design
    assert oracle.rel_fro(Y64, oracle.dense(inp.X, inp.W)) > 0.1


def test_determinism(E):
    dev = need_gpu()
    for shape in [(1003, 1500, 200, 16), (1000, 600, 136, 300)]:
        inp = _inputs(*shape, "bf16", seed=9)
        X, Pt, W = _dev_inputs(inp, dev)
        Wf = E.espace_fold_weights(W, Pt)
        ref = E.espace_projected_linear(X, Pt, Wf).clone()
        for _ in range(20):
            assert torch.equal(E.espace_projected_linear(X, Pt, Wf), ref)


def test_empty_sizes_are_no_ops(E):
    dev = need_gpu()
    inp = _inputs(256, 128, 32, 8, "bf16", seed=10)
    X, Pt, W = _dev_inputs(inp, dev)
    Wf = E.espace_fold_weights(W, Pt)
    Y0 = E.espace_projected_linear(X[:0], Pt, Wf)
    assert Y0.shape == (0, 128)
    Yd0 = E.espace_dense_linear(X[:0], W)
    assert Yd0.shape == (0, 128)
    Ym0 = E.espace_projected_linear(X, Pt, Wf[:0])
    assert Ym0.shape == (8, 0)


def test_invalid_arguments_write_nothing(E):
    dev = need_gpu()
    inp = _inputs(256, 128, 32, 8, "bf16", seed=11)
    X, Pt, W = _dev_inputs(inp, dev)
    Wf = E.espace_fold_weights(W, Pt)
    Y = out_mat(8, 128, "bf16", dev, fill=7.0)
    # L > K
    with pytest.raises(E.EspaceError) as ei:
        E.espace_projected_linear(X, dev_mat(np.zeros((300, 256), np.uint16), "bf16", dev),
                                  Wf, Y)
    assert ei.value.status in (2,)
    # output aliasing an input
    with pytest.raises(E.EspaceError) as ei:
        E.espace_dense_linear(X, W, W[:8, :128])
    assert ei.value.status == 5
    # misaligned base pointer (a view starting one element in)
    big = torch.zeros(9 * 256, dtype=torch.bfloat16, device=dev)
    Xm = big[1:1 + 8 * 256].view(8, 256)
    with pytest.raises(E.EspaceError) as ei:
        E.espace_dense_linear(Xm, W, Y)
    assert ei.value.status == 3
    torch.cuda.synchronize()
    assert (host64(Y) == 7.0).all()


DECODE_SHAPES = [s for s in SHAPES if s[3] <= 32] + [(4096, 3000, 1536, 16), (11008, 700, 1536, 3)]


@pytest.mark.parametrize("shape", DECODE_SHAPES, ids=lambda s: "K%d_M%d_L%d_N%d" % s)
def test_one_launch_decode_path(E, shape, monkeypatch):
    """The one-launch decode path (selected with ESPACE_DECODE=fused) against
    the oracle, over ragged shapes, one and two token groups and depth splits."""
    dev = need_gpu()
    monkeypatch.setenv("ESPACE_DECODE", "fused")
    K, M, L, N = shape
    inp = _inputs(K, M, L, N, "bf16", seed=30)
    X, Pt, W = _dev_inputs(inp, dev)
    Wf = E.espace_fold_weights(W, Pt)
    Y = E.espace_projected_linear(X, Pt, Wf, out_mat(N, M, "bf16", dev))
    torch.cuda.synchronize()
    Y64 = oracle.projected_linear_from_weights(inp.X, inp.Pt, inp.W)
    assert oracle.rel_fro(host64(Y), Y64) <= TOL["bf16"]


def test_decode_workspace_contents_do_not_matter(E, monkeypatch):
    """The one-launch decode path keeps its counters in the workspace, which
    need no initialisation: leftover bytes (zeros, all ones, random, another
    shape's counter state) give the same, bitwise identical output."""
    dev = need_gpu()
    monkeypatch.setenv("ESPACE_DECODE", "fused")
    shapes = [(1003, 1500, 200, 16), (768, 1000, 96, 17), (1024, 2000, 256, 1), (4096, 3000, 1536, 8)]
    cases = []
    for i, (K, M, L, N) in enumerate(shapes):
        inp = _inputs(K, M, L, N, "bf16", seed=20 + i)
        X, Pt, W = _dev_inputs(inp, dev)
        Wf = E.espace_fold_weights(W, Pt)
        ref = E.espace_projected_linear(X, Pt, Wf).clone()
        torch.cuda.synchronize()
        Y64 = oracle.projected_linear_from_weights(inp.X, inp.Pt, inp.W)
        assert oracle.rel_fro(host64(ref), Y64) <= TOL["bf16"]
        cases.append((X, Pt, Wf, ref))
    need = max(E.espace_workspace_bytes(E.OP_PROJECTED_LINEAR, Wf.shape[0], X.shape[1], Pt.shape[0],
                                        X.shape[0], torch.bfloat16) for X, Pt, Wf, _ in cases)
    ws = torch.empty(need, dtype=torch.uint8, device=dev)
    gen = torch.Generator(device="cpu").manual_seed(5)
    fills = ["zeros", "ones", "random", "keep", "keep"]
    for fill in fills:
        for X, Pt, Wf, ref in cases + cases[::-1]:
            if fill == "zeros":
                ws.zero_()
            elif fill == "ones":
                ws.fill_(255)
            elif fill == "random":
                ws.copy_(torch.randint(0, 256, (need,), dtype=torch.uint8, generator=gen))
            Y = E.espace_projected_linear(X, Pt, Wf, workspace=ws)
            assert torch.equal(Y, ref), fill


def test_matrices_past_2g_elements(E):
    """A weight of 524296 x 4096 bf16 (more than 2^31 elements, 4 GiB) takes the
    kernel with 64-bit row offsets; sampled outputs, including the last rows,
    against the oracle."""
    dev = need_gpu()
    M, K, N = (1 << 19) + 8, 4096, 48
    assert M * K >= 1 << 31
    W = torch.empty((M, K), dtype=torch.bfloat16, device=dev)
    kk = torch.arange(K, device=dev, dtype=torch.int32)[None, :]
    for r0 in range(0, M, 1 << 16):
        r1 = min(M, r0 + (1 << 16))
        mm = torch.arange(r0, r1, device=dev, dtype=torch.int32)[:, None]
        W[r0:r1] = synth.index_pattern(mm, kk).to(torch.float32).to(torch.bfloat16)
    inp = _inputs(K, 64, 32, N, "bf16", seed=40)
    X = dev_mat(inp.X_s, "bf16", dev)
    Y = E.espace_dense_linear(X, W)
    torch.cuda.synchronize()
    rng = np.random.default_rng(3)
    cols = np.unique(np.concatenate([rng.choice(M, 200, replace=False), np.arange(M - 40, M)]))
    W_sel = synth.index_pattern(cols[:, None].astype(np.int64), np.arange(K)[None, :])
    ref = oracle.dense(inp.X, W_sel)
    got = host64(Y[:, torch.as_tensor(cols, device=dev)])
    assert oracle.rel_fro(got, ref) <= TOL["bf16"]
    del W


# (K, M, L, N) whose projection (N x L, depth K) the tile planner runs as two
# depth halves combined inside the GEMM kernel: on the 128x192 and 256x128
# tiles, and on the four-wave 256x192 tile (also the Llama2-7B FFN-down
# workload's plan), there with ragged rows, a column count that is not a
# multiple of 8 and a depth tail
PAIR_SHAPES = [(1100, 600, 700, 1000), (4100, 500, 1100, 2500), (3003, 520, 1300, 2500),
               (4100, 300, 1536, 3000), (4100, 300, 1100, 4096)]


@pytest.mark.parametrize("shape", PAIR_SHAPES, ids=lambda s: "K%d_M%d_L%d_N%d" % s)
def test_pair_combined_depth_halves(E, shape):
    """Projection with the in-kernel pair combine against the oracle; the
    combine is order-independent, so repeated calls are bitwise identical
    whatever the workspace held before (its state words are tagged per call)."""
    dev = need_gpu()
    K, M, L, N = shape
    inp = _inputs(K, M, L, N, "bf16", seed=50)
    X, Pt, W = _dev_inputs(inp, dev)
    Z = E.espace_project(Pt, X, out_mat(N, L, "bf16", dev))
    torch.cuda.synchronize()
    assert oracle.rel_fro(host64(Z), oracle.project(inp.Pt, inp.X)) <= TOL["bf16"]
    assert np.isnan(padding(Z)).all()
    need = E.espace_workspace_bytes(E.OP_PROJECT, 0, K, L, N, torch.bfloat16)
    ws = torch.empty(need, dtype=torch.uint8, device=dev)
    gen = torch.Generator(device="cpu").manual_seed(6)
    for fill in ["zeros", "ones", "random", "keep", "keep"]:
        if fill == "zeros":
            ws.zero_()
        elif fill == "ones":
            ws.fill_(255)
        elif fill == "random":
            ws.copy_(torch.randint(0, 256, (need,), dtype=torch.uint8, generator=gen))
        assert torch.equal(E.espace_project(Pt, X, workspace=ws), Z), fill


@pytest.mark.parametrize("shape", [PAIR_SHAPES[0], PAIR_SHAPES[4]], ids=lambda s: "K%d_M%d_L%d_N%d" % s)
def test_pair_combine_under_graph_replay(E, shape):
    """A captured projection that uses the pair combine replays correctly: each
    replay, with new inputs copied in between and eager work in between,
    matches the eager call bitwise."""
    dev = need_gpu()
    K, M, L, N = shape
    inps = [_inputs(K, M, L, N, "bf16", seed=60 + i) for i in range(3)]
    X, Pt, _ = _dev_inputs(inps[0], dev)
    Z = out_mat(N, L, "bf16", dev)
    ws = torch.empty(E.espace_workspace_bytes(E.OP_PROJECT, 0, K, L, N, torch.bfloat16),
                     dtype=torch.uint8, device=dev)
    E.espace_project(Pt, X, Z, ws)          # warm-up outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        E.espace_project(Pt, X, Z, ws)
    torch.cuda.synchronize()
    for rep in range(6):
        Xi = dev_mat(inps[rep % 3].X_s, "bf16", dev)
        X.copy_(Xi)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = Z.clone()
        ref = E.espace_project(Pt, X)          # eager, its own workspace and call tag
        torch.cuda.synchronize()
        assert torch.equal(got, ref), rep
        if rep < 3:
            assert oracle.rel_fro(host64(got), oracle.project(inps[0].Pt, inps[rep].X)) <= TOL["bf16"]


def test_prefill_layer_under_graph_replay(E):
    """A prefill layer call (tiled GEMMs, Z in the workspace) captured once in
    a HIP graph and replayed with new inputs copied in between: every replay
    equals the eager call bitwise, and the oracle on the first input."""
    dev = need_gpu()
    K, M, L, N = 1024, 4096, 256, 2048
    inps = [_inputs(K, M, L, N, "bf16", seed=70 + i) for i in range(2)]
    X, Pt, W = _dev_inputs(inps[0], dev)
    Wf = E.espace_fold_weights(W, Pt)
    Y = out_mat(N, M, "bf16", dev)
    ws = torch.empty(max(E.espace_workspace_bytes(E.OP_PROJECTED_LINEAR, M, K, L, N, torch.bfloat16), 1),
                     dtype=torch.uint8, device=dev)
    E.espace_projected_linear(X, Pt, Wf, Y, ws)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        E.espace_projected_linear(X, Pt, Wf, Y, ws)
    torch.cuda.synchronize()
    for rep in range(4):
        X.copy_(dev_mat(inps[rep % 2].X_s, "bf16", dev))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = Y.clone()
        ref = E.espace_projected_linear(X, Pt, Wf)
        torch.cuda.synchronize()
        assert torch.equal(got, ref), rep
    X.copy_(dev_mat(inps[0].X_s, "bf16", dev))
    g.replay()
    torch.cuda.synchronize()
    assert oracle.rel_fro(host64(Y), oracle.projected_linear_from_weights(inps[0].X, inps[0].Pt, inps[0].W)) <= 1e-2
