"""GPU path vs the fp64 CPU oracle, through the C ABI.

Every output is compared whole, entry by entry, with the criteria of
tests/parity.py: finite everywhere (outputs are NaN-prefilled), each entry
within the rounding bound derived from the GPU's arithmetic, and a relative
Frobenius error of at most 1e-2 (bfloat16) or 1e-5 (float32) over the whole
output and over every 64 x 64 block.  Parity is against the method's result
(W·P)(Pᵀ·X), never W·X.  Inputs carry NaN in their row padding, so any read
of padding values would poison the result.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests import parity
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
# row groups (3 and 5 tokens); two depth segments with two token groups of
# eight (9 to 16 tokens: 12 tokens on the 141-step projection with 16 waves,
# 16 tokens on a 125-step projection and its 10-step expansion with 8 waves,
# 9 tokens, the second group holding one, over 32 and 5 steps).
DECODE_PLANS = [
    (4500, 900, 136, 8),
    (4500, 900, 136, 12),
    (4000, 700, 300, 16),
    (1003, 517, 131, 9),
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


# 3 to 16 tokens on weights of at least 16 rows per CU (the persistent
# streaming kernel on the expansion and the dense product): a ragged last
# group of 16 rows (4100, 8200), workgroups taking two or more groups (8200
# rows), depths whose last 512-element piece holds 1, 131 and 188 elements
# (the piece straddling the depth masked in registers) and the deepest
# supported depth (6144, twelve pieces); workgroups with one group more than
# others (5000 and 22016 rows: 313 and 1376 groups over the CUs).
STREAM_PLANS = [
    (1600, 4100, 1537, 3),
    (6144, 4096, 131, 8),
    (700, 8200, 700, 16),
    (1000, 5000, 700, 5),
    (2000, 22016, 1536, 16),
]


@pytest.mark.parametrize("shape", STREAM_PLANS, ids=lambda s: "K%d_M%d_L%d_N%d" % s)
def test_stream_plans(E, shape):
    _check_entry_points(E, "bf16", shape, seed=47)


def _check_entry_points(E, dtype, shape, seed=0):
    dev = need_gpu()
    K, M, L, N = shape
    inp = _inputs(K, M, L, N, dtype, seed=seed)
    X, Pt, W = _dev_inputs(inp, dev)
    tol = TOL[dtype]

    Wf64 = oracle.fold(inp.W, inp.Pt)
    Z64 = oracle.project(inp.Pt, inp.X)
    Y64 = oracle.expand(Z64, Wf64)
    Yd64 = oracle.dense(inp.X, inp.W)

    Wf = E.espace_fold_weights(W, Pt, out_mat(M, L, dtype, dev))
    Z = E.espace_project(Pt, X, out_mat(N, L, dtype, dev))
    Y = E.espace_projected_linear(X, Pt, Wf, out_mat(N, M, dtype, dev))
    Ye = E.espace_expand(Z, Wf, out_mat(N, M, dtype, dev))
    Yd = E.espace_dense_linear(X, W, out_mat(N, M, dtype, dev))
    torch.cuda.synchronize()

    u = parity.UNIT[dtype]
    xn, pn, wn = parity.row_norms(inp.X), parity.row_norms(inp.Pt), parity.row_norms(inp.W)
    parity.check(host64(Wf), Wf64, parity.product_bound(Wf64, wn, pn, K, u), tol, "fold")
    parity.check(host64(Z), Z64, parity.product_bound(Z64, xn, pn, K, u), tol, "project")
    By = parity.layer_bound(Y64, Z64, Wf64, xn, pn, wn, K, L, u)
    parity.check(host64(Y), Y64, By, tol, "projected linear")
    parity.check(host64(Ye), Y64, By, tol, "expand")
    parity.check(host64(Yd), Yd64, parity.product_bound(Yd64, xn, wn, K, u), tol, "dense")
    # the fused call computes exactly what project followed by expand computes
    assert torch.equal(Y, Ye)
    # outputs keep their padding untouched (prefilled with NaN)
    for t in (Wf, Z, Y, Yd):
        assert np.isnan(padding(t)).all()


# Products whose tiles would leave the last round of workgroups partly empty
# run as two launches split by rows: the fold of a 12288-row weight at depths
# 1560 (ragged steps) and 4096 (the Llama2-7B QKV fold: 4096 rows on 128 x 192
# tiles, then 8192 rows on 256 x 192 tiles), and a dense product of 6500
# tokens (a ragged second part).
ROW_SPLIT = [("fold", (1560, 12288, 1536, 64)), ("fold", (4096, 12288, 1536, 64)),
             ("dense", (1000, 3000, 64, 6500))]


@pytest.mark.parametrize("case", ROW_SPLIT, ids=lambda c: "%s_K%d_M%d_L%d_N%d" % ((c[0],) + c[1]))
def test_row_split_launches(E, case):
    dev = need_gpu()
    op, (K, M, L, N) = case
    inp = _inputs(K, M, L, N, "bf16", seed=61)
    X, Pt, W = _dev_inputs(inp, dev)
    u = parity.UNIT["bf16"]
    if op == "fold":
        got = E.espace_fold_weights(W, Pt, out_mat(M, L, "bf16", dev))
        want = oracle.fold(inp.W, inp.Pt)
        B = parity.product_bound(want, parity.row_norms(inp.W), parity.row_norms(inp.Pt), K, u)
    else:
        got = E.espace_dense_linear(X, W, out_mat(N, M, "bf16", dev))
        want = oracle.dense(inp.X, inp.W)
        B = parity.product_bound(want, parity.row_norms(inp.X), parity.row_norms(inp.W), K, u)
    torch.cuda.synchronize()
    parity.check(host64(got), want, B, TOL["bf16"], op)
    assert np.isnan(padding(got)).all()


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
    Y = E.espace_projected_linear(X, Pt, Wf, out_mat(N, M, "bf16", dev))
    torch.cuda.synchronize()
    Z64 = oracle.project(inp.Pt, inp.X)
    Y64 = oracle.expand(Z64, Wf_exact)
    B = parity.layer_bound(Y64, Z64, Wf_exact, parity.row_norms(inp.X), parity.row_norms(inp.Pt), None, K, L,
                           parity.U_BF16)
    parity.check(host64(Y), Y64, B, 1e-2, "projected linear, given folded weight")


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
    Y = E.espace_projected_linear(Xd, Pd, E.espace_fold_weights(Wd, Pd), out_mat(N, M, "bf16", dev))
    torch.cuda.synchronize()
    Hr = synth.f64_from_bf16_bits(synth.bf16_bits_from_f64(H.T.copy())).reshape(K, K)
    assert np.array_equal(Hr, H.T)
    Z64 = oracle.project(Hr, inp.X)
    Wf64 = oracle.fold(inp.W, Hr)
    Yd64 = oracle.dense(inp.X, inp.W)
    assert oracle.rel_fro(oracle.expand(Z64, Wf64), Yd64) < 1e-12
    B = parity.layer_bound(Yd64, Z64, Wf64, parity.row_norms(inp.X), parity.row_norms(Hr),
                           parity.row_norms(inp.W), K, K, parity.U_BF16)
    parity.check(host64(Y), Yd64, B, 1e-2, "full-rank Hadamard P against W·X")


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
    Y = E.espace_projected_linear(Xd, Pd, E.espace_fold_weights(Wd, Pd), out_mat(N, M, "f32", dev))
    torch.cuda.synchronize()
    assert oracle.rel_fro(host64(Y), oracle.dense(X, W)) <= 1e-5
    X32, P32, W32 = (a.astype(np.float32).astype(np.float64) for a in (X, Pt, W))
    Z64 = oracle.project(P32, X32)
    Wf64 = oracle.fold(W32, P32)
    Y64 = oracle.expand(Z64, Wf64)
    B = parity.layer_bound(Y64, Z64, Wf64, parity.row_norms(X32), parity.row_norms(P32), parity.row_norms(W32),
                           K, L, parity.U_F32)
    parity.check(host64(Y), Y64, B, 1e-5, "exact-rank tokens")


def test_tiny_fp32_workload(E):
    """Workload 0 (K=M=256, L=64, N=128, float32) end to end."""
    dev = need_gpu()
    w = synth.workload(0)
    inp = synth.make_inputs(w)
    X, Pt, W = _dev_inputs(inp, dev)
    Y = E.espace_projected_linear(X, Pt, E.espace_fold_weights(W, Pt), out_mat(w.N, w.M, "f32", dev))
    torch.cuda.synchronize()
    Z64 = oracle.project(inp.Pt, inp.X)
    Wf64 = oracle.fold(inp.W, inp.Pt)
    Y64 = oracle.expand(Z64, Wf64)
    B = parity.layer_bound(Y64, Z64, Wf64, parity.row_norms(inp.X), parity.row_norms(inp.Pt),
                           parity.row_norms(inp.W), w.K, w.L, parity.U_F32)
    rel, blk, ratio = parity.check(host64(Y), Y64, B, 1e-5, "tiny fp32 workload")
    print(f"tiny fp32: rel_fro {rel:.2e}, worst block {blk:.2e}, worst error/bound {ratio:.3f}")
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


def test_matrices_past_2g_elements(E):
    """A weight of 524296 x 4096 bf16 (more than 2^31 elements, 4 GiB) takes the
    kernel with 64-bit row offsets; every output against the oracle."""
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
    Y = E.espace_dense_linear(X, W, out_mat(N, M, "bf16", dev))
    torch.cuda.synchronize()
    del W
    Yh = host64(Y)
    # index_pattern(m, k) depends on m only through m mod 255 (73 m mod 255
    # has period 255), so the 255 distinct weight rows give every output
    period = np.arange(255)
    W255 = synth.index_pattern(period[:, None], np.arange(K)[None, :])
    ref255 = oracle.dense(inp.X, W255)
    B255 = parity.product_bound(ref255, parity.row_norms(inp.X), parity.row_norms(W255), K, parity.U_BF16)
    cols = np.arange(M) % 255
    parity.check(Yh, ref255[:, cols], B255[:, cols], TOL["bf16"], "dense with a weight of 2^31+ elements")
    del Y, Yh


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
    Z64 = oracle.project(inp.Pt, inp.X)
    B = parity.product_bound(Z64, parity.row_norms(inp.X), parity.row_norms(inp.Pt), K, parity.U_BF16)
    parity.check(host64(Z), Z64, B, TOL["bf16"], "pair-combined projection")
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


def _tiles_ok_or_nan(got, ref, bm, bn):
    """Every bm x bn output tile either equals the reference bitwise or is NaN
    throughout; returns the number of NaN tiles."""
    R, C = ref.shape
    nan_tiles = 0
    for r0 in range(0, R, bm):
        for c0 in range(0, C, bn):
            g = got[r0:r0 + bm, c0:c0 + bn]
            if np.isnan(g).all():
                nan_tiles += 1
            else:
                assert np.array_equal(g, ref[r0:r0 + bm, c0:c0 + bn]), (r0, c0)
    return nan_tiles


@pytest.mark.parametrize("shape", [PAIR_SHAPES[0], PAIR_SHAPES[3]], ids=lambda s: "K%d_M%d_L%d_N%d" % s)
def test_pair_wait_that_gives_up_writes_nan(E, shape):
    """The failure path of the bounded wait in the pair combine, forced from
    the host with a wait limit of one poll: a tile whose second half finds
    the first half's sums not yet stored gives up at once, writes NaN over the
    whole tile and is counted; every other tile is exact.  The default limit
    restores correct results."""
    dev = need_gpu()
    K, M, L, N = shape
    inp = _inputs(K, M, L, N, "bf16", seed=55)
    X, Pt, _ = _dev_inputs(inp, dev)
    ref = host64(E.espace_project(Pt, X))
    torch.cuda.synchronize()
    n0 = E.espace_wait_timeouts()
    nan_tiles = 0
    try:
        E.espace_set_wait_limit(1)
        for _ in range(4):
            got = host64(E.espace_project(Pt, X, out_mat(N, L, "bf16", dev)))
            torch.cuda.synchronize()
            # the pair plans of these shapes use 128 x 192 and 256 x 192 tiles:
            # compare on 128 x 64 pieces, which both tile sizes cover whole
            nan_tiles += _tiles_ok_or_nan(got, ref, 128, 64)
    finally:
        E.espace_set_wait_limit(0)
    n1 = E.espace_wait_timeouts()
    assert (n1 > n0) == (nan_tiles > 0), (n0, n1, nan_tiles)
    again = host64(E.espace_project(Pt, X))
    torch.cuda.synchronize()
    assert np.array_equal(again, ref)
    assert E.espace_wait_timeouts() == n1


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
            Z64 = oracle.project(inps[0].Pt, inps[rep].X)
            B = parity.product_bound(Z64, parity.row_norms(inps[rep].X), parity.row_norms(inps[0].Pt), K,
                                     parity.U_BF16)
            parity.check(host64(got), Z64, B, TOL["bf16"], f"replay {rep}")


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
    i0 = inps[0]
    Z64 = oracle.project(i0.Pt, i0.X)
    Wf64 = oracle.fold(i0.W, i0.Pt)
    Y64 = oracle.expand(Z64, Wf64)
    B = parity.layer_bound(Y64, Z64, Wf64, parity.row_norms(i0.X), parity.row_norms(i0.Pt), parity.row_norms(i0.W),
                           K, L, parity.U_BF16)
    parity.check(host64(Y), Y64, B, 1e-2, "prefill layer under graph replay")


# (K, M, L, N) of prefill layers: a projection whose tiles split their depth
# in two halves combined in-kernel (the Llama2-7B shape class), ragged token
# blocks, components and features (a feature count that is not a multiple of
# 8 takes the scalar stores), a projection of more tiles than CUs
PREFILL_SHAPES = [(4100, 3000, 1536, 4096), (1003, 517, 131, 301), (700, 1234, 520, 5000),
                (4500, 1000, 4000, 4096), (2048, 4096, 256, 40)]


def _layer_ref(inp):
    w = inp.w
    Z64 = oracle.project(inp.Pt, inp.X)
    Wf64 = oracle.fold(inp.W, inp.Pt)
    Y64 = oracle.expand(Z64, Wf64)
    B = parity.layer_bound(Y64, Z64, Wf64, parity.row_norms(inp.X), parity.row_norms(inp.Pt),
                           parity.row_norms(inp.W), w.K, w.L, parity.U_BF16)
    return Y64, B


@pytest.mark.parametrize("shape", PREFILL_SHAPES, ids=lambda s: "K%d_M%d_L%d_N%d" % s)
def test_prefill_layer_shapes(E, shape):
    """The projected linear layer at prefill shapes against the oracle on every
    output, and bitwise identical whatever its workspace held before (zeros,
    all ones, random bytes, the previous call's state): the in-kernel pair
    combine's state words carry a per-call tag."""
    dev = need_gpu()
    K, M, L, N = shape
    inp = _inputs(K, M, L, N, "bf16", seed=80)
    X, Pt, W = _dev_inputs(inp, dev)
    Wf = E.espace_fold_weights(W, Pt)
    Y = E.espace_projected_linear(X, Pt, Wf, out_mat(N, M, "bf16", dev))
    torch.cuda.synchronize()
    Y64, B = _layer_ref(inp)
    parity.check(host64(Y), Y64, B, TOL["bf16"], "prefill layer")
    assert np.isnan(padding(Y)).all()
    need = E.espace_workspace_bytes(E.OP_PROJECTED_LINEAR, M, K, L, N, torch.bfloat16)
    ws = torch.empty(need, dtype=torch.uint8, device=dev)
    gen = torch.Generator(device="cpu").manual_seed(8)
    for fill in ["zeros", "ones", "random", "keep", "keep"]:
        if fill == "zeros":
            ws.zero_()
        elif fill == "ones":
            ws.fill_(255)
        elif fill == "random":
            ws.copy_(torch.randint(0, 256, (need,), dtype=torch.uint8, generator=gen))
        assert torch.equal(E.espace_projected_linear(X, Pt, Wf, workspace=ws), Y), fill


# (K, M, L, N) of prefill layers that keep Z in the row-pair layout (an odd
# token count, whose last pair has one token; a component count that is not a
# multiple of 64, or of 8, with the expand GEMM's masked depth tail on row
# pairs; projections on the 128 x 192 tile, on the four-wave 256 x 192 tile
# in two depth halves (depth 11008), with a projection depth tail, in two
# launches split by rows (the first in two depth halves; the GPT3-22B FFN-up
# class at L = 2458), and in four depth ranges summed by the reduction pass)
ROW_PAIR_SHAPES = [(4096, 12288, 1536, 4095), (4096, 6000, 1500, 4095), (4100, 12288, 1300, 4095),
                   (11008, 4096, 1536, 4095), (6144, 2048, 2458, 8191), (8192, 12288, 1000, 2047)]


def _row_pairs(Z, ldp):
    """Z [N][L] (float32 values of bf16 entries) in the row-pair layout with
    pair pitch ldp: element (n, l) at (n // 2) * ldp + (l // 32) * 64 +
    (n % 2) * 32 + l % 32; the unused places are left at zero."""
    N, L = Z.shape
    out = np.zeros(((N + 1) // 2) * ldp, dtype=np.float32)
    n = np.arange(N)[:, None]
    l = np.arange(L)[None, :]
    out[(n // 2) * ldp + (l // 32) * 64 + (n % 2) * 32 + l % 32] = Z
    return out


@pytest.mark.parametrize("shape", ROW_PAIR_SHAPES, ids=lambda s: "K%d_M%d_L%d_N%d" % s)
def test_prefill_layer_row_pair_z(E, shape):
    """The prefill layer keeps Z in its workspace in row pairs (two tokens' 32
    consecutive components per 128-byte block): the workspace's Z region holds
    exactly the projection's Z in that layout, the layer's result equals the
    projection followed by the expansion on a plain Z bitwise (the layout moves
    no arithmetic), and it is within the oracle's bounds on every output."""
    dev = need_gpu()
    K, M, L, N = shape
    inp = _inputs(K, M, L, N, "bf16", seed=85)
    X, Pt, W = _dev_inputs(inp, dev)
    Wf = E.espace_fold_weights(W, Pt)
    need = E.espace_workspace_bytes(E.OP_PROJECTED_LINEAR, M, K, L, N, torch.bfloat16)
    ws = torch.zeros(need, dtype=torch.uint8, device=dev)
    Y = E.espace_projected_linear(X, Pt, Wf, out_mat(N, M, "bf16", dev), ws)
    Z = E.espace_project(Pt, X)
    Ye = E.espace_expand(Z, Wf)
    torch.cuda.synchronize()
    ldp = 2 * ((L + 63) // 64 * 64)
    pairs = _row_pairs(Z.float().cpu().numpy(), ldp)
    got = ws[:pairs.size * 2].view(torch.bfloat16).float().cpu().numpy()
    keep = np.zeros(pairs.size, dtype=bool)
    n = np.arange(N)[:, None]
    l = np.arange(L)[None, :]
    keep[(n // 2) * ldp + (l // 32) * 64 + (n % 2) * 32 + l % 32] = True
    assert np.array_equal(got[keep], pairs[keep]), "workspace Z is not the projection in row pairs"
    assert torch.equal(Y, Ye), "layer != project then expand"
    Y64, B = _layer_ref(inp)
    parity.check(host64(Y), Y64, B, TOL["bf16"], "prefill layer, Z in row pairs")
    assert np.isnan(padding(Y)).all()


# (K, M, L, N) of decode layers on the whole-row kernels: one and two tokens,
# Wf rows of one to eight 512-element passes, projection depths with a
# partial block of passes
DECODE_LAYER_SHAPES = [(4096, 22016, 1536, 1), (4096, 12288, 1536, 2), (11008, 4096, 1536, 1),
                       (6144, 24576, 3686, 1), (4500, 3001, 2458, 2), (700, 1234, 520, 2), (64, 17, 8, 1)]


@pytest.mark.parametrize("shape", DECODE_LAYER_SHAPES, ids=lambda s: "K%d_M%d_L%d_N%d" % s)
def test_decode_layer_shapes(E, shape):
    """The decode layer against the oracle on every output, equal bitwise to
    the projection followed by the expansion, and bitwise the same whatever
    its workspace held before (zeros, all ones, random bytes, the previous
    call's Z)."""
    dev = need_gpu()
    K, M, L, N = shape
    inp = _inputs(K, M, L, N, "bf16", seed=90)
    X, Pt, W = _dev_inputs(inp, dev)
    Wf = E.espace_fold_weights(W, Pt)
    Y = E.espace_projected_linear(X, Pt, Wf, out_mat(N, M, "bf16", dev))
    Ye = E.espace_expand(E.espace_project(Pt, X), Wf)
    torch.cuda.synchronize()
    assert torch.equal(Y, Ye), "layer != project then expand"
    Y64, B = _layer_ref(inp)
    parity.check(host64(Y), Y64, B, TOL["bf16"], "decode layer")
    assert np.isnan(padding(Y)).all()
    need = E.espace_workspace_bytes(E.OP_PROJECTED_LINEAR, M, K, L, N, torch.bfloat16)
    ws = torch.empty(need, dtype=torch.uint8, device=dev)
    gen = torch.Generator(device="cpu").manual_seed(9)
    for fill in ["zeros", "ones", "random", "keep", "keep"]:
        if fill == "zeros":
            ws.zero_()
        elif fill == "ones":
            ws.fill_(255)
        elif fill == "random":
            ws.copy_(torch.randint(0, 256, (need,), dtype=torch.uint8, generator=gen))
        assert torch.equal(E.espace_projected_linear(X, Pt, Wf, workspace=ws), Y), fill


@pytest.mark.parametrize("N", [1, 16])
def test_decode_layer_under_graph_replay(E, N):
    """The decode layer captured in a HIP graph and replayed with new tokens
    copied in between: every replay equals the eager call bitwise (one token:
    the whole-row kernels; 16 tokens: the depth-segmented projection and the
    LDS-ring expansion)."""
    dev = need_gpu()
    K, M, L = 4096, 12288, 1536
    inps = [_inputs(K, M, L, N, "bf16", seed=95 + i) for i in range(2)]
    X, Pt, W = _dev_inputs(inps[0], dev)
    Wf = E.espace_fold_weights(W, Pt)
    Y = out_mat(N, M, "bf16", dev)
    ws = torch.empty(E.espace_workspace_bytes(E.OP_PROJECTED_LINEAR, M, K, L, N, torch.bfloat16),
                     dtype=torch.uint8, device=dev)
    E.espace_projected_linear(X, Pt, Wf, Y, ws)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        E.espace_projected_linear(X, Pt, Wf, Y, ws)
    torch.cuda.synchronize()
    for rep in range(6):
        X.copy_(dev_mat(inps[rep % 2].X_s, "bf16", dev))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = Y.clone()
        ref = E.espace_projected_linear(X, Pt, Wf)
        torch.cuda.synchronize()
        assert torch.equal(got, ref), rep
