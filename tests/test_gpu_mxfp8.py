"""The MX-FP8 layer on the GPU against the oracle (criteria in
tests/mx_parity.py).

Both sides quantise the same bfloat16 inputs: the GPU with
espace_quantize_mxfp8, the oracle with mx_quantize; the two are compared
byte for byte first, and each side then runs its own layer.  The projection's
Z codes and scales are checked for validity entry by entry, the expansion
against the oracle's exact product within the MFMA chain's bound, and the
layer against the oracle's layer within that bound plus what a valid
re-quantisation of Z may move."""
import numpy as np
import pytest
import torch

import oracle
import synth
from synth.bf16 import bf16_bits_from_f64
from tests import mx_parity as MP
from tests.gpu_util import dev_mat, host64, need_gpu, out_mat

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def E():
    need_gpu()
    import paper_2410_05437_amd as e
    return e


def _bf16_values(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


class _Case:
    """Seeded inputs of one layer shape: X and Pt from the workload generator,
    Wf = the oracle's fold rounded to bfloat16 (the input both sides
    quantise)."""

    def __init__(self, K, M, L, N, seed):
        w = synth.Workload(cfg=-1, name="mx", K=K, M=M, L=L, N=N, dtype="bf16", recipe="gaussian",
                           lam_floor=1e-4, proj="leading", cov_key=seed, w_key=seed + 1)
        inp = synth.make_inputs(w)
        self.K, self.M, self.L, self.N = K, M, L, N
        self.X_s, self.Pt_s = inp.X_s, inp.Pt_s
        self.X, self.Pt = inp.X, inp.Pt
        self.Wf_s = bf16_bits_from_f64(oracle.fold(inp.W, inp.Pt))
        self.Wf = _bf16_values(self.Wf_s)
        self.Xq, self.Xb = oracle.mx_quantize(self.X)
        self.Pq, self.Pb = oracle.mx_quantize(self.Pt)
        self.Wq, self.Wb = oracle.mx_quantize(self.Wf)

    def gpu_operands(self, E, dev):
        X = E.espace_quantize_mxfp8(dev_mat(self.X_s, "bf16", dev))
        Pt = E.espace_quantize_mxfp8(dev_mat(self.Pt_s, "bf16", dev))
        Wf = E.espace_quantize_mxfp8(dev_mat(self.Wf_s, "bf16", dev))
        torch.cuda.synchronize()
        return X, Pt, Wf


def _check_quantized(m, q, b, what):
    """GPU MX tensor equals the oracle's codes and scale bytes byte for byte;
    its padding columns and padding blocks are zero."""
    vals, sb, codes, scales = MP.gpu_mx(m)
    want = oracle.e4m3_encode(q)
    got = codes[:, :m.cols]
    bad = np.argwhere(got != want)
    assert not len(bad), f"{what}: {len(bad)} codes differ, first {bad[0].tolist()}: {got[tuple(bad[0])]:#x} " \
                         f"vs {want[tuple(bad[0])]:#x}"
    assert np.array_equal(sb, b.astype(np.int64)), f"{what}: scale bytes differ"
    cp = (m.cols + 127) // 128 * 128
    assert not codes[:, m.cols:cp].any(), f"{what}: padding codes not zero"
    assert not scales[:, -(-m.cols // 32):cp // 32].any(), f"{what}: padding scale bytes not zero"


# (K, M, L, N).  The fourth and fifth: more 256 x 256 expansion tiles than CUs
# (264: workgroups take a second tile, whose first two steps the first one
# loads), and a ragged width (M % 8 = 4: element-wise stores) with one depth
# step.  The last three: projections on 128 x 192 tiles with three stages
# (between 128 and 256 tiles): ragged tokens, width and depth over 25 steps,
# and depths of two steps and one step.
SHAPES = [(512, 384, 200, 300), (1024, 2048, 256, 4096), (704, 1000, 520, 1000), (256, 8448, 256, 2048),
          (300, 1100, 100, 333), (3100, 256, 3000, 2000), (250, 200, 200, 9000), (100, 64, 100, 20000)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "K%d_M%d_L%d_N%d" % s)
def test_mxfp8_layer(E, shape):
    """Quantisation byte for byte, the projection's codes valid entry by entry,
    the expansion and the layer within their bounds, and the layer equal to
    the projection followed by the expansion."""
    dev = need_gpu()
    K, M, L, N = shape
    c = _Case(K, M, L, N, seed=300 + K % 97)
    X, Pt, Wf = c.gpu_operands(E, dev)
    _check_quantized(X, c.Xq, c.Xb, "X")
    _check_quantized(Pt, c.Pq, c.Pb, "Pt")
    _check_quantized(Wf, c.Wq, c.Wb, "Wf")

    # projection: every code and scale byte valid for the exact Z within the bound
    Z = E.espace_project_mxfp8(Pt, X)
    torch.cuda.synchronize()
    Xd, Pd, Wd = oracle.mx_dequantize(c.Xq, c.Xb), oracle.mx_dequantize(c.Pq, c.Pb), oracle.mx_dequantize(c.Wq, c.Wb)
    Zx, Ez = MP.chain_bound(Xd, Pd, MP.STEP_PROJECT)
    assert np.allclose(Zx, oracle.mx_project(c.Xq, c.Xb, c.Pq, c.Pb), rtol=1e-12, atol=0)
    zv, zb, _, _ = MP.gpu_mx(Z)
    same = MP.check_mx_codes(Zx, Ez, zv, zb, "Z")
    _check_padding_zero(Z)

    # expansion on the oracle's quantisation of Z (the same bytes through the GPU's quantiser)
    Zo, Zob = oracle.mx_quantize(Zx)
    Zod = oracle.mx_dequantize(Zo, Zob)
    Zin = E.espace_quantize_mxfp8(dev_mat(bf16_bits_from_f64(Zod), "bf16", dev)) if _bf16_exact(Zod) else None
    Yo, Ey = MP.chain_bound(Zod, Wd, MP.STEP_EXPAND)
    if Zin is not None:
        _check_quantized(Zin, Zo, Zob, "Z (oracle's, through the GPU quantiser)")
        Ye = E.espace_expand_mxfp8(Zin, Wf, out_mat(N, M, "bf16", dev))
        torch.cuda.synchronize()
        ratio, rel = MP.check_bound(host64(Ye), Yo, Ey + MP.U_BF16 * (np.abs(Yo) + Ey), "expand")
        print(f"expand: worst error/bound {ratio:.3f}, rel_fro {rel:.2e}")

    # the layer, and the layer as the two calls
    Y = E.espace_projected_linear_mxfp8(X, Pt, Wf, out_mat(N, M, "bf16", dev))
    Y2 = E.espace_expand_mxfp8(Z, Wf, out_mat(N, M, "bf16", dev))
    torch.cuda.synchronize()
    assert torch.equal(Y, Y2), "layer != project then expand"
    width = MP.z_value_width(Zx, Ez)
    spread = width @ np.abs(Wd).T
    B = Ey + spread * (1 + 1 / 8) + MP.U_BF16 * (np.abs(Yo) + Ey + spread)
    ratio, rel = MP.check_bound(host64(Y), Yo, B, "layer")
    exact = c.X @ c.Pt.T @ c.Wf.T
    qerr = float(np.linalg.norm(host64(Y) - exact) / np.linalg.norm(exact))
    print(f"layer {shape}: Z codes equal to the oracle's {same:.4f}, worst error/bound {ratio:.3f}, "
          f"rel_fro {rel:.2e}; against the unquantised layer {qerr:.3e}")


def _bf16_exact(A):
    """True when every entry is a bfloat16 value (MX-FP8 values with scales in
    the bfloat16 range are)."""
    bits = bf16_bits_from_f64(A)
    return np.array_equal(_bf16_values(bits), A)


def _check_padding_zero(m):
    _, _, codes, scales = MP.gpu_mx(m)
    cp = (m.cols + 127) // 128 * 128
    assert not codes[:, m.cols:cp].any(), "Z padding codes not zero"
    assert not scales[:, -(-m.cols // 32):cp // 32].any(), "Z padding scale bytes not zero"


def test_mxfp8_quantize_edges(E):
    """Quantisation of blocks with zeros, one dominant entry, values past the
    E4M3 range after scaling (clamped), tiny magnitudes and a ragged tail, byte
    for byte against the oracle; padding columns hold NaN, which is never read."""
    dev = need_gpu()
    rng = np.random.default_rng(7)
    R, C = 9, 333
    A = rng.standard_normal((R, C)) * np.exp(rng.uniform(-20, 20, (R, 1)))
    A[0, :64] = 0.0
    A[1, 3] = 3e4
    A[2, 32:64] = 1.0
    A[2, 40] = 1.9375          # block max 1.9375: 1.9375 / 2^-8 = 496 -> clamped to 448
    A[3, :] = 1e-30
    A[4, ::7] = -A[4, ::7]
    bits = bf16_bits_from_f64(A)
    vals = _bf16_values(bits)
    m = E.espace_quantize_mxfp8(dev_mat(bits, "bf16", dev))
    torch.cuda.synchronize()
    q, b = oracle.mx_quantize(vals)
    _check_quantized(m, q, b, "edge blocks")
    assert oracle.mx_quantize(np.array([[1.9375] + [1.0] * 31]))[0][0, 0] == 448.0


@pytest.mark.timeout(600)
def test_mxfp8_llama2_7b_qkv_sampled(E):
    """The Llama2-7B fused QKV layer at full size (K=4096, M=12288, L=1536,
    N=4096) in the benchmark's launch configuration: quantisation byte for
    byte on every entry, the projection's codes on 256 sampled tokens (all
    components), and the layer on those tokens (all features)."""
    dev = need_gpu()
    inp = synth.make_inputs(synth.workload(1))
    K, M, L, N = 4096, 12288, 1536, 4096
    Wf_s = bf16_bits_from_f64(oracle.fold(inp.W, inp.Pt))
    Wf64 = _bf16_values(Wf_s)
    Xq, Xb = oracle.mx_quantize(inp.X)
    Pq, Pb = oracle.mx_quantize(inp.Pt)
    Wq, Wb = oracle.mx_quantize(Wf64)
    X = E.espace_quantize_mxfp8(dev_mat(inp.X_s, "bf16", dev))
    Pt = E.espace_quantize_mxfp8(dev_mat(inp.Pt_s, "bf16", dev))
    Wf = E.espace_quantize_mxfp8(dev_mat(Wf_s, "bf16", dev))
    torch.cuda.synchronize()
    _check_quantized(X, Xq, Xb, "X")
    _check_quantized(Pt, Pq, Pb, "Pt")
    _check_quantized(Wf, Wq, Wb, "Wf")
    Z = E.espace_project_mxfp8(Pt, X)
    Y = E.espace_projected_linear_mxfp8(X, Pt, Wf, out_mat(N, M, "bf16", dev))
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(11).choice(N, 256, replace=False))
    Xd = oracle.mx_dequantize(Xq[rows], Xb[rows])
    Pd, Wd = oracle.mx_dequantize(Pq, Pb), oracle.mx_dequantize(Wq, Wb)
    Zx, Ez = MP.chain_bound(Xd, Pd, MP.STEP_PROJECT)
    zv, zb, _, _ = MP.gpu_mx(Z, rows)
    same = MP.check_mx_codes(Zx, Ez, zv, zb, "Z")
    Zo, Zob = oracle.mx_quantize(Zx)
    Yo, Ey = MP.chain_bound(oracle.mx_dequantize(Zo, Zob), Wd, MP.STEP_EXPAND)
    spread = MP.z_value_width(Zx, Ez) @ np.abs(Wd).T
    B = Ey + spread * (1 + 1 / 8) + MP.U_BF16 * (np.abs(Yo) + Ey + spread)
    ratio, rel = MP.check_bound(host64(Y)[rows], Yo, B, "layer")
    print(f"llama2-7b qkv mxfp8: Z codes equal to the oracle's {same:.4f}, worst error/bound {ratio:.3f}, "
          f"rel_fro {rel:.2e}")


# (N, L, K) of projections whose operands' scale rows are laid out twice: at
# the smallest leading dimension (not a multiple of 16 bytes: one scale
# dword per row and step) and padded to 16 bytes as the library allocates
# them (four steps' scales per 16-byte load), on 128 x 192 tiles with three stages (6 steps: a last group
# of two), 128 x 128 tiles with two stages, and 256 x 256 tiles (33 steps).
SCALE_LAYOUTS = [(5000, 700, 700), (1000, 300, 700), (4096, 4096, 4100)]


@pytest.mark.parametrize("shape", SCALE_LAYOUTS, ids=lambda s: "N%d_L%d_K%d" % s)
def test_mxfp8_projection_scale_layouts(E, shape):
    """The projection gives the same codes and scale bytes, bit for bit,
    whichever scale-load path the operands' layout selects."""
    dev = need_gpu()
    N, L, K = shape
    gen = torch.Generator(device="cpu").manual_seed(N + L + K)
    X = E.padded_empty(N, K, torch.bfloat16, dev)
    X.copy_(torch.randn(N, K, generator=gen).to(torch.bfloat16))
    Pt = E.padded_empty(L, K, torch.bfloat16, dev)
    Pt.copy_((torch.randn(L, K, generator=gen) * K ** -0.5).to(torch.bfloat16))
    cp = (K + 127) // 128 * 128
    assert (cp // 32) % 16 != 0, "the smallest scale rows must not be 16-byte multiples"
    spad = (cp // 32 + 15) // 16 * 16

    def tight(rows):
        return E.MXTensor(torch.empty((rows, cp), dtype=torch.uint8, device=dev),
                          torch.empty((rows, cp // 32), dtype=torch.uint8, device=dev), K)

    X1 = E.espace_quantize_mxfp8(X, out=tight(N))
    P1 = E.espace_quantize_mxfp8(Pt, out=tight(L))
    X4, P4 = E.espace_quantize_mxfp8(X), E.espace_quantize_mxfp8(Pt)
    assert X4.scales.stride(0) == spad and P4.scales.stride(0) == spad
    Z1, Z4 = E.espace_project_mxfp8(P1, X1), E.espace_project_mxfp8(P4, X4)
    torch.cuda.synchronize()
    assert torch.equal(X1.scales, X4.scales) and torch.equal(P1.scales, P4.scales)
    assert torch.equal(Z1.codes, Z4.codes), "Z codes differ between the scale layouts"
    assert torch.equal(Z1.scales, Z4.scales), "Z scale bytes differ between the scale layouts"
    assert Z1.codes[:, :L].any(), "Z is all zero"


# (N, M, L) of expansions run on both scale layouts: 6 steps over 528 tiles of
# 256 x 256 (workgroups take two or three tiles, the next tile's first steps
# loaded ahead, groups of four steps continuing across tiles), 11 steps on
# the same tiles, and 5 and 25 steps on 256 x 128 tiles.
EXPAND_LAYOUTS = [(4096, 8448, 700), (4096, 8448, 1400), (2000, 1000, 600), (1000, 3000, 3100)]


@pytest.mark.parametrize("shape", EXPAND_LAYOUTS, ids=lambda s: "N%d_M%d_L%d" % s)
def test_mxfp8_expansion_scale_layouts(E, shape):
    """The expansion gives the same output, bit for bit, with one scale dword
    per step loaded (scale rows not 16-byte multiples) and with four steps'
    scales per load (the library's padded rows)."""
    dev = need_gpu()
    N, M, L = shape
    gen = torch.Generator(device="cpu").manual_seed(N + M + L)
    Zb = E.padded_empty(N, L, torch.bfloat16, dev)
    Zb.copy_(torch.randn(N, L, generator=gen).to(torch.bfloat16))
    Wb = E.padded_empty(M, L, torch.bfloat16, dev)
    Wb.copy_((torch.randn(M, L, generator=gen) * L ** -0.5).to(torch.bfloat16))
    cp = (L + 127) // 128 * 128
    assert (cp // 32) % 16 != 0, "the smallest scale rows must not be 16-byte multiples"

    def tight(rows):
        return E.MXTensor(torch.empty((rows, cp), dtype=torch.uint8, device=dev),
                          torch.empty((rows, cp // 32), dtype=torch.uint8, device=dev), L)

    Z1, W1 = E.espace_quantize_mxfp8(Zb, out=tight(N)), E.espace_quantize_mxfp8(Wb, out=tight(M))
    Z4, W4 = E.espace_quantize_mxfp8(Zb), E.espace_quantize_mxfp8(Wb)
    assert Z4.scales.stride(0) % 16 == 0 and W4.scales.stride(0) % 16 == 0
    Y1 = E.espace_expand_mxfp8(Z1, W1, out_mat(N, M, "bf16", dev))
    Y4 = E.espace_expand_mxfp8(Z4, W4, out_mat(N, M, "bf16", dev))
    torch.cuda.synchronize()
    assert torch.equal(Y1, Y4), "Y differs between the scale layouts"
    assert torch.isfinite(Y4.float()).all() and Y4.abs().sum() > 0
