"""The GPU path on the five full-size workloads, against the fp64 oracle.

Every output of the projected linear layer and of the dense baseline is
compared, entry by entry, with the criteria of tests/parity.py (finite
everywhere in NaN-prefilled outputs, the derived rounding bound per entry,
relative Frobenius error <= 1e-2 over the whole output and over every 64 x 64
block), in the launch configuration the benchmark times.  For the GPT3-22B
layers the oracle's folded weight is computed once per (layer, L) and reused
across the token counts."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests import parity
from tests.gpu_util import dev_mat, host64, need_gpu, out_mat

pytestmark = pytest.mark.gpu

U = parity.U_BF16
TOL = parity.TOL["bf16"]


@pytest.fixture(scope="module")
def E():
    need_gpu()
    import paper_2410_05437_amd as e
    return e


class _Ref:
    """Oracle quantities of one (layer, L): the exact fold and the row norms."""

    def __init__(self, inp):
        self.Wf64 = oracle.fold(inp.W, inp.Pt)
        self.pn = parity.row_norms(inp.Pt)
        self.wn = parity.row_norms(inp.W)


def _gpu_layer(E, inp, dev, Wf=None):
    w = inp.w
    X = dev_mat(inp.X_s, "bf16", dev)
    Pt = dev_mat(inp.Pt_s, "bf16", dev)
    if Wf is None:
        W = dev_mat(inp.W_s, "bf16", dev)
        Wf = E.espace_fold_weights(W, Pt, out_mat(w.M, w.L, "bf16", dev))
        del W
    Y = E.espace_projected_linear(X, Pt, Wf, out_mat(w.N, w.M, "bf16", dev))
    torch.cuda.synchronize()
    return host64(Y), Wf


def _gpu_dense(E, inp, dev):
    w = inp.w
    X = dev_mat(inp.X_s, "bf16", dev)
    W = dev_mat(inp.W_s, "bf16", dev)
    Yd = E.espace_dense_linear(X, W, out_mat(w.N, w.M, "bf16", dev))
    torch.cuda.synchronize()
    return host64(Yd)


def _check_layer(Yg, inp, ref, what):
    w = inp.w
    Z64 = oracle.project(inp.Pt, inp.X)
    Y64 = oracle.expand(Z64, ref.Wf64)
    B = parity.layer_bound(Y64, Z64, ref.Wf64, parity.row_norms(inp.X), ref.pn, ref.wn, w.K, w.L, U)
    rel, blk, ratio = parity.check(Yg, Y64, B, TOL, what)
    print(f"{what}: rel_fro {rel:.3e}, worst 64x64 block {blk:.3e}, worst error/bound {ratio:.3f}")


def _check_dense(Ydg, inp, wn, what):
    w = inp.w
    Yd64 = oracle.dense(inp.X, inp.W)
    B = parity.product_bound(Yd64, parity.row_norms(inp.X), wn, w.K, U)
    rel, blk, ratio = parity.check(Ydg, Yd64, B, TOL, what)
    print(f"{what}: rel_fro {rel:.3e}, worst 64x64 block {blk:.3e}, worst error/bound {ratio:.3f}")


def _fold_check(Wf_gpu, inp, ref, what):
    Wfg = host64(Wf_gpu)
    B = parity.product_bound(ref.Wf64, ref.wn, ref.pn, inp.w.K, U)
    parity.check(Wfg, ref.Wf64, B, TOL, what)


@pytest.mark.timeout(600)
def test_llama2_7b_qkv_full(E):
    """Llama2-7B fused QKV (K=4096, M=12288, L=1536, N=4096), the benchmark's
    workload: fold, layer and dense baseline, every output."""
    dev = need_gpu()
    inp = synth.make_inputs(synth.workload(1))
    ref = _Ref(inp)
    Yg, Wf = _gpu_layer(E, inp, dev)
    _fold_check(Wf, inp, ref, "llama2-7b qkv fold")
    del Wf
    _check_layer(Yg, inp, ref, "llama2-7b qkv")
    del Yg
    _check_dense(_gpu_dense(E, inp, dev), inp, ref.wn, "llama2-7b qkv dense")


@pytest.mark.timeout(900)
def test_llama2_7b_ffn_upgate(E):
    """Llama2-7B FFN up+gate (K=4096, M=22016, L=1536) at N = 4096, 1, 8 and
    16 tokens (decode uses the first N tokens of the prefill draw)."""
    dev = need_gpu()
    ref = None
    Wf = None
    for N in (4096, 1, 8, 16):
        inp = synth.make_inputs(synth.workload(2, N=N))
        if ref is None:
            ref = _Ref(inp)
        Yg, Wf = _gpu_layer(E, inp, dev, Wf)
        if N == 4096:
            _fold_check(Wf, inp, ref, "llama2-7b ffn up+gate fold")
        _check_layer(Yg, inp, ref, f"llama2-7b ffn up+gate N={N}")
        del Yg
        _check_dense(_gpu_dense(E, inp, dev), inp, ref.wn, f"llama2-7b ffn up+gate dense N={N}")


@pytest.mark.timeout(600)
def test_llama2_7b_ffn_down_full(E):
    """Llama2-7B FFN down (K=11008, M=4096, L=1536, N=4096): SiLU-gated tokens,
    P calibrated on 16384 separate tokens."""
    dev = need_gpu()
    inp = synth.make_inputs(synth.workload(3))
    ref = _Ref(inp)
    Yg, Wf = _gpu_layer(E, inp, dev)
    _fold_check(Wf, inp, ref, "llama2-7b ffn down fold")
    del Wf
    _check_layer(Yg, inp, ref, "llama2-7b ffn down")
    del Yg
    _check_dense(_gpu_dense(E, inp, dev), inp, ref.wn, "llama2-7b ffn down dense")


def _gpt3_cases():
    seen = []
    for w in synth.workloads(4):
        if (w.layer, w.L) not in seen:
            seen.append((w.layer, w.L))
    return seen


@pytest.mark.timeout(900)
@pytest.mark.parametrize("layer_L", _gpt3_cases(), ids=lambda c: f"{c[0]}_L{c[1]}")
def test_gpt3_22b_ffn_full(E, layer_L):
    """GPT3-22B FFN up (K=6144, M=24576) and down (K=24576, M=6144) over the
    compression sweep L in {3686, 2458, 1966}, each at N in {8192, 1, 16}:
    the layer, every output; the fold once per (layer, L)."""
    dev = need_gpu()
    layer, L = layer_L
    ref = None
    Wf = None
    for w in synth.workloads(4):
        if (w.layer, w.L) != (layer, L):
            continue
        inp = synth.make_inputs(w)
        if ref is None:
            ref = _Ref(inp)
        Yg, Wf = _gpu_layer(E, inp, dev, Wf)
        if w.N == 8192:
            _fold_check(Wf, inp, ref, f"gpt3-22b {layer} L={L} fold")
        _check_layer(Yg, inp, ref, f"gpt3-22b {layer} L={L} N={w.N}")
        del Yg


@pytest.mark.timeout(900)
@pytest.mark.parametrize("layer", ["up", "down"])
def test_gpt3_22b_ffn_dense_full(E, layer):
    """The dense baseline of the GPT3-22B FFN layers at N in {8192, 1, 16},
    every output."""
    dev = need_gpu()
    wn = None
    for w in synth.workloads(4):
        if w.layer != layer or w.L != 2458:
            continue
        inp = synth.make_inputs(w)
        if wn is None:
            wn = parity.row_norms(inp.W)
        _check_dense(_gpu_dense(E, inp, dev), inp, wn, f"gpt3-22b {layer} dense N={w.N}")
