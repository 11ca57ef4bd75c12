"""The C ABI without a GPU: the library loads, exports every function the
header declares, and rejects invalid arguments before touching any device."""
import ctypes

import pytest

import paper_2410_05437_amd as E
from paper_2410_05437_amd import _lib

L = E.lib
P16 = ctypes.c_void_p(0x10000)      # fake, 16-byte aligned; never dereferenced
P16b = ctypes.c_void_p(0x20000000)
P16c = ctypes.c_void_p(0x40000000)
NULL = ctypes.c_void_p(0)


def test_exports_every_declared_function():
    names = E.header_functions()
    assert set(names) == {
        "espace_fold_weights", "espace_project", "espace_expand", "espace_projected_linear",
        "espace_dense_linear", "espace_workspace_bytes", "espace_status_string",
        "espace_last_error", "espace_abi_version", "espace_autocorrelation_update",
        "espace_principal_components", "espace_symmetrized_product", "espace_projected_linear_backward",
        "espace_dense_linear_backward", "espace_wait_timeouts", "espace_set_wait_limit",
        "espace_projected_linear_noalloc", "espace_quantize_mxfp8", "espace_project_mxfp8",
        "espace_expand_mxfp8", "espace_projected_linear_mxfp8"}
    for n in names:
        assert hasattr(L, n)
    assert E.ABI_VERSION == 7


def _fold(W=P16, ldw=64, Pt=P16b, ldp=64, Wf=P16c, ldwf=16, M=32, K=64, Lc=16, dt=1,
          ws=NULL, wsb=0):
    return L.espace_fold_weights(W, ldw, Pt, ldp, Wf, ldwf, M, K, Lc, dt, ws, wsb, NULL)


def _pl(X=P16, ldx=64, Pt=P16b, ldp=64, Wf=P16c, ldwf=16, Y=ctypes.c_void_p(0x60000000),
        ldy=32, M=32, K=64, Lc=16, N=8, dt=1, ws=ctypes.c_void_p(0x70000000), wsb=1 << 20):
    return L.espace_projected_linear(X, ldx, Pt, ldp, Wf, ldwf, Y, ldy, M, K, Lc, N, dt, ws, wsb, NULL)


def _status_and_msg(s):
    return s, L.espace_last_error().decode()


def test_validation_errors():
    assert _fold(W=NULL) == 1                                           # NULL
    assert _fold(Lc=65) == 2                                            # L > K
    assert _fold(Lc=0) == 2
    assert _fold(K=0) == 2
    assert _fold(M=-1) == 2
    assert _fold(ldw=60) == 2                                           # ld < cols
    assert _fold(ldw=68) == 3                                           # ld % 8
    assert _fold(W=ctypes.c_void_p(0x10008)) == 3                       # pointer alignment
    assert _fold(dt=7) == 4
    assert _fold(Wf=ctypes.c_void_p(0x10000 + 64)) == 5                 # Wf inside W
    s, msg = _status_and_msg(_fold(Wf=ctypes.c_void_p(0x10000 + 64)))
    assert "overlaps" in msg
    assert _pl(ws=NULL, wsb=0) == 6                                     # workspace missing
    assert _pl(wsb=16) == 6                                             # workspace too small
    assert _pl(ws=ctypes.c_void_p(0x70000010)) == 3                     # workspace alignment
    assert _pl(ws=ctypes.c_void_p(0x10000)) == 5                        # workspace over X


def test_empty_sizes_return_ok_without_a_device():
    assert _fold(M=0, W=NULL, Wf=NULL) == 0
    assert _pl(N=0, X=NULL, Y=NULL, ws=NULL, wsb=0) == 0
    assert _pl(M=0, Wf=NULL, Y=NULL, ws=NULL, wsb=0) == 0


def test_valid_call_without_gpu_reports_device_error():
    # every argument is valid, so the library asks the HIP runtime for the device
    s = _pl()
    assert s in (7, 8), (s, L.espace_last_error())


def test_workspace_sizes():
    bf16, f32 = 1, 0
    ws = L.espace_workspace_bytes
    # prefill Llama2-7B QKV: only Z (N x round_up(L, 64) bf16)
    assert ws(3, 12288, 4096, 1536, 4096, bf16) == 4096 * 1536 * 2
    assert ws(4, 12288, 4096, 0, 4096, bf16) == 0
    assert ws(3, 12288, 4096, 1536, 0, bf16) == 0
    assert ws(3, 12288, 4096, 5000, 4096, bf16) == ctypes.c_size_t(-1).value
    assert ws(99, 1, 1, 1, 1, bf16) == ctypes.c_size_t(-1).value
    assert ws(3, 256, 256, 64, 128, f32) == 128 * 64 * 4
    # ragged L: Z rows padded to a multiple of 64 elements
    assert ws(3, 6144, 24576, 2458, 8192, bf16) >= 8192 * 2496 * 2


def test_status_strings():
    for s in range(9):
        assert L.espace_status_string(s)
    assert isinstance(_lib.header_functions(), list)


def _ac(X=P16, ldx=64, C=P16b, ldc=64, K=64, N=100, norm=0, alpha=1.0, dt=1,
        ws=ctypes.c_void_p(0x70000000), wsb=1 << 24):
    return L.espace_autocorrelation_update(X, ldx, C, ldc, K, N, norm, alpha, dt, ws, wsb, NULL)


def _pca(C=P16, ldc=64, Pt=P16b, ldp=64, ev=P16c, info=ctypes.c_void_p(0x50000000), K=64, Lc=16, mag=0, dt=1,
         ws=ctypes.c_void_p(0x70000000), wsb=1 << 24):
    return L.espace_principal_components(C, ldc, Pt, ldp, ev, info, K, Lc, mag, dt, ws, wsb, NULL)


def _sym(A=P16, lda=64, B=P16b, ldb=64, C=P16c, ldc=64, K=64, ws=ctypes.c_void_p(0x70000000), wsb=1 << 24):
    return L.espace_symmetrized_product(A, lda, B, ldb, C, ldc, K, 1.0, 0.0, ws, wsb, NULL)


def test_calibration_validation():
    assert _ac(X=NULL) == 1
    assert _ac(C=NULL) == 1
    assert _ac(K=0) == 2
    assert _ac(N=-1) == 2
    assert _ac(ldc=60) == 2                                             # C ld < K
    assert _ac(ldc=66) == 3                                             # C is float32: ld % 4
    assert _ac(ldx=68) == 3                                             # bf16 X: ld % 8
    assert _ac(dt=3) == 4
    assert _ac(C=ctypes.c_void_p(0x10000 + 128)) == 5                   # C inside X
    assert _ac(C=ctypes.c_void_p(0x70000000 + 256)) == 5                # C inside the workspace
    assert _ac(ws=NULL, wsb=0) == 6
    assert _ac(wsb=1024) == 6
    assert _ac(K=1 << 16, ldx=1 << 16, ldc=1 << 16, N=10) == 2          # K·K above 2^31
    assert _ac(N=0, X=NULL, ws=NULL, wsb=0) == 0                        # empty batch: nothing to do
    assert _pca(C=NULL) == 1
    assert _pca(Pt=NULL) == 1
    assert _pca(Lc=0) == 2
    assert _pca(Lc=65) == 2                                             # L > K
    assert _pca(K=40000, ldc=40000, ldp=40000, Lc=10) == 2              # above the solver limit
    assert _pca(ev=ctypes.c_void_p(0x30000002)) == 3
    assert _pca(Pt=ctypes.c_void_p(0x10000 + 64)) == 5                  # Pt inside C
    assert _pca(ev=ctypes.c_void_p(0x70000000)) == 5                    # eigenvalues in the workspace
    assert _pca(ws=NULL, wsb=0) == 6
    assert _sym(A=NULL) == 1
    assert _sym(K=0) == 2
    assert _sym(ldc=62) == 2
    assert _sym(ldb=66) == 3
    assert _sym(C=ctypes.c_void_p(0x20000000 + 64)) == 5                # C inside B
    assert _sym(ws=NULL, wsb=0) == 6
    assert _sym(K=50000, lda=50000, ldb=50000, ldc=50000) == 2
    # every argument valid: the library asks the runtime for the device
    assert _sym() in (7, 8)
    assert _pca(mag=1) in (7, 8)
    assert _ac() in (7, 8)
    assert _pca() in (7, 8)
    assert _pca(ev=NULL, info=NULL) in (7, 8)


def test_calibration_workspace_sizes():
    bf16, f32 = 1, 0
    ws = L.espace_workspace_bytes
    K, N = 4096, 16384
    # transposed tokens K x N (bf16), the inverse norms, fp32 sums of one depth range
    assert ws(5, 0, K, 0, N, bf16) >= K * N * 2 + N * 4 + K * K * 4
    assert ws(5, 0, K, 0, N, f32) >= K * N * 4 + K * K * 4
    assert ws(5, 0, K, 0, 0, bf16) == 0
    assert ws(5, 0, 0, 0, N, bf16) == ctypes.c_size_t(-1).value
    # the eigensolver works on a float64 copy of C
    assert ws(6, 0, K, 1536, 0, bf16) >= K * K * 8 + 2 * K * 8
    assert ws(6, 0, K, K + 1, 0, bf16) == ctypes.c_size_t(-1).value
    assert ws(6, 0, K, 0, 0, bf16) == ctypes.c_size_t(-1).value
    # the symmetrised product keeps one fp32 K x K product
    assert ws(7, 0, K, 0, 0, f32) == K * K * 4
    assert ws(7, 0, 0, 0, 0, f32) == ctypes.c_size_t(-1).value


def _bwd(dY=P16, lddy=32, Z=P16b, ldz=16, Pt=P16c, ldp=64, Wf=ctypes.c_void_p(0x50000000), ldwf=16,
         dX=ctypes.c_void_p(0x60000000), lddx=64, dW=ctypes.c_void_p(0x68000000), lddw=64, M=32, K=64, Lc=16,
         N=8, dt=1, ws=ctypes.c_void_p(0x70000000), wsb=1 << 24):
    return L.espace_projected_linear_backward(dY, lddy, Z, ldz, Pt, ldp, Wf, ldwf, dX, lddx, dW, lddw, M, K, Lc, N,
                                              dt, ws, wsb, NULL)


def test_backward_validation():
    assert _bwd(dY=NULL) == 1
    assert _bwd(Lc=65) == 2
    assert _bwd(lddx=60) == 2
    assert _bwd(dX=ctypes.c_void_p(0x10000 + 32)) == 5                  # dX over dY
    assert _bwd(dW=ctypes.c_void_p(0x60000000 + 64)) == 5               # dW over dX
    assert _bwd(ws=NULL, wsb=0) == 6
    # only what is asked for is checked: dW alone needs no Wf
    assert _bwd(dX=NULL, Wf=NULL) in (7, 8)
    assert _bwd(dW=NULL, Z=NULL) in (7, 8)
    assert _bwd(dX=NULL, dW=NULL, dY=NULL, Z=NULL, Pt=NULL, Wf=NULL, ws=NULL, wsb=0) == 0   # nothing asked
    assert _bwd(N=0, dY=NULL, Z=NULL, dX=NULL, ws=NULL, wsb=0) == 0
    d = L.espace_dense_linear_backward
    assert d(P16, 32, P16b, 64, P16c, 64, ctypes.c_void_p(0x60000000), 64, ctypes.c_void_p(0x68000000), 64,
             32, 64, 8, 1, ctypes.c_void_p(0x70000000), 1 << 24, NULL) in (7, 8)
    assert d(NULL, 32, P16b, 64, P16c, 64, ctypes.c_void_p(0x60000000), 64, NULL, 64,
             32, 64, 8, 1, ctypes.c_void_p(0x70000000), 1 << 24, NULL) == 1
    ws = L.espace_workspace_bytes
    assert ws(8, 12288, 4096, 1536, 4096, 1) > 0
    assert ws(8, 12288, 4096, 5000, 4096, 1) == ctypes.c_size_t(-1).value
    assert ws(9, 12288, 4096, 0, 4096, 1) >= 4096 * 12288 * 2


def test_binding_rejects_mixed_operand_types():
    """The binding checks, before any library call, that every operand, output
    and workspace has the first operand's dtype and device: the library uses
    one element size for all of them, so a float32 input with a bfloat16
    output (or the reverse) would read or write past the smaller buffer."""
    import torch
    f32, bf = torch.float32, torch.bfloat16
    X = torch.zeros(8, 64, dtype=f32)
    Pt = torch.zeros(16, 64, dtype=f32)
    Wf = torch.zeros(32, 16, dtype=f32)
    W = torch.zeros(32, 64, dtype=f32)
    with pytest.raises(TypeError, match="Y"):
        E.espace_projected_linear(X, Pt, Wf, Y=torch.zeros(8, 32, dtype=bf))
    with pytest.raises(TypeError, match="Pt"):
        E.espace_projected_linear(X, Pt.to(bf), Wf)
    with pytest.raises(TypeError, match="Wf"):
        E.espace_projected_linear(X, Pt, Wf.to(bf))
    with pytest.raises(TypeError, match="Pt"):
        E.espace_fold_weights(W, Pt.to(bf))
    with pytest.raises(TypeError, match="Wf"):
        E.espace_fold_weights(W, Pt, Wf=torch.zeros(32, 16, dtype=bf))
    with pytest.raises(TypeError, match="Pt"):
        E.espace_project(Pt.to(bf), X)
    with pytest.raises(TypeError, match="Z"):
        E.espace_project(Pt, X, Z=torch.zeros(8, 16, dtype=bf))
    with pytest.raises(TypeError, match="Wf"):
        E.espace_expand(torch.zeros(8, 16, dtype=f32), Wf.to(bf))
    with pytest.raises(TypeError, match="W"):
        E.espace_dense_linear(X, W.to(bf))
    with pytest.raises(TypeError, match="Y"):
        E.espace_dense_linear(X, W, Y=torch.zeros(8, 32, dtype=bf))
    with pytest.raises(TypeError, match="Wf"):
        E.espace_projected_linear_backward(torch.zeros(8, 32, dtype=f32), torch.zeros(8, 16, dtype=f32), Pt,
                                           Wf.to(bf))
    with pytest.raises(TypeError, match="X"):
        E.espace_dense_linear_backward(torch.zeros(8, 32, dtype=f32), X.to(bf), W)
    with pytest.raises(ValueError, match="B"):
        E.espace_symmetrized_product(torch.zeros(4, 4), torch.zeros(4, 4, dtype=bf))


NOALLOC_MAX = 64 << 20


def test_noalloc_rejects_sizes_beyond_its_scratch():
    """The allocation-free call refuses, before touching any device, sizes
    whose Z and partial sums exceed its static scratch."""
    big_n = 1 << 16
    need = E.espace_workspace_bytes(E.OP_PROJECTED_LINEAR, 4096, 4096, 1536, big_n, __import__("torch").bfloat16)
    assert need > NOALLOC_MAX
    s = L.espace_projected_linear_noalloc(P16, 4096, ctypes.c_void_p(0x100000000000), 4096,
                                          ctypes.c_void_p(0x200000000000), 1536, ctypes.c_void_p(0x300000000000),
                                          4096, 4096, 4096, 1536, big_n, 1, NULL)
    assert s == 6
    assert "scratch" in L.espace_last_error().decode()
    # sizes that fit get past validation and fail only for want of a device
    s = L.espace_projected_linear_noalloc(P16, 64, P16b, 64, P16c, 16, ctypes.c_void_p(0x60000000), 32,
                                          32, 64, 16, 8, 1, NULL)
    assert s in (7, 8)
    assert L.espace_projected_linear_noalloc(NULL, 64, P16b, 64, P16c, 16, ctypes.c_void_p(0x60000000), 32,
                                             32, 64, 16, 8, 1, NULL) == 1


# MX-FP8 operands: codes [rows][ldq] (ldq >= round_up(cols, 128), % 16), scales
# [rows][lds] (lds >= round_up(cols, 128) / 32, % 4)
Q1, S1 = ctypes.c_void_p(0x1000000), ctypes.c_void_p(0x2000000)
Q2, S2 = ctypes.c_void_p(0x3000000), ctypes.c_void_p(0x4000000)
Q3, S3 = ctypes.c_void_p(0x5000000), ctypes.c_void_p(0x6000000)
YM = ctypes.c_void_p(0x7000000)
WSM = ctypes.c_void_p(0x8000000)


def _mxl(Xq=Q1, ldxq=256, Xs=S1, ldxs=8, Pq=Q2, ldpq=256, Ps=S2, ldps=8, Wq=Q3, ldwq=128, Ws=S3, ldws=4,
         Y=YM, ldy=32, M=32, K=200, Lc=100, N=8, ws=WSM, wsb=1 << 20):
    return L.espace_projected_linear_mxfp8(Xq, ldxq, Xs, ldxs, Pq, ldpq, Ps, ldps, Wq, ldwq, Ws, ldws, Y, ldy,
                                           M, K, Lc, N, ws, wsb, NULL)


def _mxq(A=P16, lda=208, R=8, C=200, Q=Q1, ldq=256, S=S1, lds=8):
    return L.espace_quantize_mxfp8(A, lda, R, C, Q, ldq, S, lds, NULL)


def test_mxfp8_validation_errors():
    assert _mxq(A=NULL) == 1
    assert _mxq(S=NULL) == 1
    assert _mxq(C=0) == 2
    assert _mxq(ldq=240) == 2                           # codes below round_up(200, 128)
    assert _mxq(lds=4) == 2                             # scales below 256 / 32
    assert _mxq(ldq=264) == 3                           # codes ld % 16
    assert _mxq(lds=10) == 3                            # scales ld % 4
    assert _mxq(Q=ctypes.c_void_p(0x1000008)) == 3      # codes alignment
    assert _mxq(S=ctypes.c_void_p(0x2000002)) == 3      # scales alignment
    assert _mxq(Q=ctypes.c_void_p(0x10000 + 256)) == 5  # codes over A
    assert _mxq(R=1 << 24, ldq=256) == 2                # codes span 2^32 bytes
    assert _mxl(Lc=201) == 2                            # L > K
    assert _mxl(ldwq=112) == 2                          # Wf codes below round_up(100, 128)
    assert _mxl(ldy=36) == 3                            # Y ld % 8
    assert _mxl(ws=NULL, wsb=0) == 6                    # workspace missing
    assert _mxl(wsb=64) == 6                            # workspace too small
    assert _mxl(Y=ctypes.c_void_p(0x1000000 + 512)) == 5   # Y over X's codes
    assert _mxl(ws=Q2) == 5                             # workspace over Pt's codes
    assert L.espace_workspace_bytes(10, 32, 200, 100, 8, 1) == 1024 + 256   # Z codes 8 x 128, scales 8 x 4
    assert L.espace_workspace_bytes(10, 32, 200, 201, 8, 1) == ctypes.c_size_t(-1).value


def test_mxfp8_empty_and_device():
    assert _mxl(N=0, Xq=NULL, Xs=NULL, Y=NULL, ws=NULL, wsb=0) == 0
    assert _mxq(R=0, A=NULL, Q=NULL, S=NULL) == 0
    assert _mxq() in (7, 8), L.espace_last_error()
    assert _mxl() in (7, 8), L.espace_last_error()
