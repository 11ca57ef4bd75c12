"""ctypes binding of libespace.so (argument marshalling only).

Every computation runs in the library's HIP kernels; this module only turns
torch tensors into (device pointer, leading dimension) pairs, allocates
outputs and workspaces with torch, passes torch's current HIP stream, and
raises EspaceError on a non-OK status.  It has no fallback: if the library is
missing, importing the package fails.
"""
import ctypes
import os
import re

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libespace.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "espace.h")

F32 = 0
BF16 = 1
(OP_FOLD, OP_PROJECT, OP_EXPAND, OP_PROJECTED_LINEAR, OP_DENSE, OP_AUTOCORR, OP_PCA, OP_SYMPRODUCT, OP_BACKWARD,
 OP_DENSE_BACKWARD, OP_PROJECTED_LINEAR_MXFP8) = range(11)

_c_i64 = ctypes.c_int64
_c_p = ctypes.c_void_p
_c_sz = ctypes.c_size_t
_c_int = ctypes.c_int

_SIGS = {
    # name: (argtypes, restype)
    "espace_fold_weights": ([_c_p, _c_i64, _c_p, _c_i64, _c_p, _c_i64, _c_i64, _c_i64, _c_i64,
                             _c_int, _c_p, _c_sz, _c_p], _c_int),
    "espace_project": ([_c_p, _c_i64, _c_p, _c_i64, _c_p, _c_i64, _c_i64, _c_i64, _c_i64,
                        _c_int, _c_p, _c_sz, _c_p], _c_int),
    "espace_expand": ([_c_p, _c_i64, _c_p, _c_i64, _c_p, _c_i64, _c_i64, _c_i64, _c_i64,
                       _c_int, _c_p, _c_sz, _c_p], _c_int),
    "espace_projected_linear": ([_c_p, _c_i64, _c_p, _c_i64, _c_p, _c_i64, _c_p, _c_i64,
                                 _c_i64, _c_i64, _c_i64, _c_i64, _c_int, _c_p, _c_sz, _c_p], _c_int),
    "espace_projected_linear_noalloc": ([_c_p, _c_i64, _c_p, _c_i64, _c_p, _c_i64, _c_p, _c_i64,
                                         _c_i64, _c_i64, _c_i64, _c_i64, _c_int, _c_p], _c_int),
    "espace_dense_linear": ([_c_p, _c_i64, _c_p, _c_i64, _c_p, _c_i64, _c_i64, _c_i64, _c_i64,
                             _c_int, _c_p, _c_sz, _c_p], _c_int),
    "espace_autocorrelation_update": ([_c_p, _c_i64, _c_p, _c_i64, _c_i64, _c_i64, _c_int, ctypes.c_float,
                                       _c_int, _c_p, _c_sz, _c_p], _c_int),
    "espace_principal_components": ([_c_p, _c_i64, _c_p, _c_i64, _c_p, _c_p, _c_i64, _c_i64, _c_int, _c_int,
                                     _c_p, _c_sz, _c_p], _c_int),
    "espace_symmetrized_product": ([_c_p, _c_i64, _c_p, _c_i64, _c_p, _c_i64, _c_i64, ctypes.c_float,
                                    ctypes.c_float, _c_p, _c_sz, _c_p], _c_int),
    "espace_projected_linear_backward": ([_c_p, _c_i64] * 6 + [_c_i64] * 4 + [_c_int, _c_p, _c_sz, _c_p], _c_int),
    "espace_dense_linear_backward": ([_c_p, _c_i64] * 5 + [_c_i64] * 3 + [_c_int, _c_p, _c_sz, _c_p], _c_int),
    "espace_workspace_bytes": ([_c_int, _c_i64, _c_i64, _c_i64, _c_i64, _c_int], _c_sz),
    "espace_quantize_mxfp8": ([_c_p, _c_i64, _c_i64, _c_i64, _c_p, _c_i64, _c_p, _c_i64, _c_p], _c_int),
    "espace_project_mxfp8": ([_c_p, _c_i64] * 6 + [_c_i64] * 3 + [_c_p], _c_int),
    "espace_expand_mxfp8": ([_c_p, _c_i64] * 5 + [_c_i64] * 3 + [_c_p], _c_int),
    "espace_projected_linear_mxfp8": ([_c_p, _c_i64] * 7 + [_c_i64] * 4 + [_c_p, _c_sz, _c_p], _c_int),
    "espace_status_string": ([_c_int], ctypes.c_char_p),
    "espace_last_error": ([], ctypes.c_char_p),
    "espace_abi_version": ([], _c_int),
    "espace_wait_timeouts": ([ctypes.POINTER(ctypes.c_ulonglong)], _c_int),
    "espace_set_wait_limit": ([ctypes.c_uint], _c_int),
}


class EspaceError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"espace status {status}: {message}")
        self.status = status
        self.message = message


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built (python paper_2410_05437_amd/build.py)")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (args, res) in _SIGS.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


lib = _load()
ABI_VERSION = lib.espace_abi_version()


def header_functions():
    """Names of the functions include/espace.h declares."""
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\**\s+\**(espace_\w+)\s*\(", text, re.M)))


def _check(status):
    if status != 0:
        msg = lib.espace_last_error().decode()
        raise EspaceError(status, msg or lib.espace_status_string(status).decode())


def espace_wait_timeouts():
    """Count of bounded in-kernel waits that gave up on the current device
    (synchronous read; synchronise the streams first)."""
    n = ctypes.c_ulonglong(0)
    _check(lib.espace_wait_timeouts(ctypes.byref(n)))
    return int(n.value)


def espace_set_wait_limit(spins):
    """Polls after which an in-kernel wait gives up (0: the default)."""
    _check(lib.espace_set_wait_limit(int(spins)))


def _dt(t):
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _mat(t, name):
    """(pointer, leading dimension) of a row-major 2-D tensor whose storage
    holds rows*ld elements (the library may read the padding of the last row)."""
    if t.dim() != 2:
        raise ValueError(f"{name} must be 2-D")
    if t.stride(1) != 1 and t.shape[1] > 1:
        raise ValueError(f"{name} must have unit column stride")
    ld = t.stride(0) if t.shape[0] > 1 else max(t.stride(0), t.shape[1])
    need = (t.storage_offset() + t.shape[0] * ld) * t.element_size()
    if t.numel() and t.untyped_storage().nbytes() < need:
        raise ValueError(f"{name}: storage must hold rows*ld elements (use padded_empty)")
    return ctypes.c_void_p(t.data_ptr()), ld


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def padded_empty(rows, cols, dtype, device, align=8):
    """Uninitialised rows x cols tensor with a leading dimension rounded up to
    `align` elements (its storage holds rows*ld elements)."""
    ld = max((cols + align - 1) // align * align, align)
    return torch.empty((rows, ld), dtype=dtype, device=device)[:, :cols]


def _same(first, fname, *others):
    """Every (tensor, name) in `others` has the dtype and device of `first`: the
    library reads and writes every operand with one element size, so a mixed
    call would index outside the smaller buffers."""
    for t, name in others:
        if t is None:
            continue
        if t.dtype != first.dtype:
            raise TypeError(f"{name} is {t.dtype}, {fname} is {first.dtype}: operands and outputs must share one dtype")
        if t.device != first.device:
            raise ValueError(f"{name} is on {t.device}, {fname} on {first.device}")


def _out(out, rows, cols, like, name):
    if out is None:
        return padded_empty(rows, cols, like.dtype, like.device, 8 if like.dtype == torch.bfloat16 else 4)
    if tuple(out.shape) != (rows, cols):
        raise ValueError(f"{name} must be {rows}x{cols}")
    _same(like, "the input", (out, name))
    return out


def espace_workspace_bytes(op, M, K, L, N, dtype):
    dt = BF16 if dtype == torch.bfloat16 else F32
    n = lib.espace_workspace_bytes(op, M, K, L, N, dt)
    if n == ctypes.c_size_t(-1).value:
        raise EspaceError(2, "invalid sizes for workspace query")
    return n


def _ws(workspace, nbytes, device):
    if nbytes == 0:
        return None, 0
    if workspace is None:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
    if workspace.device != device:
        raise ValueError(f"workspace is on {workspace.device}, the operands on {device}")
    if not workspace.is_contiguous():
        raise ValueError("workspace must be contiguous")
    return workspace, workspace.numel() * workspace.element_size()


def espace_fold_weights(W, Pt, Wf=None, workspace=None):
    """Wf = W·P  (W [M][K], Pt [L][K] -> Wf [M][L])."""
    M, K = W.shape
    L = Pt.shape[0]
    _same(W, "W", (Pt, "Pt"))
    Wf = _out(Wf, M, L, W, "Wf")
    ws, wsb = _ws(workspace, espace_workspace_bytes(OP_FOLD, M, K, L, 0, W.dtype), W.device)
    pw, ldw = _mat(W, "W")
    pp, ldp = _mat(Pt, "Pt")
    po, ldo = _mat(Wf, "Wf")
    with torch.cuda.device(W.device):
        _check(lib.espace_fold_weights(pw, ldw, pp, ldp, po, ldo, M, K, L, _dt(W),
                                       ctypes.c_void_p(ws.data_ptr() if ws is not None else 0),
                                       wsb, _stream(W.device)))
    return Wf


def espace_project(Pt, X, Z=None, workspace=None):
    """Z = Pᵀ·X  (Pt [L][K], X [N][K] -> Z [N][L])."""
    L, K = Pt.shape
    N = X.shape[0]
    _same(X, "X", (Pt, "Pt"))
    Z = _out(Z, N, L, X, "Z")
    ws, wsb = _ws(workspace, espace_workspace_bytes(OP_PROJECT, 0, K, L, N, X.dtype), X.device)
    pp, ldp = _mat(Pt, "Pt")
    px, ldx = _mat(X, "X")
    pz, ldz = _mat(Z, "Z")
    with torch.cuda.device(X.device):
        _check(lib.espace_project(pp, ldp, px, ldx, pz, ldz, K, L, N, _dt(X),
                                  ctypes.c_void_p(ws.data_ptr() if ws is not None else 0),
                                  wsb, _stream(X.device)))
    return Z


def espace_expand(Z, Wf, Y=None, workspace=None):
    """Y = Wf·Z  (Z [N][L], Wf [M][L] -> Y [N][M])."""
    N, L = Z.shape
    M = Wf.shape[0]
    _same(Z, "Z", (Wf, "Wf"))
    Y = _out(Y, N, M, Z, "Y")
    ws, wsb = _ws(workspace, espace_workspace_bytes(OP_EXPAND, M, L, L, N, Z.dtype), Z.device)
    pz, ldz = _mat(Z, "Z")
    pw, ldw = _mat(Wf, "Wf")
    py, ldy = _mat(Y, "Y")
    with torch.cuda.device(Z.device):
        _check(lib.espace_expand(pz, ldz, pw, ldw, py, ldy, M, L, N, _dt(Z),
                                 ctypes.c_void_p(ws.data_ptr() if ws is not None else 0),
                                 wsb, _stream(Z.device)))
    return Y


def espace_projected_linear(X, Pt, Wf, Y=None, workspace=None):
    """Y = Wf·(Pᵀ·X)  (X [N][K], Pt [L][K], Wf [M][L] -> Y [N][M])."""
    N, K = X.shape
    L = Pt.shape[0]
    M = Wf.shape[0]
    _same(X, "X", (Pt, "Pt"), (Wf, "Wf"))
    Y = _out(Y, N, M, X, "Y")
    ws, wsb = _ws(workspace, espace_workspace_bytes(OP_PROJECTED_LINEAR, M, K, L, N, X.dtype), X.device)
    px, ldx = _mat(X, "X")
    pp, ldp = _mat(Pt, "Pt")
    pw, ldw = _mat(Wf, "Wf")
    py, ldy = _mat(Y, "Y")
    with torch.cuda.device(X.device):
        _check(lib.espace_projected_linear(px, ldx, pp, ldp, pw, ldw, py, ldy, M, K, L, N, _dt(X),
                                           ctypes.c_void_p(ws.data_ptr() if ws is not None else 0),
                                           wsb, _stream(X.device)))
    return Y


def espace_projected_linear_noalloc(X, Pt, Wf, Y):
    """Y = Wf·(Pᵀ·X) into a caller-provided Y, with the library's static device
    scratch in place of a workspace (the C call allocates nothing)."""
    N, K = X.shape
    L = Pt.shape[0]
    M = Wf.shape[0]
    _same(X, "X", (Pt, "Pt"), (Wf, "Wf"))
    Y = _out(Y, N, M, X, "Y")
    px, ldx = _mat(X, "X")
    pp, ldp = _mat(Pt, "Pt")
    pw, ldw = _mat(Wf, "Wf")
    py, ldy = _mat(Y, "Y")
    with torch.cuda.device(X.device):
        _check(lib.espace_projected_linear_noalloc(px, ldx, pp, ldp, pw, ldw, py, ldy, M, K, L, N, _dt(X),
                                                   _stream(X.device)))
    return Y


def espace_dense_linear(X, W, Y=None, workspace=None):
    """Y = W·X  (X [N][K], W [M][K] -> Y [N][M])."""
    N, K = X.shape
    M = W.shape[0]
    _same(X, "X", (W, "W"))
    Y = _out(Y, N, M, X, "Y")
    ws, wsb = _ws(workspace, espace_workspace_bytes(OP_DENSE, M, K, 1, N, X.dtype), X.device)
    px, ldx = _mat(X, "X")
    pw, ldw = _mat(W, "W")
    py, ldy = _mat(Y, "Y")
    with torch.cuda.device(X.device):
        _check(lib.espace_dense_linear(px, ldx, pw, ldw, py, ldy, M, K, N, _dt(X),
                                       ctypes.c_void_p(ws.data_ptr() if ws is not None else 0),
                                       wsb, _stream(X.device)))
    return Y


def espace_autocorrelation_update(X, C, alpha, normalize=False, workspace=None):
    """C += alpha · Σ_n x̂_n x̂_nᵀ over the tokens (rows) of X [N][K]; x̂_n = x_n,
    or x_n/||x_n|| with `normalize` (Section 3.1, Eq. 5; Corollary 1).  C is a
    float32 [K][K] tensor updated in place."""
    N, K = X.shape
    if C.dtype != torch.float32 or tuple(C.shape) != (K, K):
        raise ValueError(f"C must be a float32 {K}x{K} tensor")
    if C.device != X.device:
        raise ValueError(f"C is on {C.device}, X on {X.device}")
    ws, wsb = _ws(workspace, espace_workspace_bytes(OP_AUTOCORR, 0, K, 0, N, X.dtype), X.device)
    px, ldx = _mat(X, "X")
    pc, ldc = _mat(C, "C")
    with torch.cuda.device(X.device):
        _check(lib.espace_autocorrelation_update(px, ldx, pc, ldc, K, N, 1 if normalize else 0, float(alpha),
                                                 _dt(X), ctypes.c_void_p(ws.data_ptr() if ws is not None else 0),
                                                 wsb, _stream(X.device)))
    return C


def espace_symmetrized_product(A, B, C=None, workspace=None, alpha=1.0, beta=0.0):
    """C = beta·C + alpha·(A·Bᵀ + B·Aᵀ) for float32 [K][K] A and B: with the
    autocorrelations C_X and C_W, Theorem 2's GO-MSE matrix C_X·C_W +
    C_W·C_X; accumulated over calibration sequences (beta = 1) with the
    gradients' autocorrelation in place of C_W, its NL-MSE matrix."""
    K = A.shape[0]
    for t, n in ((A, "A"), (B, "B")):
        if t.dtype != torch.float32 or tuple(t.shape) != (K, K):
            raise ValueError(f"{n} must be a float32 {K}x{K} tensor")
    _same(A, "A", (B, "B"), (C, "C"))
    if C is None:
        if beta != 0.0:
            raise ValueError("beta != 0 needs C")
        C = padded_empty(K, K, torch.float32, A.device, 4)
    elif C.dtype != torch.float32 or tuple(C.shape) != (K, K):
        raise ValueError(f"C must be a float32 {K}x{K} tensor")
    ws, wsb = _ws(workspace, espace_workspace_bytes(OP_SYMPRODUCT, 0, K, 0, 0, torch.float32), A.device)
    pa, lda = _mat(A, "A")
    pb, ldb = _mat(B, "B")
    pc, ldc = _mat(C, "C")
    with torch.cuda.device(A.device):
        _check(lib.espace_symmetrized_product(pa, lda, pb, ldb, pc, ldc, K, float(alpha), float(beta),
                                              ctypes.c_void_p(ws.data_ptr() if ws is not None else 0), wsb,
                                              _stream(A.device)))
    return C


def espace_principal_components(C, L, dtype=torch.bfloat16, Pt=None, eigenvalues=None, info=None,
                                workspace=None, by_magnitude=False):
    """Pt [L][K]: the eigenvectors of the L largest eigenvalues of the
    symmetric float32 C [K][K] (Theorem 1) — largest in absolute value with
    `by_magnitude` (Theorem 2) — each signed so that its entry of largest
    magnitude is positive.  Returns (Pt, eigenvalues [K] in the selection
    order, info: a one-element int32 tensor, 0 on success)."""
    K = C.shape[0]
    if C.dtype != torch.float32 or tuple(C.shape) != (K, K):
        raise ValueError("C must be a square float32 tensor")
    if Pt is None:
        Pt = padded_empty(L, K, dtype, C.device, 8 if dtype == torch.bfloat16 else 4)
    if tuple(Pt.shape) != (L, K):
        raise ValueError(f"Pt must be {L}x{K}")
    if Pt.device != C.device:
        raise ValueError(f"Pt is on {Pt.device}, C on {C.device}")
    for t, n, dt, size in ((eigenvalues, "eigenvalues", torch.float32, K), (info, "info", torch.int32, 1)):
        if t is not None and (t.dtype != dt or t.device != C.device or t.numel() < size or not t.is_contiguous()):
            raise ValueError(f"{n} must be a contiguous {dt} tensor of {size} elements on {C.device}")
    if eigenvalues is None:
        eigenvalues = torch.empty(K, dtype=torch.float32, device=C.device)
    if info is None:
        info = torch.zeros(1, dtype=torch.int32, device=C.device)
    ws, wsb = _ws(workspace, espace_workspace_bytes(OP_PCA, 0, K, L, 0, Pt.dtype), C.device)
    pc, ldc = _mat(C, "C")
    pp, ldp = _mat(Pt, "Pt")
    with torch.cuda.device(C.device):
        _check(lib.espace_principal_components(pc, ldc, pp, ldp, ctypes.c_void_p(eigenvalues.data_ptr()),
                                               ctypes.c_void_p(info.data_ptr()), K, L, 1 if by_magnitude else 0,
                                               _dt(Pt),
                                               ctypes.c_void_p(ws.data_ptr() if ws is not None else 0), wsb,
                                               _stream(C.device)))
    return Pt, eigenvalues, info


def _opt_out(t, rows, cols, like, name, want):
    if not want:
        return None, ctypes.c_void_p(0), 0
    t = _out(t, rows, cols, like, name)
    p, ld = _mat(t, name)
    return t, p, ld


def espace_projected_linear_backward(dY, Z, Pt, Wf, dX=None, dW=None, want_dx=True, want_dw=True,
                                     workspace=None):
    """Gradients of the training view Y = W·(P·Pᵀ·X) (Section 2.2) for an
    upstream gradient dY [N][M]: dX = (dY·Wf)·Pt [N][K] and dW = (dYᵀ·Z)·Pt
    [M][K], from the forward pass's Z = Pᵀ·X [N][L] and Wf = W·P [M][L].
    Returns (dX, dW); either is None when not wanted."""
    N, M = dY.shape
    L, K = Pt.shape
    _same(dY, "dY", (Z, "Z"), (Pt, "Pt"), (Wf, "Wf"))
    dX, pdx, lddx = _opt_out(dX, N, K, dY, "dX", want_dx)
    dW, pdw, lddw = _opt_out(dW, M, K, dY, "dW", want_dw)
    ws, wsb = _ws(workspace, espace_workspace_bytes(OP_BACKWARD, M, K, L, N, dY.dtype), dY.device)
    pdy, lddy = _mat(dY, "dY")
    pz, ldz = _mat(Z, "Z")
    pp, ldp = _mat(Pt, "Pt")
    pw, ldw = _mat(Wf, "Wf")
    with torch.cuda.device(dY.device):
        _check(lib.espace_projected_linear_backward(pdy, lddy, pz, ldz, pp, ldp, pw, ldw, pdx, lddx, pdw, lddw,
                                                    M, K, L, N, _dt(dY),
                                                    ctypes.c_void_p(ws.data_ptr() if ws is not None else 0), wsb,
                                                    _stream(dY.device)))
    return dX, dW


def espace_dense_linear_backward(dY, X, W, dX=None, dW=None, want_dx=True, want_dw=True, workspace=None):
    """Gradients of the dense layer Y = W·X: dX = dY·W [N][K], dW = dYᵀ·X
    [M][K].  Returns (dX, dW); either is None when not wanted."""
    N, M = dY.shape
    K = W.shape[1]
    _same(dY, "dY", (X, "X"), (W, "W"))
    dX, pdx, lddx = _opt_out(dX, N, K, dY, "dX", want_dx)
    dW, pdw, lddw = _opt_out(dW, M, K, dY, "dW", want_dw)
    ws, wsb = _ws(workspace, espace_workspace_bytes(OP_DENSE_BACKWARD, M, K, 1, N, dY.dtype), dY.device)
    pdy, lddy = _mat(dY, "dY")
    px, ldx = _mat(X, "X")
    pw, ldw = _mat(W, "W")
    with torch.cuda.device(dY.device):
        _check(lib.espace_dense_linear_backward(pdy, lddy, px, ldx, pw, ldw, pdx, lddx, pdw, lddw, M, K, N,
                                                _dt(dY), ctypes.c_void_p(ws.data_ptr() if ws is not None else 0),
                                                wsb, _stream(dY.device)))
    return dX, dW


# ---- MX-FP8 ------------------------------------------------------------------

class MXTensor:
    """An MX-FP8 matrix of `rows` x `cols`: E4M3 codes [rows][ldq] (uint8,
    ldq >= round_up(cols, 128); the columns past `cols` hold zeros) and E8M0
    scale bytes [rows][lds] (byte b scales columns 32b .. 32b + 31)."""

    def __init__(self, codes, scales, cols):
        self.codes = codes
        self.scales = scales
        self.cols = int(cols)

    @property
    def rows(self):
        return self.codes.shape[0]

    @property
    def device(self):
        return self.codes.device


def mx_empty(rows, cols, device):
    """Uninitialised MX-FP8 matrix: codes at the smallest leading dimension,
    scale rows padded to 16 bytes (the layout the kernels load fastest)."""
    cp = (cols + 127) // 128 * 128
    lds = (cp // 32 + 15) // 16 * 16
    return MXTensor(torch.empty((rows, cp), dtype=torch.uint8, device=device),
                    torch.empty((rows, lds), dtype=torch.uint8, device=device)[:, :cp // 32], cols)


def _mx(m, name, rows=None, cols=None):
    """(codes pointer, ldq, scales pointer, lds) of an MXTensor."""
    if not isinstance(m, MXTensor):
        raise TypeError(f"{name} must be an MXTensor")
    for t, what in ((m.codes, "codes"), (m.scales, "scales")):
        if t.dtype != torch.uint8 or t.dim() != 2 or (t.stride(1) != 1 and t.shape[1] > 1):
            raise ValueError(f"{name} {what}: a 2-D uint8 tensor with unit column stride")
    if m.scales.shape[0] != m.rows or m.scales.device != m.device:
        raise ValueError(f"{name}: codes and scales must share rows and device")
    if rows is not None and m.rows != rows:
        raise ValueError(f"{name} has {m.rows} rows, expected {rows}")
    if cols is not None and m.cols != cols:
        raise ValueError(f"{name} has {m.cols} columns, expected {cols}")
    pq, ldq = _mat(m.codes, name + " codes")
    ps, lds = _mat(m.scales, name + " scales")
    return pq, ldq, ps, lds


def espace_quantize_mxfp8(A, out=None):
    """MX-FP8 of a bfloat16 matrix A [R][C] along its rows -> MXTensor."""
    if A.dtype != torch.bfloat16:
        raise TypeError("A must be bfloat16")
    R, C = A.shape
    out = mx_empty(R, C, A.device) if out is None else out
    pq, ldq, ps, lds = _mx(out, "out", R, C)
    if out.device != A.device:
        raise ValueError("out and A must share a device")
    pa, lda = _mat(A, "A")
    with torch.cuda.device(A.device):
        _check(lib.espace_quantize_mxfp8(pa, lda, R, C, pq, ldq, ps, lds, _stream(A.device)))
    return out


def espace_project_mxfp8(Pt, X, Z=None):
    """Z = Pᵀ·X from MX-FP8 Pt [L][K] and X [N][K] -> MX-FP8 Z [N][L]."""
    L, K, N = Pt.rows, Pt.cols, X.rows
    Z = mx_empty(N, L, X.device) if Z is None else Z
    a = _mx(Pt, "Pt")
    b = _mx(X, "X", cols=K)
    c = _mx(Z, "Z", N, L)
    if len({Pt.device, X.device, Z.device}) != 1:
        raise ValueError("operands must share a device")
    with torch.cuda.device(X.device):
        _check(lib.espace_project_mxfp8(*a, *b, *c, K, L, N, _stream(X.device)))
    return Z


def espace_expand_mxfp8(Z, Wf, Y=None):
    """Y = Wf·Z from MX-FP8 Z [N][L] and Wf [M][L] -> bfloat16 Y [N][M]."""
    N, L, M = Z.rows, Z.cols, Wf.rows
    a = _mx(Z, "Z")
    b = _mx(Wf, "Wf", cols=L)
    if Y is None:
        Y = padded_empty(N, M, torch.bfloat16, Z.device)
    if tuple(Y.shape) != (N, M) or Y.dtype != torch.bfloat16 or Y.device != Z.device:
        raise ValueError(f"Y must be a bfloat16 {N}x{M} tensor on {Z.device}")
    if Wf.device != Z.device:
        raise ValueError("operands must share a device")
    py, ldy = _mat(Y, "Y")
    with torch.cuda.device(Z.device):
        _check(lib.espace_expand_mxfp8(*a, *b, py, ldy, M, L, N, _stream(Z.device)))
    return Y


def espace_projected_linear_mxfp8(X, Pt, Wf, Y=None, workspace=None):
    """Y = Wf·(Pᵀ·X) from MX-FP8 X [N][K], Pt [L][K], Wf [M][L] -> bfloat16
    Y [N][M], Z in MX-FP8 in the workspace."""
    N, K, L, M = X.rows, X.cols, Pt.rows, Wf.rows
    a = _mx(X, "X")
    b = _mx(Pt, "Pt", cols=K)
    c = _mx(Wf, "Wf", cols=L)
    if len({X.device, Pt.device, Wf.device}) != 1:
        raise ValueError("operands must share a device")
    if Y is None:
        Y = padded_empty(N, M, torch.bfloat16, X.device)
    if tuple(Y.shape) != (N, M) or Y.dtype != torch.bfloat16 or Y.device != X.device:
        raise ValueError(f"Y must be a bfloat16 {N}x{M} tensor on {X.device}")
    ws, wsb = _ws(workspace, espace_workspace_bytes(OP_PROJECTED_LINEAR_MXFP8, M, K, L, N, torch.bfloat16),
                  X.device)
    py, ldy = _mat(Y, "Y")
    with torch.cuda.device(X.device):
        _check(lib.espace_projected_linear_mxfp8(*a, *b, *c, py, ldy, M, K, L, N,
                                                 ctypes.c_void_p(ws.data_ptr() if ws is not None else 0), wsb,
                                                 _stream(X.device)))
    return Y
