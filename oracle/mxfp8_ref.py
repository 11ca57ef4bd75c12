"""Plain float64 reference of the projected linear layer on MX-FP8 operands.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper notes that its activation projection can be carried out in low
precision (Section 1.1, related work) and leaves combining ESPACE with
quantisation to future work (Section 5); it fixes no number format.  The
reading implemented here, and by the library's fp8 path:

* Element format: FP8 E4M3 as in the OCP 8-bit floating-point format
  (sign, 4 exponent bits with bias 7, 3 mantissa bits; subnormal spacing
  2^-9 below 2^-6; largest finite magnitude 448; no infinities).
* Block format: OCP Microscaling (MX).  Each run of 32 consecutive values
  along the reduction dimension of an operand shares one power-of-two scale
  2^S, stored as a biased exponent byte S + 127 (E8M0).  S is
  floor(log2(max |v|)) - 8, 8 being the exponent of E4M3's largest binade,
  with the byte clamped to [0, 254]; a block of zeros stores the byte 0.  An
  element is v / 2^S rounded to the nearest E4M3 value, ties to the even
  mantissa, magnitudes above 448 clamped to 448.
* Layer: X (per token, blocks along K), Pt (per component, blocks along K)
  and Wf (per output feature, blocks along L) are MX-FP8 operands.
  Z = X·Ptᵀ is formed exactly from the decoded values, quantised again to
  MX-FP8 (per token, blocks along L), and Y = Z·Wfᵀ is formed exactly from
  the decoded values of the quantised Z and of Wf.  This is Eq. 3 of
  Section 2.2 with every operand of both products in the block format.

Arrays use the storage orientation of espace_ref (X[N][K], Pt[L][K],
Wf[M][L], Z[N][L], Y[N][M]).  Codes are uint8 arrays of the operand's shape
(E4M3 bit patterns); scale bytes are uint8 arrays [rows][ceil(cols / 32)].
"""
import numpy as np

BLOCK = 32
E4M3_MAX = 448.0
E4M3_EMAX = 8          # exponent of the largest E4M3 binade (256 .. 448)
E4M3_MIN_NORMAL_EXP = -6
E4M3_MANT_BITS = 3


def e4m3_round(v):
    """Nearest E4M3 value of each entry (float64 in, float64 out): ties to the
    even mantissa, magnitudes above 448 clamped to 448, signs kept (a value
    that rounds to zero keeps its sign)."""
    v = np.asarray(v, dtype=np.float64)
    a = np.minimum(np.abs(v), E4M3_MAX)
    # spacing of the E4M3 values around a: 2^(e - 3) in the binade
    # [2^e, 2^(e+1)) for e >= -6, 2^-9 below 2^-6 (subnormals)
    _, e = np.frexp(a)                       # a = m * 2^e, m in [0.5, 1)
    e = np.maximum(e - 1, E4M3_MIN_NORMAL_EXP)
    step = np.ldexp(1.0, e - E4M3_MANT_BITS)
    q = np.rint(a / step) * step             # np.rint: round half to even
    q = np.minimum(q, E4M3_MAX)
    return np.copysign(q, v)


def e4m3_decode(codes):
    """float64 values of E4M3 bit patterns (0x7F / 0xFF are NaN)."""
    b = np.asarray(codes, dtype=np.int64)
    sign = np.where(b & 0x80, -1.0, 1.0)
    e = (b >> 3) & 0xF
    m = (b & 0x7).astype(np.float64)
    mag = np.where(e == 0, np.ldexp(m / 8.0, -6), np.ldexp(1.0 + m / 8.0, e - 7))
    mag = np.where((b & 0x7F) == 0x7F, np.nan, mag)
    return sign * mag


def e4m3_encode(values):
    """E4M3 bit patterns of values that lie on the E4M3 grid (as returned by
    e4m3_round); the sign bit follows the sign of the value, zeros included."""
    v = np.asarray(values, dtype=np.float64)
    a = np.abs(v)
    _, e = np.frexp(a)
    e = e - 1
    sub = a < 2.0 ** E4M3_MIN_NORMAL_EXP
    mant_sub = np.rint(a / 2.0 ** -9)
    mant_norm = np.rint((np.ldexp(a, -np.where(sub, 0, e)) - 1.0) * 8.0)
    code = np.where(sub, mant_sub, ((e + 7) << 3) + mant_norm).astype(np.int64)
    code = np.where(np.signbit(v), code | 0x80, code)
    back = e4m3_decode(code)
    if not np.array_equal(np.abs(back), a):
        raise ValueError("e4m3_encode: a value is not on the E4M3 grid")
    return code.astype(np.uint8)


def _blocks(A):
    A = np.asarray(A, dtype=np.float64)
    rows, cols = A.shape
    nb = -(-cols // BLOCK)
    pad = np.zeros((rows, nb * BLOCK))
    pad[:, :cols] = A
    return pad.reshape(rows, nb, BLOCK), cols


def mx_quantize(A):
    """MX-FP8 of a matrix, blocks of 32 along each row.  Returns (values,
    scale_bytes): values are the E4M3 elements as float64 (the decoded codes,
    before the block scale), scale_bytes the E8M0 bytes [rows][blocks]."""
    blk, cols = _blocks(A)
    amax = np.abs(blk).max(axis=2)
    _, e = np.frexp(amax)                    # floor(log2 amax) = e - 1 for amax > 0
    s = (e - 1) - E4M3_EMAX
    byte = np.clip(s + 127, 0, 254)
    byte = np.where(amax == 0, 0, byte)
    scale = np.ldexp(1.0, byte - 127)
    q = e4m3_round(blk / scale[:, :, None])
    rows = blk.shape[0]
    return q.reshape(rows, -1)[:, :cols], byte.astype(np.uint8)


def mx_scale(scale_bytes, cols):
    """Per-element scale 2^(byte - 127) of a [rows][blocks] byte array."""
    s = np.ldexp(1.0, np.asarray(scale_bytes, dtype=np.int64) - 127)
    return np.repeat(s, BLOCK, axis=1)[:, :cols]


def mx_dequantize(values, scale_bytes):
    """Real values of MX-FP8 elements: element times its block's scale."""
    values = np.asarray(values, dtype=np.float64)
    return values * mx_scale(scale_bytes, values.shape[1])


def mx_project(Xq, Xs, Ptq, Pts):
    """Z = X·Ptᵀ from MX-FP8 operands, exact (float64), before re-quantisation
    (Section 2.2, Eq. 3, right factor)."""
    return mx_dequantize(Xq, Xs) @ mx_dequantize(Ptq, Pts).T


def mx_expand(Zq, Zs, Wfq, Wfs):
    """Y = Z·Wfᵀ from MX-FP8 operands, exact (float64) (Section 2.2, Eq. 3)."""
    return mx_dequantize(Zq, Zs) @ mx_dequantize(Wfq, Wfs).T


def mx_projected_linear(Xq, Xs, Ptq, Pts, Wfq, Wfs):
    """The layer on MX-FP8 operands: Z = X·Ptᵀ, Z quantised to MX-FP8 along L,
    then Y = Z·Wfᵀ.  Returns (Y, Zq, Zs)."""
    Z = mx_project(Xq, Xs, Ptq, Pts)
    Zq, Zs = mx_quantize(Z)
    return mx_expand(Zq, Zs, Wfq, Wfs), Zq, Zs
