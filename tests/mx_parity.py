"""Parity criteria of the MX-FP8 path (element-wise, against the oracle).

Accumulation model.  The products run on gfx950's block-scaled MFMAs, each
instruction adding its block-scaled dot product to the running fp32 sum C:
the projection on v_mfma_scale_f32_16x16x128_f8f6f4 (one instruction per
128 of depth), the expansion on v_mfma_scale_f32_32x32x64_f8f6f4 (one per
64).  Measured on the hardware, one instruction's result differs from the
exact C + sum(a·b) by at most 2^-11.6 of sum|a·b| (C = 0) and 2^-12.2 of
|C| + sum|a·b| (C != 0) for the 16x16x128 form (600 + 600 random trials),
and by at most 2^-11.55 of |C| + sum|a·b| for the 32x32x64 form (1200
trials, |C| from 0 to 1e3 times the products' magnitude): the instruction
rounds inside.  The bound here takes eps = 2^-10 per instruction, so after
instruction t of a product

    |computed - exact| <= eps · sum_{s<=t} (|P_{s-1}| + S_s)

with P_s the exact partial sum after instruction s and S_s = sum over its
depth of |a·b| (block scales applied), both evaluated by the oracle side in
float64; `step` is the depth of one instruction.

Z's re-quantisation.  The projection quantises its fp32 Z; the oracle's
exact Z may sit on the other side of a rounding boundary.  A GPU scale byte
is valid when it is the byte of some block maximum within the bound of the
exact one, and a GPU code is valid when it is the E4M3 rounding of some value
within the bound of the exact entry (rounding is monotone, so the two ends of
the interval give the range of valid codes).
"""
import numpy as np
import torch

import oracle

EPS_MFMA = 2.0 ** -10
STEP_PROJECT = 128    # depth of one MFMA of the projection (16x16x128)
STEP_EXPAND = 64      # of the expansion (32x32x64)
U_BF16 = 2.0 ** -8


def e4m3_table():
    """float64 value of each E4M3 byte, from torch's float8_e4m3fn."""
    return torch.arange(256, dtype=torch.int32).to(torch.uint8).view(torch.float8_e4m3fn).to(
        torch.float64).numpy()


_TABLE = None


def gpu_mx(m, rows=None):
    """(element values, scale bytes) of an MXTensor's logical part, as float64
    and int64 arrays; `rows` selects token rows."""
    global _TABLE
    if _TABLE is None:
        _TABLE = e4m3_table()
    nb = -(-m.cols // 32)
    codes = m.codes.cpu().numpy()
    scales = m.scales.cpu().numpy()
    if rows is not None:
        codes, scales = codes[rows], scales[rows]
    return _TABLE[codes[:, :m.cols]], scales[:, :nb].astype(np.int64), codes, scales


def chain_bound(A, B, step):
    """(exact product A·Bᵀ, element bound of the MFMA chain) for real-valued
    operands A [R][D], B [C][D] (block scales applied), one instruction per
    `step` of depth."""
    R, D = A.shape
    P = np.zeros((R, B.shape[0]))
    E = np.zeros_like(P)
    for t0 in range(0, D, step):
        At, Bt = A[:, t0:t0 + step], B[:, t0:t0 + step]
        S = np.abs(At) @ np.abs(Bt).T
        E += EPS_MFMA * (np.abs(P) + S)
        P += At @ Bt.T
    return P, E


def _scale_byte(amax):
    """E8M0 byte of blocks with largest magnitudes amax (oracle's rule)."""
    _, e = np.frexp(amax)
    b = np.clip((e - 1) - 8 + 127, 0, 254)
    return np.where(amax > 0, b, 0)


def check_mx_codes(Z, E, vals, sbytes, what):
    """Every GPU scale byte and code of Z [R][C] valid for some Z' with
    |Z' - Z| <= E.  Returns the fraction of entries whose code equals the
    oracle's own quantisation of Z."""
    R, C = Z.shape
    nb = -(-C // 32)
    pad = nb * 32
    Zp = np.zeros((R, pad))
    Ep = np.zeros((R, pad))
    Zp[:, :C], Ep[:, :C] = Z, E
    lo_amax = np.maximum(np.abs(Zp) - Ep, 0).reshape(R, nb, 32).max(axis=2)
    hi_amax = (np.abs(Zp) + Ep).reshape(R, nb, 32).max(axis=2)
    blo, bhi = _scale_byte(lo_amax), _scale_byte(hi_amax)
    bad = np.argwhere((sbytes < blo) | (sbytes > bhi))
    if len(bad):
        r, b = bad[0]
        raise AssertionError(f"{what}: {len(bad)} scale bytes outside the valid range, first ({r}, {b}): "
                             f"{sbytes[r, b]} not in [{blo[r, b]}, {bhi[r, b]}]")
    s = np.repeat(np.ldexp(1.0, sbytes - 127), 32, axis=1)[:, :C]
    lo = oracle.e4m3_round((Z - E) / s)
    hi = oracle.e4m3_round((Z + E) / s)
    bad = np.argwhere((vals < lo) | (vals > hi) | ~np.isfinite(vals))
    if len(bad):
        r, c = bad[0]
        raise AssertionError(f"{what}: {len(bad)} codes outside the valid range, first ({r}, {c}): "
                             f"{vals[r, c]} not in [{lo[r, c]}, {hi[r, c]}] (Z {Z[r, c]!r}, bound {E[r, c]!r})")
    oq, ob = oracle.mx_quantize(Z)
    return float(np.mean((oq == vals) & (np.repeat(ob, 32, axis=1)[:, :C] == np.repeat(sbytes, 32, axis=1)[:, :C])))


def z_value_width(Z, E, sbytes_lo_hi=None):
    """Largest spread of the real value (code times scale) a valid GPU
    quantisation of each Z entry can take: the distance between the extreme
    valid values over the valid scale bytes of its block."""
    R, C = Z.shape
    nb = -(-C // 32)
    pad = nb * 32
    Zp = np.zeros((R, pad))
    Ep = np.zeros((R, pad))
    Zp[:, :C], Ep[:, :C] = Z, E
    blo = _scale_byte(np.maximum(np.abs(Zp) - Ep, 0).reshape(R, nb, 32).max(axis=2))
    bhi = _scale_byte((np.abs(Zp) + Ep).reshape(R, nb, 32).max(axis=2))
    vmin = np.full((R, C), np.inf)
    vmax = np.full((R, C), -np.inf)
    for db in range(0, int((bhi - blo).max()) + 1):
        b = np.minimum(blo + db, bhi)
        s = np.repeat(np.ldexp(1.0, b - 127), 32, axis=1)[:, :C]
        lo = oracle.e4m3_round((Z - E) / s) * s
        hi = oracle.e4m3_round((Z + E) / s) * s
        vmin, vmax = np.minimum(vmin, lo), np.maximum(vmax, hi)
    oz, os_ = oracle.mx_quantize(Z)
    ov = oracle.mx_dequantize(oz, os_)
    return np.maximum(vmax - ov, ov - vmin)


def check_bound(got, ref, bound, what):
    """|got - ref| <= bound everywhere, outputs finite; returns the largest
    ratio of error to bound and the relative Frobenius error."""
    got = np.asarray(got, dtype=np.float64)
    if not np.isfinite(got).all():
        bad = np.argwhere(~np.isfinite(got))
        raise AssertionError(f"{what}: {len(bad)} non-finite entries, first at {bad[0].tolist()}")
    err = np.abs(got - ref)
    over = err > bound
    if over.any():
        r, c = np.argwhere(over)[0]
        raise AssertionError(f"{what}: {int(over.sum())} entries outside the bound, first ({r}, {c}): "
                             f"got {got[r, c]!r}, oracle {ref[r, c]!r}, bound {bound[r, c]!r}")
    rel = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))
    assert rel <= 1e-2, f"{what}: relative Frobenius error {rel:.3e}"
    return float((err / np.maximum(bound, 1e-300)).max()), rel
