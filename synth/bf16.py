"""Bit-exact bfloat16 encoding of float64 arrays (round to nearest, ties to even).

Inputs are generated in float64 and rounded once to the storage type; both the
GPU path and the oracle then consume exactly the rounded values.
"""
import numpy as np


def bf16_bits_from_f64(x):
    """Round float64 values to bfloat16 (RNE, a single rounding) and return the
    16-bit patterns as uint16.

    bfloat16 keeps the float32 exponent range and 7 stored significand bits, so
    the float64 significand (52 bits) is rounded at bit 45 and the exponent is
    re-biased from 1023 to 127.  Zero maps to (signed) zero; values outside the
    normal bfloat16 range are rejected, since the generators never produce them.
    """
    x = np.ascontiguousarray(x, dtype=np.float64)
    u = x.view(np.uint64)
    sign = (u >> np.uint64(63)).astype(np.uint64)
    mag = u & np.uint64(0x7FFFFFFFFFFFFFFF)
    # round the magnitude at bit 45 with ties to even
    lsb = (mag >> np.uint64(45)) & np.uint64(1)
    rounded = (mag + np.uint64((1 << 44) - 1) + lsb) >> np.uint64(45)
    exp11 = rounded >> np.uint64(7)
    mant7 = rounded & np.uint64(0x7F)
    zero = mag == 0
    exp8 = exp11.astype(np.int64) - 1023 + 127
    bad = (~zero) & ((exp8 < 1) | (exp8 > 254))
    if np.any(bad):
        raise ValueError("value outside the normal bfloat16 range")
    exp8 = np.where(zero, 0, exp8).astype(np.uint64)
    mant7 = np.where(zero, np.uint64(0), mant7)
    bits = (sign << np.uint64(15)) | (exp8 << np.uint64(7)) | mant7
    return bits.astype(np.uint16)


def f64_from_bf16_bits(bits):
    """Widen bfloat16 bit patterns (uint16) to the float64 values they encode."""
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)
