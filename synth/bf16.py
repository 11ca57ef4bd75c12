"""Bit-exact bfloat16 encoding of float64 arrays (round to nearest, ties to even).

Inputs are generated in float64 and rounded once to the storage type; both the
GPU path and the oracle then consume exactly the rounded values.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np


def _workers():
    return max(1, min(16, os.cpu_count() or 1))


_CHUNK = 1 << 18   # elements rounded per pass (temporaries stay in cache)


def _bits_chunk(x):
    u = x.view(np.uint64)
    sign = u >> np.uint64(63)
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
    return ((sign << np.uint64(15)) | (exp8 << np.uint64(7)) | mant7).astype(np.uint16)


def bf16_bits_from_f64(x):
    """Round float64 values to bfloat16 (RNE, a single rounding) and return the
    16-bit patterns as uint16 (same shape).

    bfloat16 keeps the float32 exponent range and 7 stored significand bits, so
    the float64 significand (52 bits) is rounded at bit 45 and the exponent is
    re-biased from 1023 to 127.  Zero maps to (signed) zero; values outside the
    normal bfloat16 range are rejected, since the generators never produce them.
    """
    x = np.ascontiguousarray(x, dtype=np.float64)
    flat = x.reshape(-1)
    out = np.empty(flat.shape, dtype=np.uint16)

    def work(i):
        out[i:i + _CHUNK] = _bits_chunk(flat[i:i + _CHUNK])

    starts = range(0, flat.size, _CHUNK)
    if len(starts) > 4:
        with ThreadPoolExecutor(max_workers=_workers()) as ex:
            list(ex.map(work, starts))
    else:
        for i in starts:
            work(i)
    return out.reshape(x.shape)


def f64_from_bf16_bits(bits):
    """Widen bfloat16 bit patterns (uint16) to the float64 values they encode."""
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)
