"""bf16 storage rounding (test infrastructure only).

The cache stores its per-block states in bf16 (Sec. 4, environment).  bf16 is
the top half of an IEEE binary32: 1 sign, 8 exponent and 7 fraction bits.
Rounding to nearest with ties to even is defined here from the two bf16
neighbours of each value and exact fp64 distances, without bit tricks.
"""
from __future__ import annotations

import math

import numpy as np


def _truncate(x32: np.ndarray) -> np.ndarray:
    """bf16 value nearer to zero: the float32 with its low 16 bits cleared."""
    return (x32.view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32)


def round_bf16(x) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); returned as float32
    holding the bf16 values.  NaN -> NaN, +-inf and +-0 kept, overflow -> inf."""
    x32 = np.ascontiguousarray(x, dtype=np.float32)
    flat = x32.reshape(-1)
    out = np.empty_like(flat)
    for i, v in enumerate(flat):
        if np.isnan(v):
            out[i] = np.nan
            continue
        if np.isinf(v) or v == 0:
            out[i] = v
            continue
        lo = _truncate(np.array([v], np.float32))[0]           # toward zero
        lo_bits = int(np.array([lo], np.float32).view(np.uint32)[0])
        hi = np.array([lo_bits + 0x10000], np.uint32).view(np.float32)[0]  # next bf16 away from zero
        # past the largest finite bf16 the next step up is 2^128 (exponent unbounded):
        # a value that rounds there overflows to infinity
        hi_val = float(hi) if np.isfinite(hi) else math.copysign(2.0 ** 128, float(v))
        d_lo = abs(float(v) - float(lo))
        d_hi = abs(hi_val - float(v))
        if d_lo < d_hi:
            out[i] = lo
        elif d_hi < d_lo:
            out[i] = hi
        else:  # tie: the neighbour whose last fraction bit is 0
            out[i] = lo if ((lo_bits >> 16) & 1) == 0 else hi
    return out.reshape(x32.shape)
