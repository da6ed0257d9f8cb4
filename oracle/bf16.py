"""bfloat16 helpers for the oracle (test infrastructure only).

The paper keeps every module outside the FP8 linears at its original 16-bit
precision (Sec. 3.4); the 16-bit type here is bfloat16, stored as raw
uint16 bit patterns (the upper half of an IEEE fp32).
"""

import numpy as np


def bf16_to_f32(bits):
    """Exact widening of bf16 bit patterns (uint16) to float32."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


def rne_bf16(v):
    """Round float64 (or float32) values to bf16, nearest with ties to even.

    Rounds the given value once, directly (no intermediate fp32 rounding).
    Returns uint16 bit patterns. Overflow goes to +-Inf; NaN is not expected.
    """
    x = np.asarray(v, dtype=np.float64)
    if np.any(np.isnan(x)):
        raise ValueError("rne_bf16: NaN input")
    _, ex = np.frexp(x)  # |x| = f * 2^ex, f in [0.5, 1)
    # bf16 has 8 significant bits; below 2^-126 the spacing stays 2^-133.
    e = np.maximum(ex, -125)
    scale = np.exp2((8 - e).astype(np.float64))
    q = np.rint(x * scale) / scale  # exact: power-of-two scaling, RNE to integer
    with np.errstate(over="ignore"):
        q32 = q.astype(np.float32)  # exact for every bf16 value; 2^128 -> inf
    return (q32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
