"""OCP e4m3fn codec (oracle; test infrastructure only).

The paper quantizes FFN activations and weights to "fp8" with
x' = clip(x / scale_g, Q_min, Q_max) (Sec. 3.4, Eq. 7) but names neither the
FP8 variant nor a rounding rule. Reading taken here: the OCP E4M3 "fn" format
(bias 7, no infinities, NaN = S.1111.111, largest finite 448) with
round-to-nearest, ties to the even code, after clipping to [-448, 448].
Clipping to +-448 and then rounding equals saturating rounding because 448 is
representable.

Decode (closed form):
    e == 0      ->  (m / 8) * 2^-6                (subnormal; 0x00 = +0)
    e in 1..15  ->  (1 + m / 8) * 2^(e - 7)       (e = 15, m = 7 is NaN)
with sign bit 7.

Encode E(v), for finite fp32 or fp64 v:
    sign bit kept (so -0 and negative values that round to zero give 0x80);
    |v| >= 448 saturates to 0x7E | sign;
    otherwise |v| is rounded to the nearest point of the e4m3 grid, ties to
    the code whose least significant bit is 0.
NaN and Inf inputs are outside the quantizer's contract (the group scale
makes every |v| at most 448 * (1 + 2^-23)); the encoder raises on them.
"""

import numpy as np

E4M3_MAX = 448.0
CODE_MAX = 0x7E  # +448
NAN_CODES = (0x7F, 0xFF)


def e4m3_decode(codes):
    """Decode e4m3fn codes (uint8 array) to float64; NaN codes give NaN."""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    s = (c >> 7) & 1
    e = (c >> 3) & 15
    m = c & 7
    mag = np.where(
        e == 0,
        (m / 8.0) * 2.0 ** -6,
        (1.0 + m / 8.0) * np.exp2((e - 7).astype(np.float64)),
    )
    val = np.where(s == 1, -mag, mag)
    return np.where((c & 0x7F) == 0x7F, np.nan, val)


# Non-negative finite grid, in code order 0x00..0x7E; strictly increasing.
_GRID = e4m3_decode(np.arange(0, CODE_MAX + 1, dtype=np.uint8))


def e4m3_encode(v):
    """Saturating round-to-nearest-even encode of finite values to e4m3fn codes.

    ``v`` may be float32 or float64; every fp32 value is exactly representable
    in fp64, so the arithmetic below (a power-of-two scaling and an RNE round
    to an integer) is exact.
    """
    x = np.asarray(v, dtype=np.float64)
    if not np.all(np.isfinite(x)):
        raise ValueError("e4m3_encode: NaN/Inf input is outside the quantizer's contract")
    neg = np.signbit(x)
    a = np.abs(x)
    # Binade of a: a = f * 2^ex with f in [0.5, 1), so floor(log2 a) = ex - 1.
    _, ex = np.frexp(a)
    e = np.maximum(ex - 1, -6)  # subnormal e4m3 numbers share the 2^-6 binade's step
    step = np.exp2((e - 3).astype(np.float64))  # 3 mantissa bits
    n = np.rint(a / step)  # exact quotient; np.rint rounds half to even
    q = n * step  # nearest grid value (may carry into the next binade)
    # Codes are monotone in value over 0x00..0x7E, so the grid index is the code.
    mag = np.searchsorted(_GRID, np.minimum(q, E4M3_MAX)).astype(np.uint8)
    mag = np.where(a >= E4M3_MAX, np.uint8(CODE_MAX), mag)
    return np.where(neg, mag | np.uint8(0x80), mag).astype(np.uint8)
