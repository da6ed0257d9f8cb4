"""Exact-arithmetic helpers used by the oracle pins (test code, not oracle code).

They recompute results from definitions with Python integers and Fractions, so
that a pin never re-runs the oracle's own formula.
"""

import math
import struct
from fractions import Fraction

_GRID = [Fraction(m, 512) for m in range(8)] + [
    Fraction(8 + m) * Fraction(2) ** (e - 10) for e in range(1, 16) for m in range(8) if not (e == 15 and m == 7)
]


def f32_bits(x) -> int:
    return struct.unpack("<I", struct.pack("<f", float(x)))[0]


def rn32(q: Fraction) -> float:
    """Round an exact rational to the nearest fp32 value (ties to even).

    Handles subnormals; overflow is not expected here and raises.
    """
    if q == 0:
        return 0.0
    sign = -1.0 if q < 0 else 1.0
    a = abs(q)
    # e = floor(log2 a)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    elif Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, -126)
    unit = Fraction(2) ** (e - 23)
    n = a / unit
    fl = n.numerator // n.denominator
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    v = Fraction(fl) * unit
    if v >= Fraction(2) ** 128:
        raise OverflowError
    return sign * float(v)  # exact: fl has at most 24 bits


def encode_nearest(v) -> int:
    """e4m3fn code of v by exhaustive nearest-grid search (ties to even code)."""
    a = abs(Fraction(float(v)))
    sbit = 0x80 if math.copysign(1.0, float(v)) < 0 else 0
    if a >= 448:
        return sbit | 0x7E
    return sbit | min(range(len(_GRID)), key=lambda c: (abs(_GRID[c] - a), c % 2))


def decode_exact(code: int) -> Fraction:
    s, e, m = code >> 7, (code >> 3) & 15, code & 7
    v = Fraction(m, 512) if e == 0 else Fraction(8 + m) * Fraction(2) ** (e - 10)
    return -v if s else v


def quantize_group_exact(values):
    """Eqs. 7-8 with exact rationals: returns (scale float, [codes])."""
    amax = max(abs(Fraction(float(v))) for v in values)
    s = rn32(amax / 448)
    if s == 0:
        return 0.0, [0] * len(values)
    return s, [encode_nearest(rn32(Fraction(float(v)) / Fraction(s))) for v in values]
