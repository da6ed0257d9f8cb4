"""Pins for the oracle's e4m3fn codec (OCP E4M3 read for Sec. 3.4, Eq. 7).

The codec is pinned to things other than itself:
  * the closed-form decode of all 256 codes;
  * hand-worked encodings (tests/golden/e4m3_codes.txt);
  * a pure-Python brute force that picks the nearest grid point with exact
    rational arithmetic;
  * PyTorch's float8_e4m3fn cast after clamping to +-448, over every one of
    the 2^32 fp32 bit patterns (through the plain-C copy of the encoder,
    itself checked against the NumPy encoder).
"""

import math
import os
from concurrent.futures import ThreadPoolExecutor
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import csweep
from oracle.e4m3 import e4m3_decode, e4m3_encode


def _f32(bits):
    return np.array([bits], dtype=np.uint32).view(np.float32)[0]


def test_decode_closed_form_all_codes():
    d = e4m3_decode(np.arange(256, dtype=np.uint8))
    finite = np.isfinite(d)
    assert finite.sum() == 254
    assert np.isnan(d[0x7F]) and np.isnan(d[0xFF])
    assert d[0x7E] == 448.0 and d[0xFE] == -448.0
    assert d[0x01] == 2.0 ** -9 and d[0x08] == 2.0 ** -6 and d[0x38] == 1.0
    assert d[0x00] == 0.0 and not np.signbit(d[0x00]) and np.signbit(d[0x80])
    # each code, from its fields, by the textbook formula
    for c in range(256):
        s, e, m = c >> 7, (c >> 3) & 15, c & 7
        if e == 15 and m == 7:
            continue
        ref = math.ldexp(m, -9) if e == 0 else math.ldexp(8 + m, e - 10)
        assert d[c] == (-ref if s else ref), hex(c)
    # positive codes are strictly increasing in value; negative codes mirror them
    pos = d[0:0x7F]
    assert np.all(np.diff(pos) > 0)
    assert np.array_equal(d[0x80:0xFF], -pos)


def test_roundtrip_every_finite_code():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], dtype=np.uint8)
    assert np.array_equal(e4m3_encode(e4m3_decode(codes)), codes)


def test_midpoints_round_to_even_code():
    d = e4m3_decode(np.arange(0, 0x7F, dtype=np.uint8))
    for c in range(0x7E):
        lo, hi = d[c], d[c + 1]
        mid = (lo + hi) / 2  # exact in fp64 and in fp32 (<= 5 significant bits)
        even = c if c % 2 == 0 else c + 1
        for sign, sbit in ((1.0, 0), (-1.0, 0x80)):
            v = np.float32(sign * mid)
            assert e4m3_encode(np.array([v]))[0] == (even | sbit), (hex(c), mid)
            below = np.nextafter(np.float32(mid), np.float32(0))
            above = np.nextafter(np.float32(mid), np.float32(np.inf))
            assert e4m3_encode(np.array([np.float32(sign) * below]))[0] == (c | sbit)
            assert e4m3_encode(np.array([np.float32(sign) * above]))[0] == ((c + 1) | sbit)


def test_golden_hand_worked_codes(golden_dir):
    rows = []
    with open(os.path.join(golden_dir, "e4m3_codes.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                tok = line.split()
                rows.append((np.float32(float(tok[0])), int(tok[1], 16)))
    assert len(rows) >= 20
    got = e4m3_encode(np.array([v for v, _ in rows], dtype=np.float32))
    for (v, want), g in zip(rows, got):
        assert g == want, (v, hex(want), hex(g))


_GRID_EXACT = [Fraction(m, 512) for m in range(8)] + [
    Fraction(8 + m) * Fraction(2) ** (e - 10) for e in range(1, 16) for m in range(8) if not (e == 15 and m == 7)
]


def _bruteforce_encode(v):
    """Nearest e4m3 grid point by exhaustive search with exact rationals."""
    a = abs(Fraction(float(v)))
    sbit = 0x80 if math.copysign(1.0, float(v)) < 0 else 0
    if a >= 448:
        return sbit | 0x7E
    best = min(range(len(_GRID_EXACT)), key=lambda c: (abs(_GRID_EXACT[c] - a), c % 2))
    return sbit | best


def test_encoder_matches_bruteforce_nearest():
    rng = np.random.default_rng(7)
    vals = [np.float32(x) for x in rng.standard_normal(800) * 30]
    vals += [np.float32(x) for x in rng.uniform(-2e-3, 2e-3, 300)]
    vals += list((rng.integers(0x3A000000, 0x43F00000, 900, dtype=np.uint32)).view(np.float32))
    vals += [np.float32(-x) for x in vals[:300]]
    got = e4m3_encode(np.array(vals, dtype=np.float32))
    for v, g in zip(vals, got):
        assert g == _bruteforce_encode(v), (float(v), hex(g))


def test_c_encoder_matches_numpy_encoder():
    csweep.build_csweep()
    rng = np.random.default_rng(11)
    finite = rng.integers(0, 2 ** 32, 2_000_000, dtype=np.uint64).astype(np.uint32)
    finite = finite[(finite & 0x7F800000) != 0x7F800000]
    binade = np.arange(0x3F800000, 0x40000000, 4, dtype=np.uint32)  # [1, 2), every 4th pattern
    for bits in (finite, binade, binade | np.uint32(0x80000000)):
        v = bits.view(np.float32)
        assert np.array_equal(csweep.encode_f32(v), e4m3_encode(v))


@pytest.mark.slow
def test_c_encoder_matches_torch_cast_all_fp32_patterns():
    """Every fp32 bit pattern: E(v) == float8_e4m3fn(clamp(v, -448, 448)).

    torch's cast alone does not saturate (500 and Inf become NaN), hence the
    clamp. Non-finite inputs are outside the contract and skipped.
    """
    csweep.build_csweep()
    chunk = 1 << 24

    def run(i):
        bits = np.arange(i * chunk, (i + 1) * chunk, dtype=np.uint64).astype(np.uint32)
        v = bits.view(np.float32)
        ref = torch.from_numpy(v).clamp(-448.0, 448.0).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        bad, first = csweep.sweep_check(ref, int(i * chunk))
        return bad, first

    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        results = list(ex.map(run, range((1 << 32) // chunk)))
    total = sum(b for b, _ in results)
    firsts = [hex(f) for b, f in results if b]
    assert total == 0, firsts[:4]
