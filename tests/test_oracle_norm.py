"""Pins for the oracle's fused RMSNorm + 1x128 quantization (Sec. 3.4, "AddNorm";
Sec. 3.3.2 names the norm as RMSNorm)."""

import math
from decimal import Decimal, getcontext
from fractions import Fraction

import numpy as np
import torch

from exact_helpers import f32_bits, quantize_group_exact, rn32
from oracle.bf16 import bf16_to_f32
from oracle.ffn import EPS, canonical_sumsq, rms_inv, rmsnorm, rmsnorm_quant


def _bits(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _rows(seed, M, H):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((M, H)).astype(np.float32) * np.exp(rng.uniform(-3, 3, (M, 1))).astype(np.float32)
    x[:, rng.choice(H, max(1, H // 100), replace=False)] *= 40
    return _bits(x)


def test_canonical_sum_gives_same_r_as_exactly_rounded_sum():
    for H in (256, 4096):
        xb = _rows(1, 300, H)
        x = bf16_to_f32(xb).astype(np.float64)
        ss_c = canonical_sumsq(x)
        ss_f = np.array([math.fsum(row * row) for row in x])
        # fp64 sums agree to a few ulps, and the fp32 reciprocal roots agree exactly
        assert np.all(np.abs(ss_c - ss_f) <= 8 * np.spacing(ss_f))
        assert np.array_equal(rms_inv(ss_c, H), rms_inv(ss_f, H))


def test_canonical_sum_order_on_constructed_rows():
    """Rows whose fp64 sum depends on the order, worked by hand.

    x[0] = 2^26 gives a square of 2^52, where the fp64 spacing is 1; four
    elements 0.5 give squares 0.25 that vanish one at a time when added to
    2^52 but sum to an exact 1 when added to each other first. Element i
    belongs to chunk i // 8 and partial (i // 8) mod 64.
    """
    H = 1024

    def ss(idx):
        x = np.zeros(H)
        x[0] = 2.0 ** 26
        x[list(idx)] = 0.5
        return canonical_sumsq(x[None, :])[0]

    assert ss(range(1, 5)) == 2.0 ** 52            # same chunk as x[0]: lost one by one
    assert ss(range(8, 12)) == 2.0 ** 52 + 1       # chunk 1 -> partial 1, exact 1 meets 2^52 once
    assert ss(range(512, 516)) == 2.0 ** 52        # chunk 64 -> partial 0 again (second pass)
    assert ss(range(520, 524)) == 2.0 ** 52 + 1    # chunk 65 -> partial 1
    # butterfly: partials 1..4 (0.25 each) meet partial 0 in pairs, 2^52 + 0.25 -> 2^52
    assert ss([8, 16, 24, 32]) == 2.0 ** 52


def test_rms_inv_matches_high_precision_evaluation():
    getcontext().prec = 60
    xb = _rows(2, 120, 256)
    x = bf16_to_f32(xb)
    r = rms_inv(canonical_sumsq(x), 256)
    eps = Fraction(EPS)  # the fp64 value of 1e-5, exactly
    for i in range(x.shape[0]):
        ss = sum(Fraction(float(v)) ** 2 for v in x[i])
        v = ss / 256 + eps
        d = Decimal(v.numerator) / Decimal(v.denominator)
        inv = Decimal(1) / d.sqrt()
        assert float(r[i]) == rn32(Fraction(inv)), i


def test_constant_row_closed_form():
    for c in (0.5, 3.0, 96.0):
        xb = _bits(np.full((1, 512), c))
        wb = _bits(np.ones(512))
        y, r = rmsnorm(xb, wb)
        ref = np.float32(1.0 / math.sqrt(c * c + EPS))
        assert r[0] == ref
        assert np.all(y == np.float32(np.float64(c) * np.float64(ref)))


def test_y_is_single_rounding_of_exact_product():
    rng = np.random.default_rng(4)
    xb = _rows(3, 64, 512)
    wb = _bits(1 + 0.02 * rng.standard_normal(512))
    y, r = rmsnorm(xb, wb)
    x64 = bf16_to_f32(xb).astype(np.float64)
    w64 = bf16_to_f32(wb).astype(np.float64)
    # x*w has <= 16 significant bits and r 24, so x*w*r is exact in fp64
    ref = (x64 * w64[None, :] * r.astype(np.float64)[:, None]).astype(np.float32)
    assert np.array_equal(y, ref)


def test_rmsnorm_quant_layout_and_groups():
    M, H = 5, 512
    rng = np.random.default_rng(8)
    x = rng.standard_normal((M, H)).astype(np.float32)
    x[3, 300] = 200.0  # row 3, group 2
    xb = _bits(x)
    wb = _bits(np.ones(H))
    xq, xs = rmsnorm_quant(xb, wb)
    assert xq.shape == (M, H) and xs.shape == (H // 128, M)
    assert np.argmax(xs[:, 3]) == 2 and xs[2, 3] == xs.max()
    assert xq[3, 300] == 0x7E
    y, _ = rmsnorm(xb, wb)
    for m in range(M):
        for kb in range(H // 128):
            s, codes = quantize_group_exact(y[m, kb * 128:(kb + 1) * 128])
            assert f32_bits(xs[kb, m]) == f32_bits(s)
            assert xq[m, kb * 128:(kb + 1) * 128].tolist() == codes
