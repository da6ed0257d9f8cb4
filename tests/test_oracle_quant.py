"""Pins for the oracle's group quantizer (Sec. 3.4, Eqs. 7-8) and weight blocks."""

import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from exact_helpers import decode_exact, encode_nearest, f32_bits, quantize_group_exact, rn32
from oracle.e4m3 import e4m3_decode
from oracle.ffn import quant_weights, quantize_groups


def _golden_groups(golden_dir):
    rows = []
    with open(os.path.join(golden_dir, "group_quant.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                a, sb, x, c = line.split()
                rows.append((float(a), int(sb, 16), float(x), int(c, 16)))
    return rows


def test_golden_group_examples(golden_dir):
    rows = _golden_groups(golden_dir)
    assert len(rows) >= 10
    for amax, sbits, x, code in rows:
        g = np.zeros(128, dtype=np.float32)
        g[0] = amax
        g[1] = x
        g[2:] = np.linspace(-amax / 2, amax / 2, 126, dtype=np.float32)
        codes, s = quantize_groups(g)
        assert f32_bits(s) == sbits, (amax, hex(f32_bits(s)))
        assert codes[1] == code, (amax, x, hex(codes[1]))


def test_zero_group_gives_zero_scale_and_codes():
    g = np.zeros((3, 128), dtype=np.float32)
    g[1] = -0.0
    g[2, 5] = 1e-45  # amax / 448 underflows to 0 in fp32
    codes, s = quantize_groups(g)
    assert np.all(s == 0) and np.all(codes == 0)


def test_bruteforce_exact_rationals():
    rng = np.random.default_rng(3)
    groups = [rng.standard_normal(128).astype(np.float32) * np.float32(sc) for sc in (1e-3, 0.7, 40.0, 3e4)]
    outl = rng.standard_normal(128).astype(np.float32)
    outl[17] *= 40
    groups.append(outl)
    groups.append(np.float32(2.0) ** rng.integers(-20, 10, 128).astype(np.float32))  # powers of two
    for g in groups:
        codes, s = quantize_groups(g)
        s_ref, codes_ref = quantize_group_exact(g)
        assert float(s) == s_ref
        assert codes.tolist() == codes_ref


def test_invariants_top_code_and_error_bound():
    rng = np.random.default_rng(5)
    y = (rng.standard_normal((400, 128)) * np.exp(rng.uniform(-8, 8, (400, 1)))).astype(np.float32)
    codes, s = quantize_groups(y)
    # with a normal fp32 scale, the group's largest element maps to +-448
    assert np.all((codes & 0x7F).max(axis=1) == 0x7E)
    # |D(q) s - y| <= s * (half grid step at D(q) + fp32 rounding of y/s)
    dq = e4m3_decode(codes)
    a = np.abs(dq)
    _, ex = np.frexp(np.maximum(a, 2.0 ** -9))
    half_step = np.exp2(np.maximum(ex - 1, -6) - 4.0)
    bound = s[:, None].astype(np.float64) * (half_step + 448 * 2.0 ** -24)
    assert np.all(np.abs(dq * s[:, None] - y) <= bound * (1 + 1e-12))


def test_quant_weights_block_layout():
    """Block (nb, kb) covers rows nb*128.. and columns kb*128..; scale is w_s[nb, kb]."""
    N, K = 256, 384
    rng = np.random.default_rng(9)
    w = rng.standard_normal((N, K)).astype(np.float32) * 0.02
    mags = np.array([[1.0, 2.0, 4.0], [8.0, 16.0, 32.0]], dtype=np.float32)
    for nb in range(2):
        for kb in range(3):
            w[nb * 128 + 3 * kb + nb, kb * 128 + 7 * nb + kb] = mags[nb, kb]
    bits = torch.from_numpy(w).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    wq, ws = quant_weights(bits)
    assert ws.shape == (2, 3) and wq.shape == (N, K)
    assert np.array_equal(ws, mags / np.float32(448))
    wf = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).float().numpy()
    for nb in range(2):
        for kb in range(3):
            blk = wf[nb * 128:(nb + 1) * 128, kb * 128:(kb + 1) * 128].reshape(-1)
            s = Fraction(float(ws[nb, kb]))
            got = wq[nb * 128:(nb + 1) * 128, kb * 128:(kb + 1) * 128].reshape(-1)
            for i in range(0, blk.size, 97):
                assert got[i] == encode_nearest(rn32(Fraction(float(blk[i])) / s))


@pytest.mark.parametrize("code", [0x01, 0x08, 0x38, 0x7E])
def test_decode_exact_agrees(code):
    assert float(decode_exact(code)) == e4m3_decode(np.array([code], dtype=np.uint8))[0]
