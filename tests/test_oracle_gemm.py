"""Pins for the oracle's FP8 GEMMs with per-group dequantization, the SwiGLU and
re-quantization, the bf16 helpers and the whole-FFN composition (Sec. 3.4)."""

import math
from fractions import Fraction

import numpy as np
import torch

import synth
from exact_helpers import decode_exact, f32_bits, quantize_group_exact
from oracle.bf16 import bf16_to_f32, rne_bf16
from oracle.ffn import (ffn, ffn_bf16_reference, gateup_swiglu_quant, group_gemm, quant_weights, requant,
                        residual_add, silu)


def _finite_codes(rng, shape):
    c = rng.integers(0, 256, shape, dtype=np.uint8)
    return np.where((c & 0x7F) == 0x7F, np.uint8(0x7E), c).astype(np.uint8)


def _exact_gemm(aq, as_, bq, bs, g=128, with_terms=False):
    """Triple loop in exact rationals: sum_kb a_s*b_s*sum_k D(a)D(b).

    With ``with_terms`` also returns sum_kb |a_s*b_s*dot_kb| per element.
    """
    M, K = aq.shape
    N = bq.shape[0]
    Da = [[decode_exact(int(c)) for c in row] for row in aq]
    Db = [[decode_exact(int(c)) for c in row] for row in bq]
    out = [[Fraction(0)] * N for _ in range(M)]
    mag = [[Fraction(0)] * N for _ in range(M)]
    for m in range(M):
        for n in range(N):
            tot = Fraction(0)
            for kb in range(K // g):
                dot = sum(Da[m][k] * Db[n][k] for k in range(kb * g, (kb + 1) * g))
                term = Fraction(float(as_[kb, m])) * Fraction(float(bs[n // g, kb])) * dot
                tot += term
                mag[m][n] += abs(term)
            out[m][n] = tot
    return (out, mag) if with_terms else out


def test_single_group_dot_products_are_exact():
    rng = np.random.default_rng(1)
    aq = _finite_codes(rng, (4, 128))
    bq = _finite_codes(rng, (128, 128))
    acc = group_gemm(aq, np.ones((1, 4), np.float32), bq, np.ones((1, 1), np.float32))
    # integer form: every e4m3 value is an integer times 2^-9
    ia = np.array([[int(decode_exact(int(c)) * 512) for c in r] for r in aq], dtype=object)
    ib = np.array([[int(decode_exact(int(c)) * 512) for c in r] for r in bq], dtype=object)
    ref = ia.dot(ib.T)
    for m in range(4):
        for n in range(128):
            assert acc[m, n] == float(Fraction(int(ref[m, n]), 2 ** 18))


def test_group_gemm_against_exact_rationals_nonsquare():
    rng = np.random.default_rng(2)
    M, K, N = 3, 384, 256
    aq = _finite_codes(rng, (M, K))
    bq = _finite_codes(rng, (N, K))
    as_ = rng.uniform(0.01, 2.0, (K // 128, M)).astype(np.float32)
    bs = rng.uniform(1e-4, 1e-2, (N // 128, K // 128)).astype(np.float32)
    acc = group_gemm(aq, as_, bq, bs)
    ref, mag = _exact_gemm(aq, as_, bq, bs, with_terms=True)
    for m in range(M):
        for n in range(N):
            # three terms, each rounded once in fp64, plus the roundings of the running sum
            assert abs(acc[m, n] - float(ref[m][n])) <= 6 * 2.0 ** -53 * float(mag[m][n])


def test_gateup_swiglu_against_plain_python():
    """g from fused rows [0, I), u from rows [I, 2I), h = g * sigmoid(g) * u."""
    rng = np.random.default_rng(3)
    M, H, I = 2, 256, 128
    xq = _finite_codes(rng, (M, H)) & np.uint8(0xBF)  # keep magnitudes modest
    xs = rng.uniform(0.001, 0.01, (H // 128, M)).astype(np.float32)
    wq = _finite_codes(rng, (2 * I, H)) & np.uint8(0xBF)
    ws = rng.uniform(0.001, 0.01, (2 * I // 128, H // 128)).astype(np.float32)
    r = gateup_swiglu_quant(xq, xs, wq, ws, I)
    ex = _exact_gemm(xq, xs, wq, ws)
    for m in range(M):
        for j in range(I):
            g = float(ex[m][j])
            u = float(ex[m][I + j])
            h = g / (1.0 + math.exp(-g)) * u
            assert abs(r["h64"][m, j] - h) <= 1e-13 * max(abs(h), 1e-300)
    assert np.array_equal(r["h32"], r["h64"].astype(np.float32))
    for m in range(M):
        s, codes = quantize_group_exact(r["h32"][m])
        assert f32_bits(r["hs"][0, m]) == f32_bits(s)
        assert r["hq"][m].tolist() == codes


def test_silu_special_values():
    z = np.array([0.0, 50.0, -50.0, -800.0, 1.0])
    s = silu(z)
    assert s[0] == 0.0 and s[1] == 50.0 and abs(s[2]) < 1e-19 and s[3] == 0.0
    assert abs(s[4] - 1.0 / (1.0 + math.exp(-1.0))) < 1e-16


def test_requant_layout():
    rng = np.random.default_rng(4)
    h = rng.standard_normal((3, 384)).astype(np.float32)
    h[2, 200] = 1e4
    hq, hs = requant(h)
    assert hs.shape == (3, 3) and hs[1, 2] == np.float32(1e4) / np.float32(448)
    assert hq[2, 200] == 0x7E


def test_rne_bf16_against_torch_and_fp64_ties():
    rng = np.random.default_rng(5)
    with np.errstate(invalid="ignore", over="ignore"):  # signalling NaN patterns in the raw draw
        v = np.concatenate([rng.standard_normal(100000) * np.exp(rng.uniform(-80, 80, 100000)),
                            (rng.integers(0, 2 ** 32, 100000, dtype=np.uint64).astype(np.uint32)).view(np.float32)])
        v = v.astype(np.float32)
    v = v[np.isfinite(v)]
    ref = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(rne_bf16(v), ref)
    # fp64 inputs are rounded once, directly: 1 + 2^-8 is a tie (-> 1.0), while
    # 1 + 2^-8 + 2^-40 lies above it (-> 1 + 2^-7), which a detour through fp32 would miss
    assert rne_bf16(np.array([1 + 2.0 ** -8]))[0] == 0x3F80
    assert rne_bf16(np.array([1 + 2.0 ** -8 + 2.0 ** -40]))[0] == 0x3F81
    assert rne_bf16(np.array([-(1 + 3 * 2.0 ** -8)]))[0] == 0xBF82
    assert np.array_equal(bf16_to_f32(np.array([0x3F80, 0xC000], np.uint16)), np.array([1.0, -2.0], np.float32))


def test_residual_add_against_torch():
    rng = np.random.default_rng(6)
    a = torch.from_numpy(rng.standard_normal(50000).astype(np.float32) * 10).to(torch.bfloat16)
    b = torch.from_numpy(rng.standard_normal(50000).astype(np.float32) * 0.1).to(torch.bfloat16)
    ref = (a.float() + b.float()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = residual_add(a.view(torch.int16).numpy().view(np.uint16), b.view(torch.int16).numpy().view(np.uint16))
    assert np.array_equal(got, ref)


def test_fp8_ffn_is_close_to_bf16_ffn_on_tiny_workload():
    """Composition sanity band: the FP8 FFN tracks the unquantized bf16 FFN."""
    w = synth.WORKLOADS["tiny_m64_h256_i768"]
    wts = synth.make_weights(w, layer=1)
    x = synth.make_x(w, layer=1)
    wgu_q, wgu_s = quant_weights(np.concatenate([wts["w_gate"], wts["w_up"]], axis=0))
    wd_q, wd_s = quant_weights(wts["w_down"])
    r = ffn(x, wts["norm_w"], wgu_q, wgu_s, wd_q, wd_s, w.I)
    ref = ffn_bf16_reference(x, wts["norm_w"], wts["w_gate"], wts["w_up"], wts["w_down"])
    err = np.linalg.norm(r["out64"] - ref) / np.linalg.norm(ref)
    assert 1e-3 < err < 0.12, err
    assert np.array_equal(r["out_bf16"], rne_bf16(r["out64"]))
    # gate/up blocks never straddle the gate/up boundary: quantizing the halves apart is the same
    gq, gs = quant_weights(wts["w_gate"])
    uq, us = quant_weights(wts["w_up"])
    assert np.array_equal(wgu_q, np.concatenate([gq, uq])) and np.array_equal(wgu_s, np.concatenate([gs, us]))


def _rne_bf16_exact(q: Fraction) -> Fraction:
    """Nearest bf16 value of an exact rational (ties to even), normal range."""
    if q == 0:
        return Fraction(0)
    a = abs(q)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    elif Fraction(2) ** (e + 1) <= a:
        e += 1
    unit = Fraction(2) ** (e - 7)  # 8 significant bits
    n = a / unit
    fl = n.numerator // n.denominator
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    v = fl * unit
    return v if q > 0 else -v


def _bits_value(bits):
    return [Fraction(float(v)) for v in bf16_to_f32(np.asarray(bits, np.uint16)).ravel()]


def test_ffn_bf16_reference_against_exact_rationals():
    """The unquantized bf16 FFN (the context figure of the bench line) step by
    step in exact rationals on a tiny layer: y rounded to bf16, g and u the
    exact dot products rounded once to bf16, h = SiLU(g) u (exp in fp64, the
    only inexact step) rounded to bf16, out the exact dot product rounded to
    bf16. A variant that drops any one of the roundings must differ."""
    rng = np.random.default_rng(21)
    M, H, I = 2, 128, 128
    to_bits = lambda a: torch.from_numpy(np.asarray(a, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    xb = to_bits(rng.standard_normal((M, H)))
    nw = to_bits(1 + 0.02 * rng.standard_normal(H))
    wg, wu, wd = (to_bits(rng.standard_normal(s) * 0.3) for s in ((I, H), (I, H), (H, I)))
    got = ffn_bf16_reference(xb, nw, wg, wu, wd)
    from oracle.ffn import rmsnorm
    y, _ = rmsnorm(xb, nw)  # pinned separately (test_oracle_norm.py)
    yb = [[_rne_bf16_exact(Fraction(float(v))) for v in row] for row in y]
    Wg = np.array(_bits_value(wg), dtype=object).reshape(I, H)
    Wu = np.array(_bits_value(wu), dtype=object).reshape(I, H)
    Wd = np.array(_bits_value(wd), dtype=object).reshape(H, I)
    for m in range(M):
        g = [_rne_bf16_exact(sum(yb[m][k] * Wg[n][k] for k in range(H))) for n in range(I)]
        u = [_rne_bf16_exact(sum(yb[m][k] * Wu[n][k] for k in range(H))) for n in range(I)]
        h = []
        for n in range(I):
            gf = float(g[n])
            silu = Fraction(gf / (1.0 + math.exp(-gf)))  # fp64; its error is far below a bf16 step
            h.append(_rne_bf16_exact(silu * u[n]))
        out = [_rne_bf16_exact(sum(h[k] * Wd[n][k] for k in range(I))) for n in range(H)]
        assert [Fraction(float(v)) for v in got[m]] == out, m
    # every rounding matters: dropping the one on g (or on h) changes the output
    y64 = y.astype(np.float64)
    ybf = bf16_to_f32(rne_bf16(y64)).astype(np.float64)
    wgf, wuf, wdf = (bf16_to_f32(w).astype(np.float64) for w in (wg, wu, wd))
    g_nr = ybf @ wgf.T
    u_r = bf16_to_f32(rne_bf16(ybf @ wuf.T)).astype(np.float64)
    h_nr = bf16_to_f32(rne_bf16(g_nr / (1 + np.exp(-g_nr)) * u_r)).astype(np.float64)
    assert not np.array_equal(bf16_to_f32(rne_bf16(h_nr @ wdf.T)).astype(np.float64), got)
