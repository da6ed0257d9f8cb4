"""Pins for the oracle's coarse quantization granularities (Sec. 4, Table
fp8-granularities: per tensor and per token, read as one scale per tensor
and one scale per activation row / weight output channel)."""

from fractions import Fraction

import numpy as np
import pytest

import synth
from exact_helpers import decode_exact, encode_nearest, f32_bits, quantize_group_exact, rn32
from synth import to_bf16_bits
from oracle.ffn import ffn_bf16_reference, group_gemm, quant_weights, rmsnorm, rmsnorm_quant, ffn
from oracle.granularity import GRAN_TENSOR, GRAN_TOKEN, ffn_g, quant_weights_g, quantize_rows, scaled_gemm


def test_hand_worked_tensor_and_token():
    # the Appendix-B amax-128 example spread over two rows: per tensor every
    # value shares scale RN32(128 / 448) = 0x3E924925; 1 -> 3.5 (0x46), 3 -> 10
    # (tie, 0x52), 5 -> 18 (0x59), 128 -> 448 (0x7E), -64 -> -224 (0xF6)
    v = np.array([[1, 3, 5], [128, -64, 0]], dtype=np.float32)
    codes, s = quantize_rows(v, GRAN_TENSOR)
    assert [f32_bits(x) for x in s] == [0x3E924925, 0x3E924925]
    assert codes.tolist() == [[0x46, 0x52, 0x59], [0x7E, 0xF6, 0x00]]
    # per token the first row's own amax 5 sets its scale: 5 -> 448
    codes, s = quantize_rows(v, GRAN_TOKEN)
    assert codes[0, 2] == 0x7E and codes[1].tolist() == [0x7E, 0xF6, 0x00]
    assert f32_bits(s[1]) == 0x3E924925


@pytest.mark.parametrize("gran", [GRAN_TOKEN, GRAN_TENSOR])
def test_bruteforce_exact_rationals(gran):
    rng = np.random.default_rng(11 + gran)
    v = rng.standard_normal((4, 40)).astype(np.float32)
    v[1] *= np.float32(30.0)
    v[2, 7] = np.float32(-900.0)
    v[3] = 0.0
    codes, s = quantize_rows(v, gran)
    sets = [list(r) for r in v] if gran == GRAN_TOKEN else [list(v.reshape(-1))]
    ref = [quantize_group_exact(g) for g in sets]
    if gran == GRAN_TOKEN:
        for m in range(4):
            assert float(s[m]) == ref[m][0]
            assert codes[m].tolist() == ref[m][1]
    else:
        assert np.all(s == np.float32(ref[0][0]))
        assert codes.reshape(-1).tolist() == ref[0][1]


@pytest.mark.parametrize("gran", [GRAN_TOKEN, GRAN_TENSOR])
def test_invariants(gran):
    rng = np.random.default_rng(5)
    v = (rng.standard_normal((6, 256)) * np.exp(rng.uniform(-3, 3, (6, 1)))).astype(np.float32)
    codes, s = quantize_rows(v, gran)
    mag = codes & 0x7F
    if gran == GRAN_TOKEN:
        # every non-zero row reaches the top code 448, and only where |v| / s
        # rounds to it, i.e. |v| >= 432 s (the midpoint to 416) ~ amax (1 - 1/28)
        for m in range(6):
            assert (mag[m] == 0x7E).any()
            top = np.abs(v[m]) >= np.abs(v[m]).max() * (1 - 1 / 28) * (1 - 1e-6)
            assert np.all((mag[m] == 0x7E) <= top)
    else:
        assert len(set(s.tolist())) == 1
        assert (mag == 0x7E).sum() >= 1
        assert mag.reshape(-1)[np.argmax(np.abs(v))] == 0x7E
    # dequantization error at most half an e4m3 step (relative 2^-4) of each value,
    # or half the smallest subnormal step (2^-10 s) near zero
    dq = np.array([[float(decode_exact(int(c))) for c in r] for r in codes]) * s[:, None].astype(np.float64)
    err = np.abs(dq - v.astype(np.float64))
    assert np.all(err <= np.maximum(np.abs(v) * 2.0 ** -4, 2.0 ** -10 * s[:, None]) * 1.0000001)


def test_special_cases_reduce_to_the_group_quantizer():
    rng = np.random.default_rng(9)
    # a row of exactly one 128-wide group: per token == per group
    v = rng.standard_normal((5, 128)).astype(np.float32)
    codes_t, s_t = quantize_rows(v, GRAN_TOKEN)
    for m in range(5):
        s_g, c_g = quantize_group_exact(list(v[m]))
        assert codes_t[m].tolist() == c_g and float(s_t[m]) == s_g
    # a single row: per tensor == per token
    one = rng.standard_normal((1, 384)).astype(np.float32)
    a, sa = quantize_rows(one, GRAN_TENSOR)
    b, sb = quantize_rows(one, GRAN_TOKEN)
    assert np.array_equal(a, b) and np.array_equal(sa, sb)


@pytest.mark.parametrize("gran", [GRAN_TOKEN, GRAN_TENSOR])
def test_weight_channels(gran):
    rng = np.random.default_rng(2)
    w = rng.standard_normal((256, 128)).astype(np.float32) * np.float32(0.02)
    w[3] *= np.float32(20.0)
    bits = to_bf16_bits(w)
    q, rs = quant_weights_g(bits, gran)
    assert q.shape == (256, 128) and rs.shape == (256,)
    from oracle.bf16 import bf16_to_f32
    wf = bf16_to_f32(bits)
    for n in (0, 3, 255):
        if gran == GRAN_TOKEN:
            s_ref, c_ref = quantize_group_exact(list(wf[n]))
        else:  # the tensor's scale, then row n's codes with it
            s_ref = rn32(Fraction(float(np.abs(wf).max())) / 448)
            c_ref = [encode_nearest(rn32(Fraction(float(v)) / Fraction(s_ref))) for v in wf[n]]
        assert float(rs[n]) == s_ref
        assert q[n].tolist() == c_ref


def test_scaled_gemm_exact_and_against_the_group_gemm():
    rng = np.random.default_rng(4)
    M, N, K = 3, 256, 256
    aq = rng.integers(0, 256, (M, K), dtype=np.uint8)
    bq = rng.integers(0, 256, (N, K), dtype=np.uint8)
    aq[(aq & 0x7F) == 0x7F] = 0x11  # no NaN codes
    bq[(bq & 0x7F) == 0x7F] = 0x22
    a_s = rng.uniform(0.01, 2.0, M).astype(np.float32)
    b_s = rng.uniform(0.01, 2.0, N).astype(np.float32)
    got = scaled_gemm(aq, a_s, bq, b_s)
    # brute force in exact rationals, one final rounding comparison
    for m in range(M):
        for n in (0, 77, 255):
            P = sum(decode_exact(int(aq[m, k])) * decode_exact(int(bq[n, k])) for k in range(K))
            exact = P * Fraction(float(a_s[m])) * Fraction(float(b_s[n]))
            assert abs(Fraction(got[m, n]) - exact) <= abs(exact) * Fraction(1, 2 ** 50)
    # the pinned per-group GEMM with every group's scale equal to the row's
    # (weight rows sharing one scale per 128-row block) gives the same values
    b_blk = np.repeat(b_s[::128], 128)
    g = group_gemm(aq, np.tile(a_s, (K // 128, 1)), bq, np.tile(b_s[::128, None], (1, K // 128)))
    s = scaled_gemm(aq, a_s, bq, b_blk)
    assert np.allclose(g, s, rtol=1e-12, atol=0)


def test_coarser_granularity_loses_more_accuracy():
    """The paper's finding (Table fp8-granularities), on synthetic data: against the
    unquantized bf16 FFN, per-group error < per-token error < per-tensor error
    when a few activation channels carry outliers."""
    w = synth.WORKLOADS["tiny_m64_h256_i768"]
    b = synth.make_weights(w, 1)
    x = synth.make_x(w, layer=1, step=0).copy()
    from oracle.bf16 import bf16_to_f32
    xf = bf16_to_f32(x)
    xf[:, [5, 77, 200]] *= np.float32(40.0)  # outlier channels
    xf[::7] *= np.float32(8.0)                # some tokens much larger than others
    x = to_bf16_bits(xf)
    ref = ffn_bf16_reference(x, b["norm_w"], b["w_gate"], b["w_up"], b["w_down"])
    wgu = np.concatenate([b["w_gate"], b["w_up"]], axis=0)
    errs = {}
    gq, gs = quant_weights(wgu)
    dq, ds = quant_weights(b["w_down"])
    errs["group"] = ffn(x, b["norm_w"], gq, gs, dq, ds, w.I)["out64"]
    for name, gran in (("token", GRAN_TOKEN), ("tensor", GRAN_TENSOR)):
        q1, s1 = quant_weights_g(wgu, gran)
        q2, s2 = quant_weights_g(b["w_down"], gran)
        errs[name] = ffn_g(x, b["norm_w"], q1, s1, q2, s2, w.I, gran)["out64"]
    rel = {k: float(np.sqrt(((v - ref) ** 2).mean() / (ref ** 2).mean())) for k, v in errs.items()}
    assert rel["group"] < rel["token"] < rel["tensor"], rel


def test_ffn_g_uses_the_pinned_norm():
    w = synth.WORKLOADS["tiny_m64_h256_i768"]
    b = synth.make_weights(w, 1)
    x = synth.make_x(w, layer=1, step=0)
    wgu = np.concatenate([b["w_gate"], b["w_up"]], axis=0)
    q1, s1 = quant_weights_g(wgu, GRAN_TOKEN)
    q2, s2 = quant_weights_g(b["w_down"], GRAN_TOKEN)
    r = ffn_g(x, b["norm_w"], q1, s1, q2, s2, w.I, GRAN_TOKEN)
    y, _ = rmsnorm(x, b["norm_w"])
    assert np.array_equal(r["y"], y)
    xq_g, _ = rmsnorm_quant(x, b["norm_w"])  # per-group codes differ from per-token ones
    assert r["xq"].shape == xq_g.shape and not np.array_equal(r["xq"], xq_g)
