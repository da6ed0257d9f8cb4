"""GPU parity of the coarse quantization granularities (Sec. 4, Table
fp8-granularities: per token with per-channel weights, per tensor) against
the oracle in oracle/granularity.py, through the C ABI.

Bit-exact: weight codes and row scales, the fp32 RMSNorm, activation codes
and scales (every K-group of a row carries the row's scale). Within a bound
derived from the arithmetic: the gate/up GEMM + SwiGLU (the per-group path's
MFMA error model with the row scales applied after the K sum) and, on the
same operands, the down GEMM (row-max-normalised 2e-3, bf16 = RNE of fp32).
The fused call equals its stages bit for bit, and the paper's finding holds
on the GPU's own outputs: per-group error < per-token < per-tensor.
"""

import numpy as np
import pytest
import torch

import oracle.ffn as O
import oracle.granularity as G
import paper_2607_16339_amd as lc
import synth
from gpu_util import DEV, SILU_LIP, dev_bf16, host, host_bf16, mfma_dot_bound
from oracle.bf16 import bf16_to_f32, rne_bf16

pytestmark = pytest.mark.gpu
GRANS = [(lc.LACACHE_GRAN_TOKEN, G.GRAN_TOKEN), (lc.LACACHE_GRAN_TENSOR, G.GRAN_TENSOR)]


def _say(msg):
    print(msg, flush=True)


def _inputs(M, H, I, seed=7, outliers=True):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((M, H)).astype(np.float32)
    if outliers:
        x[:, rng.choice(H, max(1, H // 100), replace=False)] *= np.float32(40.0)
        x[::5] *= np.float32(6.0)
    nw = (1.0 + 0.02 * rng.standard_normal(H)).astype(np.float32)
    wgu = (0.02 * rng.standard_normal((2 * I, H))).astype(np.float32)
    wd = (0.02 * rng.standard_normal((H, I))).astype(np.float32)
    return tuple(synth.to_bf16_bits(a) for a in (x, nw, wgu, wd))


def _weights(bits, gran):
    w_q, w_s, w_rs = lc.quantize_weights_g(dev_bf16(bits), gran)
    torch.cuda.synchronize()
    return w_q, w_s, w_rs


@pytest.mark.parametrize("gran,ogran", GRANS)
def test_weight_codes_and_row_scales_bit_exact(gran, ogran):
    _, _, wgu, wd = _inputs(8, 256, 384)
    for bits in (wgu, wd):
        w_q, w_s, w_rs = _weights(bits, gran)
        rq, rrs = G.quant_weights_g(bits, ogran)
        gq = lc.weight_codes_rowmajor(w_q)  # the device holds the codes in tiles
        assert np.array_equal(gq, rq), "codes differ in %d places" % int((gq != rq).sum())
        assert np.array_equal(host(w_rs).view(np.uint32), rrs.view(np.uint32))
        assert np.all(host(w_s) == 1.0)


@pytest.mark.parametrize("M", [1, 37, 200])
def test_rmsnorm_f32_bit_exact(M):
    x, nw, _, _ = _inputs(M, 1024, 256)
    y = torch.full((M, 1024), float("nan"), dtype=torch.float32, device=DEV)
    lc.lacache_rmsnorm_f32(dev_bf16(x), dev_bf16(nw), y)
    torch.cuda.synchronize()
    ry, _ = O.rmsnorm(x, nw)
    assert np.array_equal(host(y).view(np.uint32), ry.view(np.uint32))


@pytest.mark.parametrize("gran,ogran", GRANS + [(lc.LACACHE_GRAN_GROUP, None)])
@pytest.mark.parametrize("M,K", [(1, 256), (37, 1024), (200, 768)])
def test_quant_rows_bit_exact(gran, ogran, M, K):
    rng = np.random.default_rng(M + K)
    v = (rng.standard_normal((M, K)) * np.exp(rng.uniform(-4, 4, (M, 1)))).astype(np.float32)
    v[0, :] = 0.0  # an all-zero row
    if M > 2:
        v[2, 5] = np.float32(3e4)
    q = torch.full((M, K), 0xFF, dtype=torch.uint8, device=DEV)
    s_kgm = torch.full((K // 128, M), float("nan"), dtype=torch.float32, device=DEV)
    s_rows = torch.full((M,), float("nan"), dtype=torch.float32, device=DEV)
    lc.lacache_quant_rows_g(torch.from_numpy(v).to(DEV), q, s_kgm, None if ogran is None else s_rows, gran)
    torch.cuda.synchronize()
    if ogran is None:
        rq, rs = O.requant(v)
        assert np.array_equal(host(q), rq)
        assert np.array_equal(host(s_kgm).view(np.uint32), rs.view(np.uint32))
        return
    rq, rs = G.quantize_rows(v, ogran)
    assert np.array_equal(host(q), rq), "codes differ in %d places" % int((host(q) != rq).sum())
    assert np.array_equal(host(s_rows).view(np.uint32), rs.view(np.uint32))
    assert np.array_equal(host(s_kgm).view(np.uint32), np.tile(rs, (K // 128, 1)).view(np.uint32))


def _row_gemm_bound(aq, a_rows, bq, b_rows, acc_abs):
    """|acc_gpu - acc_exact| for acc = (sum_kb P_kb a_s[m]) * b_s[n] in fp32:
    the MFMA chunk truncation of every group, the fp32 rounding of each group
    result, of the accumulation and of the final column scale."""
    KB = aq.shape[1] // 128
    dots = mfma_dot_bound(aq, bq)
    bound = np.zeros((aq.shape[0], bq.shape[0]))
    mag = np.zeros_like(bound)
    for kb in range(KB):
        cols = slice(kb * 128, (kb + 1) * 128)
        P = np.abs(O.dequant_codes(aq[:, cols]) @ O.dequant_codes(bq[:, cols]).T)
        bound += dots[kb] + 2.0 ** -24 * P
        mag += P
    s = np.abs(a_rows.astype(np.float64))[:, None] * np.abs(b_rows.astype(np.float64))[None, :]
    return s * (bound + (KB + 18) * 2.0 ** -24 * mag) + 2.0 ** -23 * acc_abs


@pytest.mark.parametrize("gran,ogran", GRANS)
@pytest.mark.parametrize("M,H,I", [(64, 256, 768), (200, 1024, 2048)])
def test_gemms_against_the_oracle(gran, ogran, M, H, I):
    x, nw, wgu, wd = _inputs(M, H, I, seed=M)
    _say("granularity %d M=%d H=%d I=%d" % (gran, M, H, I))
    wgu_q, wgu_s, wgu_rs = _weights(wgu, gran)
    wd_q, wd_s, wd_rs = _weights(wd, gran)
    y = torch.empty((M, H), dtype=torch.float32, device=DEV)
    xq = torch.empty((M, H), dtype=torch.uint8, device=DEV)
    xs = torch.empty((H // 128, M), dtype=torch.float32, device=DEV)
    xr = torch.empty((M,), dtype=torch.float32, device=DEV)
    h = torch.full((M, I), float("nan"), dtype=torch.float32, device=DEV)
    lc.lacache_rmsnorm_f32(dev_bf16(x), dev_bf16(nw), y)
    lc.lacache_quant_rows_g(y, xq, xs, xr, gran)
    lc.lacache_gateup_swiglu_f32(xq, xs, wgu_q, wgu_s, wgu_rs, h)
    torch.cuda.synchronize()
    # gate/up + SwiGLU against the exact fp64 result of the GPU's own codes
    aq, ar, bq, br = host(xq), host(xr), lc.weight_codes_rowmajor(wgu_q), host(wgu_rs)
    acc = G.scaled_gemm(aq, ar, bq, br)
    dacc = _row_gemm_bound(aq, ar, bq, br, np.abs(acc))
    g, u, dg, du = acc[:, :I], acc[:, I:], dacc[:, :I], dacc[:, I:]
    h64 = O.silu(g) * u
    dh = SILU_LIP * dg * (np.abs(u) + du) + np.abs(O.silu(g)) * du
    dh = dh + 2.0 ** -20 * (np.abs(h64) + dh)
    hg = host(h).astype(np.float64)
    assert np.all(np.isfinite(hg))
    worst = float((np.abs(hg - h64) / np.maximum(dh, 1e-300)).max())
    _say("  h: worst err/bound %.3f" % worst)
    assert worst <= 1.0
    # re-quantization of the GPU's own h: bit-exact
    hq = torch.empty((M, I), dtype=torch.uint8, device=DEV)
    hs = torch.empty((I // 128, M), dtype=torch.float32, device=DEV)
    hr = torch.empty((M,), dtype=torch.float32, device=DEV)
    lc.lacache_quant_rows_g(h, hq, hs, hr, gran)
    out = torch.empty((M, H), dtype=torch.bfloat16, device=DEV)
    tap = torch.full((M, H), float("nan"), dtype=torch.float32, device=DEV)
    lc.lacache_down_proj_g(hq, hs, wd_q, wd_s, wd_rs, out, tap)
    torch.cuda.synchronize()
    rq, rr = G.quantize_rows(host(h), ogran)
    assert np.array_equal(host(hq), rq) and np.array_equal(host(hr).view(np.uint32), rr.view(np.uint32))
    # down on the same operands: fp32 within 2e-3 of the row max, bf16 = RNE(fp32)
    out64 = G.scaled_gemm(host(hq), host(hr), lc.weight_codes_rowmajor(wd_q), host(wd_rs))
    o32 = host(tap).astype(np.float64)
    e = float((np.abs(o32 - out64) / np.maximum(np.abs(out64).max(axis=1, keepdims=True), 1e-300)).max())
    _say("  out: err %.2e" % e)
    assert e <= 2e-3
    assert np.array_equal(host_bf16(out), rne_bf16(host(tap)))


@pytest.mark.parametrize("gran", [lc.LACACHE_GRAN_TOKEN, lc.LACACHE_GRAN_TENSOR])
@pytest.mark.parametrize("M", [32, 200])
def test_fused_call_equals_its_stages(gran, M):
    H, I = 1024, 2048
    x, nw, wgu, wd = _inputs(M, H, I, seed=3)
    wgu_q, wgu_s, wgu_rs = _weights(wgu, gran)
    wd_q, wd_s, wd_rs = _weights(wd, gran)
    xd, nwd = dev_bf16(x), dev_bf16(nw)
    fused = torch.empty((M, H), dtype=torch.bfloat16, device=DEV)
    lc.lacache_ffn_fp8_g(xd, nwd, wgu_q, wgu_s, wgu_rs, wd_q, wd_s, wd_rs, fused, gran)
    y = torch.empty((M, H), dtype=torch.float32, device=DEV)
    xq = torch.empty((M, H), dtype=torch.uint8, device=DEV)
    xs = torch.empty((H // 128, M), dtype=torch.float32, device=DEV)
    r = torch.empty((M,), dtype=torch.float32, device=DEV)
    h = torch.empty((M, I), dtype=torch.float32, device=DEV)
    hq = torch.empty((M, I), dtype=torch.uint8, device=DEV)
    hs = torch.empty((I // 128, M), dtype=torch.float32, device=DEV)
    staged = torch.empty((M, H), dtype=torch.bfloat16, device=DEV)
    lc.lacache_rmsnorm_f32(xd, nwd, y)
    lc.lacache_quant_rows_g(y, xq, xs, r, gran)
    lc.lacache_gateup_swiglu_f32(xq, xs, wgu_q, wgu_s, wgu_rs, h)
    lc.lacache_quant_rows_g(h, hq, hs, r, gran)
    lc.lacache_down_proj_g(hq, hs, wd_q, wd_s, wd_rs, staged)
    again = torch.empty_like(fused)
    lc.lacache_ffn_fp8_g(xd, nwd, wgu_q, wgu_s, wgu_rs, wd_q, wd_s, wd_rs, again, gran)
    torch.cuda.synchronize()
    assert torch.equal(fused.view(torch.int16), staged.view(torch.int16))
    assert torch.equal(fused.view(torch.int16), again.view(torch.int16))


def test_group_granularity_is_the_library_ffn():
    M, H, I = 64, 256, 768
    x, nw, wgu, wd = _inputs(M, H, I, seed=5)
    wgu_q, wgu_s, none1 = _weights(wgu, lc.LACACHE_GRAN_GROUP)
    wd_q, wd_s, none2 = _weights(wd, lc.LACACHE_GRAN_GROUP)
    assert none1 is None and none2 is None
    a = torch.empty((M, H), dtype=torch.bfloat16, device=DEV)
    b = torch.empty_like(a)
    lc.lacache_ffn_fp8_g(dev_bf16(x), dev_bf16(nw), wgu_q, wgu_s, None, wd_q, wd_s, None, a, lc.LACACHE_GRAN_GROUP)
    lc.lacache_ffn_fp8(dev_bf16(x), dev_bf16(nw), wgu_q, wgu_s, wd_q, wd_s, b)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_coarser_granularity_loses_more_accuracy_on_the_gpu():
    """Table fp8-granularities' ordering on the GPU's outputs: against the
    unquantized bf16 FFN of the same inputs, per-group < per-token < per-tensor."""
    M, H, I = 128, 1024, 2048
    x, nw, wgu, wd = _inputs(M, H, I, seed=11)
    I2 = I
    ref = O.ffn_bf16_reference(x, nw, wgu[:I2], wgu[I2:], wd)
    errs = {}
    for name, gran in (("group", lc.LACACHE_GRAN_GROUP), ("token", lc.LACACHE_GRAN_TOKEN),
                       ("tensor", lc.LACACHE_GRAN_TENSOR)):
        wgu_q, wgu_s, wgu_rs = _weights(wgu, gran)
        wd_q, wd_s, wd_rs = _weights(wd, gran)
        out = torch.empty((M, H), dtype=torch.bfloat16, device=DEV)
        lc.lacache_ffn_fp8_g(dev_bf16(x), dev_bf16(nw), wgu_q, wgu_s, wgu_rs, wd_q, wd_s, wd_rs, out, gran)
        torch.cuda.synchronize()
        got = bf16_to_f32(host_bf16(out)).astype(np.float64)
        errs[name] = float(np.sqrt(((got - ref) ** 2).mean() / (ref ** 2).mean()))
    _say("rms error vs the bf16 FFN: %s" % errs)
    assert errs["group"] < errs["token"] < errs["tensor"], errs
