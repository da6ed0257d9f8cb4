"""Quantization granularities of the FP8 FFN, written out plainly (test infrastructure only).

The paper compares its per-group FP8 scheme (1x128 activation groups, 128x128
weight blocks) with two coarser granularities of the same FFN linears, "Per
Tensor" and "Per Token" (Sec. 4, Table fp8-granularities), and finds that the
accuracy loss grows as the granularity coarsens. The paper gives no formulas
for the two; the readings used here:
  * per tensor: one scale for a whole activation tensor (all rows and
    columns), one for a whole weight matrix;
  * per token: one scale per activation row (a token: all of its K values)
    and, for the weights, one per output channel (a weight row: all of its K
    values), the usual pairing with per-token activations.
Everything else is the per-group oracle's reading of Eqs. 7-8 (``oracle.ffn``):
scale = RN32(max|v| / 448), code = E(RN32(v / scale)), an all-zero set gets
scale 0 and codes 0x00; only the set of values that share a scale changes.
Scales are returned as one fp32 value per row (all rows equal for a tensor).

Functions:
  quantize_rows       per-token / per-tensor quantization of fp32 rows;
  quant_weights_g     the same for a bf16 weight [N, K] (rows = output channels);
  scaled_gemm         acc[m, n] = (a_s[m] b_s[n]) sum_k D(a[m, k]) D(b[n, k]), fp64;
  ffn_g               the whole FFN at a granularity: RMSNorm, quantization,
                      gate/up GEMM, SwiGLU, re-quantization of h, down GEMM.
"""

import numpy as np

from .bf16 import bf16_to_f32, rne_bf16
from .ffn import EPS, dequant_codes, quantize_groups, rmsnorm, swiglu

GRAN_GROUP, GRAN_TOKEN, GRAN_TENSOR = 0, 1, 2


def quantize_rows(v32, gran):
    """Quantize float32 rows [M, K] per token (one scale per row) or per tensor
    (one scale for all). Returns (codes uint8 [M, K], scale float32 [M])."""
    v = np.asarray(v32, dtype=np.float32)
    M, K = v.shape
    if gran == GRAN_TOKEN:
        return quantize_groups(v)
    if gran == GRAN_TENSOR:
        codes, s = quantize_groups(v.reshape(1, M * K))
        return codes.reshape(M, K), np.full(M, s[0], dtype=np.float32)
    raise ValueError("granularity must be per token (1) or per tensor (2)")


def quant_weights_g(w_bits, gran):
    """Per-channel (gran 1) or per-tensor (gran 2) quantization of a bf16
    weight [N, K]. Returns (w_q uint8 [N, K], w_row_s float32 [N])."""
    return quantize_rows(bf16_to_f32(w_bits), gran)


def scaled_gemm(a_q, a_s, b_q, b_s):
    """acc[m, n] = (a_s[m] * b_s[n]) * sum_k D(a_q[m, k]) D(b_q[n, k]) in fp64.

    The K sum is exact in fp64 for K up to 2^17 (each product is an integer
    times 2^-18 below 2^36 units), so any summation order gives these bits.
    """
    P = dequant_codes(a_q) @ dequant_codes(b_q).T
    return P * (np.asarray(a_s, dtype=np.float64)[:, None] * np.asarray(b_s, dtype=np.float64)[None, :])


def ffn_g(x_bits, norm_w_bits, wgu_q, wgu_rs, wd_q, wd_rs, I, gran, eps=EPS):
    """The FP8 FFN of one layer at a coarse granularity, step by step:
    y = RMSNorm(x) (fp32, as in the per-group oracle); xq, xs = quantize_rows(y);
    acc = scaled_gemm(xq, xs, Wgu); h = SiLU(g) u in fp64, h32 = RN32(h);
    hq, hs = quantize_rows(h32); out64 = scaled_gemm(hq, hs, Wd);
    out_bf16 = RNE_bf16(out64). Returns every intermediate."""
    y, _ = rmsnorm(x_bits, norm_w_bits, eps)
    xq, xs = quantize_rows(y, gran)
    acc = scaled_gemm(xq, xs, wgu_q, wgu_rs)
    h64 = swiglu(acc, I)
    h32 = h64.astype(np.float32)
    hq, hs = quantize_rows(h32, gran)
    out64 = scaled_gemm(hq, hs, wd_q, wd_rs)
    return {"y": y, "xq": xq, "xs": xs, "acc64": acc, "h64": h64, "h32": h32, "hq": hq, "hs": hs,
            "out64": out64, "out_bf16": rne_bf16(out64)}
