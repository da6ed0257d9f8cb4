"""Oracle for the per-group FP8 FFN (test infrastructure only).

Follows the paper's mixed-precision FFN (Sec. 3.4): every layer but the first
runs its gate-up and ffout linears in FP8 with 1x128 activation groups and
128x128 weight blocks, scale_g = max|x| / Q_max and x' = clip(x / scale_g)
(Eqs. 7-8), with the activation quantization fused into the norm before the
gate-up linear and into the SwiGLU before the ffout linear (end of Sec. 3.4;
Fig. 2 caption). Everything else keeps 16-bit precision (bf16 here).

Arithmetic is fp64 unless a step states fp32. Readings taken where the paper
is silent:
  * FP8 = OCP e4m3fn, Q_max = 448, saturating RNE (see ``oracle.e4m3``).
  * scale_g is an fp32 value, RN32(amax / 448); codes are E(RN32(y / s)) with a
    correctly rounded fp32 division. An all-zero group (or one whose scale
    underflows to 0) gets s = 0 and codes 0x00.
  * RMSNorm: y = x * w / sqrt(mean(x^2) + eps), eps = 1e-5; the sum of squares
    is taken in fp64 in a fixed order (``canonical_sumsq``), the reciprocal
    root in fp64 rounded once to fp32, and y = RN32(RN32(x*w) * r) stays fp32
    (it is not rounded to 16 bits before quantization).
  * Gate/up rows [0, I) of the fused weight are the gate, [I, 2I) the up
    projection; SwiGLU h = SiLU(g) * u with SiLU(z) = z / (1 + exp(-z)).
  * The down projection output is rounded once to bf16, nearest-even.

Pins (tests/test_oracle_*.py): the quantizer, norm, GEMM, SwiGLU, bf16 and
residual steps are each checked against exact rational arithmetic, closed
forms or PyTorch's own casts. ``ffn`` is the composition of those steps and is
pinned only through them (the paper prints no values for a whole layer).
``ffn_bf16_reference`` is a context figure, not a parity target; its bf16
rounding steps are pinned against exact-rational arithmetic on a tiny layer.
"""

import numpy as np

from .bf16 import bf16_to_f32, rne_bf16
from .e4m3 import E4M3_MAX, e4m3_decode, e4m3_encode

GROUP = 128
EPS = 1e-5

# Decode table: the closed-form decode of every code (NaN codes never occur in
# quantizer output).
_DEC = e4m3_decode(np.arange(256, dtype=np.uint8))


def dequant_codes(codes):
    """fp64 values of e4m3 codes (table form of ``e4m3_decode``)."""
    return _DEC[np.asarray(codes, dtype=np.uint8)]


# --------------------------------------------------------------------------
# Group quantizer (Sec. 3.4, Eqs. 7-8)
# --------------------------------------------------------------------------

def quantize_groups(y):
    """Quantize float32 groups along the last axis.

    ``y`` has shape [..., G]; each slice along the last axis is one group.
    Returns (codes uint8 [..., G], scale float32 [...]).
      scale = RN32(max|y| / 448)             (Eq. 8; fp32 division)
      code  = E(RN32(y / scale))             (Eq. 7; clip + RNE inside E)
    """
    y = np.asarray(y, dtype=np.float32)
    amax = np.max(np.abs(y), axis=-1)  # exact in fp32
    scale = (amax / np.float32(E4M3_MAX)).astype(np.float32)  # IEEE fp32 division
    zero = scale == np.float32(0.0)
    safe = np.where(zero, np.float32(1.0), scale).astype(np.float32)
    q = (y / safe[..., None]).astype(np.float32)  # IEEE fp32 division
    codes = e4m3_encode(q)
    codes = np.where(zero[..., None], np.uint8(0), codes).astype(np.uint8)
    return codes, scale.astype(np.float32)


def quant_weights(w_bits, group=GROUP):
    """128x128 block quantization of a bf16 weight [N, K] (Sec. 3.4).

    Returns (w_q uint8 [N, K], w_s float32 [N/group, K/group]), where block
    (nb, kb) covers rows [nb*g, nb*g+g) and columns [kb*g, kb*g+g).
    """
    w = bf16_to_f32(w_bits)
    N, K = w.shape
    assert N % group == 0 and K % group == 0
    blocks = w.reshape(N // group, group, K // group, group).transpose(0, 2, 1, 3)
    codes, scale = quantize_groups(blocks.reshape(N // group, K // group, group * group))
    codes = codes.reshape(N // group, K // group, group, group).transpose(0, 2, 1, 3)
    return np.ascontiguousarray(codes.reshape(N, K)), scale


# --------------------------------------------------------------------------
# RMSNorm fused with 1x128 activation quantization (Sec. 3.4, "AddNorm")
# --------------------------------------------------------------------------

SUM_LANES = 64  # partial sums, one per wavefront lane
SUM_CHUNK = 8   # consecutive elements per partial per pass


def canonical_sumsq(x32):
    """Sum of squares of each row in fp64, in one fixed order.

    Row element i belongs to chunk c = i // 8 and partial l = c mod 64; each
    partial adds its squares in increasing i, then the 64 partials combine by
    p_l <- p_l + p_(l xor o) for o = 32, 16, 8, 4, 2, 1, and the sum is p_0.
    Every square of a bf16 value is exact in fp64 and fp64 addition is
    commutative, so this order pins the result bit for bit. It differs from
    the exactly rounded sum by a few fp64 ulps at most.
    """
    x = np.asarray(x32, dtype=np.float64)
    M, H = x.shape
    sq = x * x
    per = SUM_LANES * SUM_CHUNK
    T = -(-H // per)
    padded = np.zeros((M, T * per), dtype=np.float64)
    padded[:, :H] = sq
    v = padded.reshape(M, T, SUM_LANES, SUM_CHUNK)
    p = np.zeros((M, SUM_LANES), dtype=np.float64)
    for t in range(T):
        for j in range(SUM_CHUNK):
            p = p + v[:, t, :, j]
    lane = np.arange(SUM_LANES)
    for o in (32, 16, 8, 4, 2, 1):
        p = p + p[:, lane ^ o]
    return p[:, 0]


def rms_inv(ss, H, eps=EPS):
    """r = RN32(1 / sqrt(ss / H + eps)), every step an fp64 IEEE operation."""
    ms = np.asarray(ss, dtype=np.float64) / np.float64(H)
    return (np.float64(1.0) / np.sqrt(ms + np.float64(eps))).astype(np.float32)


def rmsnorm(x_bits, w_bits, eps=EPS):
    """RMSNorm in fp32: y = RN32(RN32(x * w) * r). Returns (y [M,H] f32, r [M] f32)."""
    x = bf16_to_f32(x_bits)
    w = bf16_to_f32(w_bits)
    r = rms_inv(canonical_sumsq(x), x.shape[1], eps)
    y = ((x * w[None, :]).astype(np.float32) * r[:, None]).astype(np.float32)
    return y, r


def rmsnorm_quant(x_bits, w_bits, eps=EPS, group=GROUP):
    """Fused norm + 1x128 quantization (Sec. 3.4).

    Returns (xq uint8 [M, H], xs float32 [H/group, M]); group kb of row m is
    columns [kb*g, kb*g+g) and its scale is xs[kb, m].
    """
    y, _ = rmsnorm(x_bits, w_bits, eps)
    M, H = y.shape
    codes, scale = quantize_groups(y.reshape(M, H // group, group))
    return codes.reshape(M, H), np.ascontiguousarray(scale.T)


# --------------------------------------------------------------------------
# FP8 GEMM with per-group dequantization (Sec. 3.4: DeepGEMM-style linears)
# --------------------------------------------------------------------------

def group_gemm(a_q, a_s, b_q, b_s, group=GROUP):
    """acc[m, n] = sum_kb (a_s[kb, m] * b_s[n // g, kb]) * sum_{k in kb} D(a[m,k]) D(b[n,k]).

    a_q [M, K] codes with scales a_s [K/g, M]; b_q [N, K] codes with block
    scales b_s [N/g, K/g]. fp64 throughout. The inner 128-term sum is exact
    in fp64 (e4m3 values are integers times 2^-9 below 2^18 in magnitude,
    so 128 products stay below 2^53 units of 2^-18), hence independent of the
    BLAS summation order.
    """
    M, K = a_q.shape
    N = b_q.shape[0]
    assert b_q.shape[1] == K and K % group == 0 and N % group == 0
    acc = np.zeros((M, N), dtype=np.float64)
    for kb in range(K // group):
        cols = slice(kb * group, (kb + 1) * group)
        A = dequant_codes(a_q[:, cols])
        B = dequant_codes(b_q[:, cols])
        P = A @ B.T
        s = a_s[kb].astype(np.float64)[:, None] * np.repeat(b_s[:, kb].astype(np.float64), group)[None, :]
        acc += P * s
    return acc


def silu(z):
    """SiLU(z) = z / (1 + exp(-z)) in fp64."""
    z = np.asarray(z, dtype=np.float64)
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def swiglu(acc, I):
    """h = SiLU(gate) * up, gate = acc[:, :I], up = acc[:, I:2I]; fp64."""
    return silu(acc[:, :I]) * acc[:, I:2 * I]


def gateup_swiglu_quant(xq, xs, wgu_q, wgu_s, I, group=GROUP):
    """Gate/up GEMM, SwiGLU and 1x128 re-quantization (Sec. 3.4).

    Returns dict with acc64 [M, 2I], h64 [M, I], h32 = RN32(h64),
    hq uint8 [M, I] and hs float32 [I/group, M] (the quantizer applied to h32).
    """
    acc = group_gemm(xq, xs, wgu_q, wgu_s, group)
    h64 = swiglu(acc, I)
    h32 = h64.astype(np.float32)
    hq, hs = requant(h32, group)
    return {"acc64": acc, "h64": h64, "h32": h32, "hq": hq, "hs": hs}


def requant(h32, group=GROUP):
    """1x128 quantization of a float32 [M, I] intermediate along I."""
    h32 = np.asarray(h32, dtype=np.float32)
    M, I = h32.shape
    codes, scale = quantize_groups(h32.reshape(M, I // group, group))
    return codes.reshape(M, I), np.ascontiguousarray(scale.T)


def down_proj(hq, hs, wd_q, wd_s, group=GROUP):
    """FP8 ffout linear: returns (out64 [M, H] fp64, out_bf16 bits = RNE_bf16(out64))."""
    out64 = group_gemm(hq, hs, wd_q, wd_s, group)
    return out64, rne_bf16(out64)


def ffn(x_bits, norm_w_bits, wgu_q, wgu_s, wd_q, wd_s, I, eps=EPS, group=GROUP):
    """The whole FP8 FFN of one layer, step by step; returns every intermediate."""
    xq, xs = rmsnorm_quant(x_bits, norm_w_bits, eps, group)
    r = gateup_swiglu_quant(xq, xs, wgu_q, wgu_s, I, group)
    out64, out_bf16 = down_proj(r["hq"], r["hs"], wd_q, wd_s, group)
    r.update({"xq": xq, "xs": xs, "out64": out64, "out_bf16": out_bf16})
    return r


def residual_add(x_bits, y_bits):
    """x' = RNE_bf16(float32(x) + float32(y)): the residual add between stacked layers."""
    s = (bf16_to_f32(x_bits) + bf16_to_f32(y_bits)).astype(np.float32)
    return rne_bf16(s)


def ffn_bf16_reference(x_bits, norm_w_bits, w_gate_bits, w_up_bits, w_down_bits, eps=EPS):
    """Unquantized 16-bit FFN, for context only: every linear output rounded to bf16.

    yb = bf16(RMSNorm(x)); g = bf16(yb Wg^T); u = bf16(yb Wu^T);
    h = bf16(SiLU(g) u); out = bf16(h Wd^T). Returns the output as fp64 values.
    """
    y, _ = rmsnorm(x_bits, norm_w_bits, eps)
    yb = bf16_to_f32(rne_bf16(y)).astype(np.float64)
    wg = bf16_to_f32(w_gate_bits).astype(np.float64)
    wu = bf16_to_f32(w_up_bits).astype(np.float64)
    wd = bf16_to_f32(w_down_bits).astype(np.float64)
    g = bf16_to_f32(rne_bf16(yb @ wg.T)).astype(np.float64)
    u = bf16_to_f32(rne_bf16(yb @ wu.T)).astype(np.float64)
    h = bf16_to_f32(rne_bf16(silu(g) * u)).astype(np.float64)
    return bf16_to_f32(rne_bf16(h @ wd.T)).astype(np.float64)
