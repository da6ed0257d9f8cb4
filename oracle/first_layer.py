"""First-layer token-wise operators with EmbedCache and RoPECache, written out
plainly (test infrastructure only).

Sec. 3.3 (EmbedCache and RoPECache): embedding, the attention RMSNorm, the
QKV projection and RoPE act on each token independently, so inside a SAR
block the results of the tokens outside the current block C are computed once
and reused; later denoising steps recompute only the rows of C,
Q, K = RoPE(Norm(Embed(x)) W_{Q,K}) and V = Norm(Embed(x)) W_V, and write them
into the cached tensors. The first layer keeps 16-bit precision (Sec. 3.4).
Readings where the paper is silent:
  * 16-bit = bf16; Norm is the RMSNorm of ``oracle.ffn.rmsnorm`` (fp32 y)
    rounded to bf16; each projection is the exact product rounded to bf16;
  * RoPE is the rotate-half form: for a head vector x = [x1, x2] (two halves of
    d/2) at position p, [x1 c - x2 s, x2 c + x1 s] with c = cos(p theta_i),
    s = sin(p theta_i), theta_i = base^(-2i/d), i < d/2; the angles are inputs
    (fp32 tables of cos and sin per position and i); each product and the
    difference or sum are fp32 operations, the result is rounded to bf16;
  * Q, K and V live as [heads, N, d] (the attention layout), the QKV weight as
    rows [Q heads; K heads; V heads] of d rows each ([3 heads d, H]).

Functions:
  rope_tables     fp64 cos/sin of p theta_i rounded to fp32 ([N, d/2] each);
  embed_norm      rows of the embedding table, and their RMSNorm in bf16;
  linear_bf16     RNE_bf16(a W^T) with the exact fp64 product;
  rope            the rotation of one [rows, d] block at given positions;
  token_rows      the whole token-wise first-layer computation for a set of
                  rows, scattered into (embed_cache, q, k, v).
"""

import numpy as np

from .bf16 import bf16_to_f32, rne_bf16
from .ffn import rmsnorm


def rope_tables(N, d, base):
    """cos and sin of p * base^(-2i/d) for p < N, i < d/2: fp64 rounded to fp32."""
    i = np.arange(d // 2, dtype=np.float64)
    theta = np.power(np.float64(base), -2.0 * i / d)
    ang = np.arange(N, dtype=np.float64)[:, None] * theta[None, :]
    return np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)


def embed_norm(token_ids, embed_bits, norm_w_bits):
    """x = embed[token_ids] (bf16 rows, exact) and y = RNE_bf16(RMSNorm(x))."""
    x = np.asarray(embed_bits)[np.asarray(token_ids)]
    y, _ = rmsnorm(x, norm_w_bits)
    return x, rne_bf16(y)


def linear_bf16(a_bits, w_bits):
    """RNE_bf16 of a [M, K] W^T (W [N, K]) taken in fp64: each bf16 product is
    exact in fp64 and the K-term sum is within K 2^-53 of the exact value
    (relative to the sum of magnitudes), then rounded once to bf16."""
    a = bf16_to_f32(a_bits).astype(np.float64)
    w = bf16_to_f32(w_bits).astype(np.float64)
    return rne_bf16(a @ w.T)


def rope(x_bits, pos, cos_t, sin_t):
    """Rotate-half RoPE of bf16 rows x [R, d] at positions pos [R] with the fp32 tables."""
    x = bf16_to_f32(x_bits)
    d = x.shape[1]
    x1, x2 = x[:, : d // 2], x[:, d // 2:]
    c, s = cos_t[pos], sin_t[pos]
    with np.errstate(over="ignore"):
        o1 = (x1 * c).astype(np.float32) - (x2 * s).astype(np.float32)
        o2 = (x2 * c).astype(np.float32) + (x1 * s).astype(np.float32)
    return rne_bf16(np.concatenate([o1.astype(np.float32), o2.astype(np.float32)], axis=1))


def token_rows(token_ids, rows, embed_bits, norm_w_bits, wqkv_bits, cos_t, sin_t, heads, d,
               embed_cache, q, k, v):
    """The token-wise first layer for the tokens token_ids at sequence rows
    `rows`: embed -> cache row, Norm, QKV projection, RoPE of Q and K at the
    row's position, scattered into q, k, v [heads, N, d] (updated in place;
    the caches are uint16 bf16 arrays). Returns the bf16 QKV projection."""
    rows = np.asarray(rows)
    x, y = embed_norm(token_ids, embed_bits, norm_w_bits)
    embed_cache[rows] = x
    qkv = linear_bf16(y, wqkv_bits)
    for part, dst in enumerate((q, k, v)):
        for h in range(heads):
            blk = qkv[:, (part * heads + h) * d:(part * heads + h + 1) * d]
            dst[h, rows] = blk if part == 2 else rope(blk, rows, cos_t, sin_t)
    return qkv
