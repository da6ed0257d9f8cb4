"""Pins for the token-wise first-layer oracle (Sec. 3.3, EmbedCache and
RoPECache): RoPE against closed forms and its invariants, the bf16 linear
against exact rationals, and the caching identity the paper states (updating
only the current block's rows equals recomputing every row)."""

from fractions import Fraction

import numpy as np

import oracle.first_layer as F
from oracle.bf16 import bf16_to_f32, rne_bf16
from oracle.ffn import rmsnorm
from synth import to_bf16_bits

D = 128


def test_rope_tables_closed_form():
    c, s = F.rope_tables(16, D, 10000.0)
    assert c.shape == (16, 64) and s.shape == (16, 64)
    assert np.all(c[0] == 1.0) and np.all(s[0] == 0.0)
    # theta_0 = 1: angle p; theta_63 = base^(-126/128)
    p = np.arange(16)
    assert np.array_equal(c[:, 0], np.cos(p).astype(np.float32))
    assert np.array_equal(s[:, 63], np.sin(p * 10000.0 ** (-126 / 128)).astype(np.float32))


def test_rope_hand_worked_pairing():
    # x = e_0 (dimension 0 of the first half) at position p: the first half
    # gets cos(p), dimension 64 (the paired one of the second half) sin(p);
    # x = e_64: dimension 0 gets -sin(p), dimension 64 cos(p)
    c, s = F.rope_tables(8, D, 10000.0)
    for p in (0, 1, 5):
        e0 = np.zeros((1, D), dtype=np.float32)
        e0[0, 0] = 1.0
        o = bf16_to_f32(F.rope(to_bf16_bits(e0), np.array([p]), c, s))
        assert o[0, 0] == bf16_to_f32(rne_bf16(c[p, 0]))
        assert o[0, 64] == bf16_to_f32(rne_bf16(s[p, 0]))
        assert np.count_nonzero(o) <= 2
        e64 = np.zeros((1, D), dtype=np.float32)
        e64[0, 64] = 1.0
        o = bf16_to_f32(F.rope(to_bf16_bits(e64), np.array([p]), c, s))
        assert o[0, 0] == bf16_to_f32(rne_bf16(-s[p, 0])) and o[0, 64] == bf16_to_f32(rne_bf16(c[p, 0]))


def test_rope_position_zero_is_identity_and_norms_are_kept():
    rng = np.random.default_rng(1)
    x = to_bf16_bits(rng.standard_normal((6, D)).astype(np.float32))
    c, s = F.rope_tables(64, D, 500000.0)
    assert np.array_equal(F.rope(x, np.zeros(6, dtype=int), c, s), x)
    pos = np.array([1, 7, 13, 30, 50, 63])
    o = bf16_to_f32(F.rope(x, pos, c, s)).astype(np.float64)
    xf = bf16_to_f32(x).astype(np.float64)
    n_in = xf[:, :64] ** 2 + xf[:, 64:] ** 2
    n_out = o[:, :64] ** 2 + o[:, 64:] ** 2
    assert np.allclose(n_out, n_in, rtol=2 ** -6, atol=1e-6)


def test_rope_scores_depend_on_the_position_difference():
    rng = np.random.default_rng(2)
    q = to_bf16_bits(rng.standard_normal((1, D)).astype(np.float32))
    k = to_bf16_bits(rng.standard_normal((1, D)).astype(np.float32))
    c, s = F.rope_tables(200, D, 10000.0)

    def score(m, n):
        a = bf16_to_f32(F.rope(q, np.array([m]), c, s)).astype(np.float64)
        b = bf16_to_f32(F.rope(k, np.array([n]), c, s)).astype(np.float64)
        return float((a * b).sum())

    ref = score(3, 10)
    for t in (5, 40, 150):
        assert abs(score(3 + t, 10 + t) - ref) <= 0.05 * (1 + abs(ref))
    assert abs(score(3, 11) - ref) > 1e-3  # and do change with the difference


def test_linear_bf16_against_exact_rationals():
    rng = np.random.default_rng(3)
    a = to_bf16_bits(rng.standard_normal((3, 96)).astype(np.float32))
    w = to_bf16_bits((0.02 * rng.standard_normal((5, 96))).astype(np.float32))
    got = F.linear_bf16(a, w)
    af, wf = bf16_to_f32(a), bf16_to_f32(w)
    for m in range(3):
        for n in range(5):
            exact = sum(Fraction(float(af[m, k])) * Fraction(float(wf[n, k])) for k in range(96))
            assert got[m, n] == rne_bf16(np.float64(exact))  # one rounding of the (fp64-exact) value


def test_embed_norm_gathers_and_uses_the_pinned_norm():
    rng = np.random.default_rng(4)
    table = to_bf16_bits(rng.standard_normal((50, 256)).astype(np.float32))
    nw = to_bf16_bits((1 + 0.02 * rng.standard_normal(256)).astype(np.float32))
    ids = np.array([7, 7, 49, 0])
    x, y = F.embed_norm(ids, table, nw)
    assert np.array_equal(x, table[ids])
    ry, _ = rmsnorm(table[ids], nw)
    assert np.array_equal(y, rne_bf16(ry))


def test_caching_identity():
    """Sec. 3.3: with the caches of a full computation, recomputing only the
    rows of C after their token ids change equals a full recomputation."""
    rng = np.random.default_rng(5)
    H, heads, N, V = 256, 2, 96, 40
    table = to_bf16_bits(rng.standard_normal((V, H)).astype(np.float32))
    nw = to_bf16_bits((1 + 0.02 * rng.standard_normal(H)).astype(np.float32))
    wqkv = to_bf16_bits((0.05 * rng.standard_normal((3 * heads * D, H))).astype(np.float32))
    c, s = F.rope_tables(N, D, 500000.0)
    ids0 = rng.integers(0, V, N)
    ids1 = ids0.copy()
    C = np.arange(32, 64)
    ids1[C] = rng.integers(0, V, len(C))

    def fresh():
        return (np.zeros((N, H), np.uint16), np.zeros((heads, N, D), np.uint16), np.zeros((heads, N, D), np.uint16),
                np.zeros((heads, N, D), np.uint16))

    full = fresh()
    F.token_rows(ids1, np.arange(N), table, nw, wqkv, c, s, heads, D, *full)
    cached = fresh()
    F.token_rows(ids0, np.arange(N), table, nw, wqkv, c, s, heads, D, *cached)
    F.token_rows(ids1[C], C, table, nw, wqkv, c, s, heads, D, *cached)
    for a, b in zip(full, cached):
        assert np.array_equal(a, b)
    # and the scatter layout: head h of V at row r is its slice of the projection
    qkv = F.linear_bf16(F.embed_norm(ids1[:1], table, nw)[1], wqkv)
    assert np.array_equal(full[3][1, 0], qkv[0, (2 * heads + 1) * D:(2 * heads + 2) * D])
