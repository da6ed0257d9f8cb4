"""GPU parity of the token-wise first layer with EmbedCache and RoPECache
(Sec. 3.3) against oracle/first_layer.py, through the C ABI.

Bit-exact: the embedding cache rows and the bf16 RMSNorm (the fused norm's
arithmetic), RoPE + scatter of a given projection, the bf16 rounding of the
linear's own fp32 result, the fused call against its three stages, and the
paper's caching identity on the GPU: updating only the current block's rows
of filled caches equals recomputing every row on the new tokens. Within a
bound: the linear's fp32 result against the exact product (K 2^-24 times the
sum of |a w|, the fp32 accumulation of exact bf16 products).
"""

import numpy as np
import pytest
import torch

import oracle.first_layer as F
import paper_2607_16339_amd as lc
from gpu_util import DEV, dev_bf16, host, host_bf16
from oracle.bf16 import bf16_to_f32, rne_bf16
from synth import to_bf16_bits

pytestmark = pytest.mark.gpu
D = 128


def _say(msg):
    print(msg, flush=True)


def _i32(a):
    return torch.from_numpy(np.asarray(a, dtype=np.int32)).to(DEV)


def _setup(H, heads, N, vocab, seed=0):
    rng = np.random.default_rng(seed)
    embed = to_bf16_bits(rng.standard_normal((vocab, H)).astype(np.float32))
    nw = to_bf16_bits((1 + 0.02 * rng.standard_normal(H)).astype(np.float32))
    wqkv = to_bf16_bits((0.02 * rng.standard_normal((3 * heads * D, H))).astype(np.float32))
    cos_t, sin_t = F.rope_tables(N, D, 500000.0)
    return rng, embed, nw, wqkv, cos_t, sin_t


def _caches(heads, N, H, fill=0x7FC0):
    mk = lambda shape: torch.full(shape, fill, dtype=torch.int16, device=DEV).view(torch.bfloat16)  # noqa: E731
    return mk((N, H)), mk((heads, N, D)), mk((heads, N, D)), mk((heads, N, D))


@pytest.mark.parametrize("R,H", [(1, 256), (33, 1024), (100, 4096)])
def test_embed_rmsnorm_bit_exact(R, H):
    N, vocab = 128, 500
    rng, embed, nw, _, _, _ = _setup(H, 1, N, vocab, seed=R)
    ids = rng.integers(0, vocab, R)
    rows = rng.permutation(N)[:R]
    cache, _, _, _ = _caches(1, N, H)
    y = torch.full((R, H), 0x7FC0, dtype=torch.int16, device=DEV).view(torch.bfloat16)
    lc.lacache_embed_rmsnorm(_i32(ids), _i32(rows), dev_bf16(embed), dev_bf16(nw), cache, y)
    torch.cuda.synchronize()
    x, ry = F.embed_norm(ids, embed, nw)
    assert np.array_equal(host_bf16(y), ry)
    c = host_bf16(cache)
    assert np.array_equal(c[rows], x)
    untouched = np.setdiff1d(np.arange(N), rows)
    assert np.all(c[untouched] == 0x7FC0)


def test_invalid_ids_and_rows_are_skipped():
    H, N, vocab = 256, 64, 50
    _, embed, nw, _, _, _ = _setup(H, 1, N, vocab)
    ids = np.array([3, -1, 50, 7, 9])
    rows = np.array([0, 1, 2, 64, 5])  # ids -1 and 50 and row 64 are out of range
    cache, _, _, _ = _caches(1, N, H)
    y = torch.full((5, H), 0x7FC0, dtype=torch.int16, device=DEV).view(torch.bfloat16)
    lc.lacache_embed_rmsnorm(_i32(ids), _i32(rows), dev_bf16(embed), dev_bf16(nw), cache, y)
    torch.cuda.synchronize()
    c, yy = host_bf16(cache), host_bf16(y)
    assert np.array_equal(c[0], embed[3]) and np.array_equal(c[5], embed[9])
    assert np.all(c[[1, 2]] == 0x7FC0) and np.all(yy[[1, 2, 3]] == 0x7FC0)


def _linear_check(a, w, out, tap):
    af = bf16_to_f32(a).astype(np.float64)
    wf = bf16_to_f32(w).astype(np.float64)
    exact = af @ wf.T
    mag = np.abs(af) @ np.abs(wf).T
    K = a.shape[1]
    t = host(tap).astype(np.float64)
    assert np.all(np.isfinite(t))
    worst = float((np.abs(t - exact) / (K * 2.0 ** -24 * mag + 1e-300)).max())
    _say("  linear: worst err / bound %.3f" % worst)
    assert worst <= 1.0
    assert np.array_equal(host_bf16(out), rne_bf16(host(tap)))


@pytest.mark.parametrize("M,N,K", [(1, 384, 256), (17, 768, 1024), (64, 384, 4096), (100, 384, 512),
                                   (200, 256, 256), (32, 12288, 256), (9, 12288, 512)])
def test_linear_bf16(M, N, K):
    rng = np.random.default_rng(M * 7 + K)
    a = to_bf16_bits(rng.standard_normal((M, K)).astype(np.float32))
    w = to_bf16_bits((0.03 * rng.standard_normal((N, K))).astype(np.float32))
    out = torch.empty((M, N), dtype=torch.bfloat16, device=DEV)
    tap = torch.full((M, N), float("nan"), dtype=torch.float32, device=DEV)
    _say("M=%d N=%d K=%d" % (M, N, K))
    lc.lacache_linear_bf16(dev_bf16(a), dev_bf16(w), out, tap)
    torch.cuda.synchronize()
    _linear_check(a, w, out, tap)


@pytest.mark.parametrize("M,N,K", [(300, 384, 1024), (129, 256, 384), (257, 128, 128), (512, 12288, 4096),
                                   (700, 12288, 512)])
def test_linear_tiled_equals_streaming(M, N, K):
    """Above 128 rows the projection runs on 128 x 128 or 128 x 192 tiles (the
    latter at N = 12288 with 512 and 700 rows); below, W is streamed per 64
    rows. Both must give every row the same bytes (the same
    K quarters, MFMA chains and quarter order), so the same rows through the
    streaming kernel (calls of at most 64 rows) equal the tiled call bit for
    bit, including ragged M, K-step counts not divisible by four and empty
    quarters (K = 128)."""
    rng = np.random.default_rng(M + N + K)
    a = to_bf16_bits(rng.standard_normal((M, K)).astype(np.float32))
    w = to_bf16_bits((0.03 * rng.standard_normal((N, K))).astype(np.float32))
    da, dw = dev_bf16(a), dev_bf16(w)
    _say("tiled vs streaming M=%d N=%d K=%d" % (M, N, K))
    out = torch.empty((M, N), dtype=torch.bfloat16, device=DEV)
    tap = torch.full((M, N), float("nan"), dtype=torch.float32, device=DEV)
    lc.lacache_linear_bf16(da, dw, out, tap)
    out_s = torch.empty_like(out)
    tap_s = torch.full_like(tap, float("nan"))
    for r0 in range(0, M, 64):
        r1 = min(M, r0 + 64)
        lc.lacache_linear_bf16(da[r0:r1], dw, out_s[r0:r1], tap_s[r0:r1])
    torch.cuda.synchronize()
    assert torch.equal(tap.view(torch.int32), tap_s.view(torch.int32))
    assert torch.equal(out.view(torch.int16), out_s.view(torch.int16))
    if M * N * K <= 2 ** 28:
        _linear_check(a, w, out, tap)


def test_linear_maximum_m():
    """M = 2^24 rows, the most the library takes (131072 row tiles): every row
    written, and sampled rows equal to the streaming kernel's bytes and within
    the oracle's bound."""
    M, N, K = 1 << 24, 128, 128
    gen = torch.Generator(device=DEV)
    gen.manual_seed(716339)
    da = torch.randn((M, K), generator=gen, device=DEV, dtype=torch.float32).to(torch.bfloat16)
    rng = np.random.default_rng(24)
    w = to_bf16_bits((0.03 * rng.standard_normal((N, K))).astype(np.float32))
    dw = dev_bf16(w)
    _say("linear M=%d" % M)
    out = torch.empty((M, N), dtype=torch.bfloat16, device=DEV)
    tap = torch.full((M, N), float("nan"), dtype=torch.float32, device=DEV)
    lc.lacache_linear_bf16(da, dw, out, tap)
    rows = np.unique(np.concatenate([[0, 1, M // 2, M - 2, M - 1], rng.choice(M, 27, replace=False)]))
    ri = torch.from_numpy(rows).to(DEV)
    sub = da.index_select(0, ri).contiguous()
    out_s = torch.empty((len(rows), N), dtype=torch.bfloat16, device=DEV)
    tap_s = torch.empty((len(rows), N), dtype=torch.float32, device=DEV)
    lc.lacache_linear_bf16(sub, dw, out_s, tap_s)
    torch.cuda.synchronize()
    assert torch.isfinite(tap).all().item()
    assert torch.equal(tap.index_select(0, ri).view(torch.int32), tap_s.view(torch.int32))
    assert torch.equal(out.index_select(0, ri).view(torch.int16), out_s.view(torch.int16))
    _linear_check(host_bf16(sub), w, out_s, tap_s)
    del da, out, tap
    torch.cuda.empty_cache()


def test_rope_scatter_bit_exact():
    heads, N, R = 3, 192, 40
    rng = np.random.default_rng(4)
    qkv = to_bf16_bits(rng.standard_normal((R, 3 * heads * D)).astype(np.float32))
    rows = rng.permutation(N)[:R]
    cos_t, sin_t = F.rope_tables(N, D, 500000.0)
    _, q, k, v = _caches(heads, N, 256)
    lc.lacache_rope_scatter(dev_bf16(qkv), _i32(rows), torch.from_numpy(cos_t).to(DEV),
                            torch.from_numpy(sin_t).to(DEV), q, k, v)
    torch.cuda.synchronize()
    for part, dst in enumerate((q, k, v)):
        got = host_bf16(dst)
        for h in range(heads):
            blk = qkv[:, (part * heads + h) * D:(part * heads + h + 1) * D]
            ref = blk if part == 2 else F.rope(blk, rows, cos_t, sin_t)
            assert np.array_equal(got[h, rows], ref), (part, h)
        assert np.all(got[:, np.setdiff1d(np.arange(N), rows)] == 0x7FC0)


def _full_call(ids, rows, embed, nw, wqkv, cos_t, sin_t, caches):
    lc.lacache_first_layer_tokens(_i32(ids), _i32(rows), dev_bf16(embed), dev_bf16(nw), dev_bf16(wqkv),
                                  torch.from_numpy(cos_t).to(DEV), torch.from_numpy(sin_t).to(DEV), *caches)


@pytest.mark.parametrize("H,heads,N", [(256, 2, 128), (4096, 32, 512)])
def test_block_update_equals_full_recompute(H, heads, N):
    """The caching identity of Sec. 3.3 on the GPU, bit for bit, plus the
    fused call against its stages and against the oracle."""
    vocab = 1000
    rng, embed, nw, wqkv, cos_t, sin_t = _setup(H, heads, N, vocab, seed=H)
    ids0 = rng.integers(0, vocab, N)
    C = np.arange(N // 2 + 32, N // 2 + 64)  # a 32-token block in the generated half
    ids1 = ids0.copy()
    ids1[C] = rng.integers(0, vocab, len(C))
    _say("H=%d heads=%d N=%d |C|=%d" % (H, heads, N, len(C)))
    full = _caches(heads, N, H)
    _full_call(ids1, np.arange(N), embed, nw, wqkv, cos_t, sin_t, full)
    cached = _caches(heads, N, H)
    _full_call(ids0, np.arange(N), embed, nw, wqkv, cos_t, sin_t, cached)
    _full_call(ids1[C], C, embed, nw, wqkv, cos_t, sin_t, cached)
    torch.cuda.synchronize()
    for a, b in zip(full, cached):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    # the stages of the block update give the same bytes
    staged = [t.clone() for t in cached]
    y = torch.empty((len(C), H), dtype=torch.bfloat16, device=DEV)
    qkv = torch.empty((len(C), 3 * heads * D), dtype=torch.bfloat16, device=DEV)
    tap = torch.empty((len(C), 3 * heads * D), dtype=torch.float32, device=DEV)
    lc.lacache_embed_rmsnorm(_i32(ids1[C]), _i32(C), dev_bf16(embed), dev_bf16(nw), staged[0], y)
    lc.lacache_linear_bf16(y, dev_bf16(wqkv), qkv, tap)
    lc.lacache_rope_scatter(qkv, _i32(C), torch.from_numpy(cos_t).to(DEV), torch.from_numpy(sin_t).to(DEV),
                            *staged[1:])
    torch.cuda.synchronize()
    for a, b in zip(full, staged):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    # against the oracle: the norm bit-exact, the projection within the bound,
    # RoPE bit-exact on the GPU's own projection
    x, ry = F.embed_norm(ids1[C], embed, nw)
    assert np.array_equal(host_bf16(y), ry)
    _linear_check(ry, wqkv, qkv, tap)
    g = host_bf16(qkv)
    for part, dst in enumerate(full[1:]):
        got = host_bf16(dst)
        for h in (0, heads - 1):
            blk = g[:, (part * heads + h) * D:(part * heads + h + 1) * D]
            ref = blk if part == 2 else F.rope(blk, C, cos_t, sin_t)
            assert np.array_equal(got[h, C], ref)
