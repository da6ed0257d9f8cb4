"""The C ABI on the host: every declared symbol is exported, and argument
validation returns the documented status before anything touches a GPU.

These run without a GPU: every call here fails validation (or is an M == 0
no-op), which the library decides before its first HIP call. The pointers are
fake, 16-byte aligned, non-overlapping addresses that are never dereferenced.
"""

import ctypes
import os
import re

import pytest

from paper_2607_16339_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OK, INVALID, UNSUP = _lib.LACACHE_OK, _lib.LACACHE_ERR_INVALID_ARG, _lib.LACACHE_ERR_UNSUPPORTED


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(_lib.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return _lib.lib()


def _declared_symbols():
    src = open(os.path.join(ROOT, "include", "lacache.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(lacache_\w+)\s*\(", src)))


def test_every_declared_symbol_is_exported(L):
    names = _declared_symbols()
    assert len(names) >= 12
    for n in names:
        assert hasattr(L, n), n
        assert n in _lib.SIGNATURES, n


class Fake:
    """Distinct aligned fake device addresses, 1 GiB apart."""

    def __init__(self):
        self.n = 0

    def __call__(self):
        self.n += 1
        return 0x10000000000 + self.n * (1 << 30)


def _ffn(L, M=32, H=4096, I=12288, group=128, **over):
    f = Fake()
    a = dict(x=f(), norm_w=f(), wgu_q=f(), wgu_s=f(), wd_q=f(), wd_s=f(), out=f())
    a.update(over)
    return L.lacache_ffn_fp8(None, a["x"], a["norm_w"], a["wgu_q"], a["wgu_s"], a["wd_q"], a["wd_s"], a["out"],
                             M, H, I, group)


def test_ffn_validation(L):
    assert _ffn(L, group=64) == UNSUP
    assert _ffn(L, H=4000) == INVALID
    assert _ffn(L, I=100) == INVALID
    assert _ffn(L, H=0) == INVALID
    assert _ffn(L, M=-1) == INVALID
    assert _ffn(L, H=16384 + 128) == UNSUP
    assert _ffn(L, I=65536 + 128) == UNSUP
    assert _ffn(L, M=(1 << 24) + 1) == UNSUP
    assert _ffn(L, x=None) == INVALID
    assert _ffn(L, out=0x10000000008) == INVALID  # misaligned
    x = 0x20000000000
    assert _ffn(L, x=x, out=x + 1024) == INVALID  # out overlaps x
    assert _ffn(L, M=0) == OK                    # no-op, nothing launched


def test_stage_validation(L):
    f = Fake()
    p = [f() for _ in range(8)]
    assert L.lacache_rmsnorm_quant(None, p[0], p[1], p[2], p[3], 4, 130, 128) == INVALID
    assert L.lacache_rmsnorm_quant(None, p[0], p[1], p[2], p[3], 0, 256, 128) == OK
    assert L.lacache_rmsnorm_quant(None, p[0], p[1], p[2], None, 4, 256, 128) == INVALID
    assert L.lacache_gateup_swiglu_quant(None, p[0], p[1], p[2], p[3], p[4], p[5], None, 4, 256, 768, 256) == UNSUP
    assert L.lacache_gateup_swiglu_quant(None, p[0], p[1], p[2], p[3], p[4], p[5], 0x8, 4, 256, 768, 128) == INVALID
    assert L.lacache_gateup_swiglu_quant(None, p[0], p[1], p[2], p[3], p[4], p[5], None, 0, 256, 768, 128) == OK
    # hq overlapping the weights
    assert L.lacache_gateup_swiglu_quant(None, p[0], p[1], p[2], p[3], p[2] + 4096, p[5], None, 4, 256, 768, 128) == INVALID
    assert L.lacache_down_proj(None, p[0], p[1], p[2], p[3], p[4], None, 4, 256, 700, 128) == INVALID
    assert L.lacache_down_proj(None, p[0], p[1], p[2], p[3], p[4], None, 0, 256, 768, 128) == OK
    assert L.lacache_quant_weights(None, p[0], p[1], p[2], 256, 200, 128) == INVALID
    assert L.lacache_quant_weights(None, p[0], p[0], p[2], 256, 256, 128) == INVALID  # w_q aliases w
    # row-major -> tile repack of weight codes
    assert L.lacache_pack_weights(None, p[0], p[1], 256, 200) == INVALID
    assert L.lacache_pack_weights(None, p[0], p[1], 0, 256) == INVALID
    assert L.lacache_pack_weights(None, p[0], p[0] + 1024, 256, 256) == INVALID  # overlap
    assert L.lacache_pack_weights(None, None, p[1], 256, 256) == INVALID
    assert L.lacache_pack_weights(None, p[0], p[1] + 8, 256, 256) == INVALID  # misaligned
    assert L.lacache_pack_weights(None, p[0], p[1], 256, 131072 + 128) == UNSUP
    assert L.lacache_add_bf16(None, p[0], p[0], 16) == INVALID
    assert L.lacache_add_bf16(None, p[0], p[1], 0) == OK
    assert L.lacache_add_bf16(None, p[0], p[1], -1) == INVALID
    assert L.lacache_encode_e4m3(None, p[0], p[1], 0) == OK
    assert L.lacache_encode_e4m3(None, p[0], None, 4) == INVALID


def test_addnorm_validation(L):
    f = Fake()
    p = [f() for _ in range(10)]
    # stage: resid += y, then norm + quant
    assert L.lacache_add_rmsnorm_quant(None, p[0], p[0], p[2], p[3], p[4], 4, 256, 128) == INVALID  # y is resid
    assert L.lacache_add_rmsnorm_quant(None, p[0], None, p[2], p[3], p[4], 4, 256, 128) == INVALID
    assert L.lacache_add_rmsnorm_quant(None, p[0], p[1], p[2], p[0] + 512, p[4], 4, 256, 128) == INVALID  # xq in resid
    assert L.lacache_add_rmsnorm_quant(None, p[0], p[1], p[2], p[3], p[4], 0, 256, 128) == OK
    assert L.lacache_add_rmsnorm_quant(None, p[0], p[1], p[2], p[3], p[4], 4, 256, 64) == UNSUP

    def fused(resid, y, out, M=32, group=128):
        return L.lacache_ffn_fp8_addnorm(None, resid, y, p[2], p[3], p[4], p[5], p[6], out, M, 4096, 12288, group)
    assert fused(p[0], p[1], p[7], group=64) == UNSUP
    assert fused(p[0], p[0], p[7]) == INVALID         # y is resid
    assert fused(p[0], p[1], p[1]) == INVALID         # out is y
    assert fused(p[0], p[1], p[0] + 1024) == INVALID  # out overlaps resid
    assert fused(p[0], None, p[7]) == INVALID
    assert fused(p[0], p[1], p[7], M=0) == OK


def test_facache_attention_validation(L):
    f = Fake()
    q, k, v, o, cm, cl, co, lse = (f() for _ in range(8))

    def att(heads=2, N=256, d=128, c0=64, c1=128, mode=0, **over):
        a = dict(q=q, k=k, v=v, o=o, lse=None, cm=cm, cl=cl, co=co)
        a.update(over)
        return L.lacache_facache_attention(None, a["q"], a["k"], a["v"], a["o"], a["lse"], a["cm"], a["cl"], a["co"],
                                           heads, N, d, c0, c1, mode)
    assert att(d=64) == UNSUP
    assert att(N=200, c1=100) == UNSUP          # N not a multiple of 64
    assert att(heads=4097) == UNSUP
    assert att(N=(1 << 20) + 64, c1=100) == UNSUP
    assert att(mode=3) == INVALID
    assert att(mode=-1) == INVALID
    assert att(heads=-1) == INVALID
    assert att(c0=130, c1=120) == INVALID       # c_begin > c_end
    assert att(c0=-1) == INVALID
    assert att(c1=257) == INVALID               # c_end > N
    assert att(q=None) == INVALID
    assert att(o=o + 8) == INVALID              # misaligned
    assert att(o=q + 4096) == INVALID           # o overlaps q
    assert att(cm=None) == INVALID              # populate needs the cache
    assert att(mode=1, co=None) == INVALID      # resume needs the cache
    assert att(mode=0, cl=k + 64) == INVALID    # cache written over k
    assert att(mode=1, cm=o + 64) == INVALID    # o written over the cache
    assert att(mode=0, co=cm) == INVALID        # two cache outputs alias
    assert att(lse=lse + 4) == INVALID          # misaligned lse
    assert att(mode=2, lse=v + 128) == INVALID  # lse written over v
    assert att(mode=1, lse=cl) == INVALID       # lse written over the cache it reads
    assert att(mode=0, lse=o + 256) == INVALID  # lse overlaps o
    assert att(heads=0) == OK and att(N=0, c0=0, c1=0) == OK  # nothing launched


def test_path_policy(L):
    assert L.lacache_set_path_policy(7) == INVALID
    prev = L.lacache_set_path_policy(1)
    try:
        f = Fake()
        p = [f() for _ in range(8)]
        # skinny kernels only take M <= 64
        assert L.lacache_gateup_swiglu_quant(None, p[0], p[1], p[2], p[3], p[4], p[5], None, 65, 256, 768, 128) == UNSUP
        assert L.lacache_down_proj(None, p[0], p[1], p[2], p[3], p[4], None, 65, 256, 768, 128) == UNSUP
        # ... whose activation rows fit the gate/up kernel's LDS (16 rows x 8192, 32 rows x 4096; 64 rows x
        # half of 4096) ...
        assert L.lacache_gateup_swiglu_quant(None, p[0], p[1], p[2], p[3], p[4], p[5], None, 17, 8192, 768, 128) == UNSUP
        assert L.lacache_gateup_swiglu_quant(None, p[0], p[1], p[2], p[3], p[4], p[5], None, 64, 4224, 768, 128) == UNSUP
        # ... and H <= 8192, I <= 16384 (the scales of a K range are staged in LDS)
        assert L.lacache_gateup_swiglu_quant(None, p[0], p[1], p[2], p[3], p[4], p[5], None, 8, 8320, 768, 128) == UNSUP
        assert L.lacache_down_proj(None, p[0], p[1], p[2], p[3], p[4], None, 8, 256, 16512, 128) == UNSUP
        assert L.lacache_set_path_policy(2) == 1
    finally:
        L.lacache_set_path_policy(prev)


def test_down_split_count_fills_one_round(L):
    """The tiled down GEMM's K splits (read back from the workspace size, whose
    largest part is the KS fp32 partials [KS][M][H]): with 128-row tiles and
    fewer tiles than the 256 CUs, as many splits as fit one round of one
    workgroup per CU, at most 6 (16 K-groups each at I = 12288)."""
    H, I = 4096, 12288

    def a256(b):
        return (b + 255) // 256 * 256
    for M in list(range(65, 2049, 37)) + [200, 320, 512, 576, 700, 1024, 1536]:
        rest = a256(M * H) + a256(H // 128 * M * 4) + a256(M * I) + a256(I // 128 * M * 4)
        scratch = L.lacache_ffn_workspace_bytes(M, H, I, 128) - rest
        ks = scratch // (M * H * 4)
        tiles = ((M + 127) // 128) * (H // 256)
        r256 = (((M + 255) // 256) * 16 + 255) // 256
        r128 = (((M + 127) // 128) * 16 + 255) // 256
        if r128 > r256 or tiles >= 256:
            assert scratch == 0, M  # 256-row tiles, or one round without a split
            continue
        if scratch == 0:
            ks = 1  # not split: no partials
        else:
            assert scratch == a256(ks * M * H * 4), M
        # the most splits that fit one round (capped at 6), never a second round
        assert 1 <= ks <= 6 and ks * tiles <= 256, (M, ks, tiles)
        assert ks == 6 or (ks + 1) * tiles > 256, (M, ks, tiles)


def test_workspace_bytes_and_status_strings(L):
    def a256(b):
        return (b + 255) // 256 * 256
    M, H, I = 32, 4096, 12288
    # one fp32 scratch buffer, big enough for either path of the shape: the
    # skinny gate/up h (M x I) or the tiled down GEMM's split-K partials
    # (16 output tiles -> 6 splits of 16 K-groups: 6 x M x H)
    scratch = max(a256(M * I * 4), a256(6 * M * H * 4))
    # (at 33..64 rows the skinny gate/up keeps the two K halves' gate and up sums: 2 x M x 2I)
    assert L.lacache_ffn_workspace_bytes(64, H, I, 128) == (
        max(a256(2 * 64 * 2 * I * 4), a256(6 * 64 * H * 4)) + a256(64 * H) + a256(H // 128 * 64 * 4)
        + a256(64 * I) + a256(I // 128 * 64 * 4))
    want = scratch + a256(M * H) + a256(H // 128 * M * 4) + a256(M * I) + a256(I // 128 * M * 4)
    assert L.lacache_ffn_workspace_bytes(M, H, I, 128) == want
    M = 512
    # the tiled down GEMM splits K 4 ways at M = 512 (64 output tiles): fp32 partials
    want = a256(4 * M * H * 4) + a256(M * H) + a256(H // 128 * M * 4) + a256(M * I) + a256(I // 128 * M * 4)
    assert L.lacache_ffn_workspace_bytes(M, H, I, 128) == want
    M = 8192  # enough tiles: no split, no scratch
    want = a256(M * H) + a256(H // 128 * M * 4) + a256(M * I) + a256(I // 128 * M * 4)
    assert L.lacache_ffn_workspace_bytes(M, H, I, 128) == want
    assert L.lacache_ffn_workspace_bytes(M, H, I, 64) == 0
    assert L.lacache_ffn_workspace_bytes(-1, H, I, 128) == 0
    for s, name in [(0, "LACACHE_OK"), (-1, "LACACHE_ERR_INVALID_ARG"), (-2, "LACACHE_ERR_UNSUPPORTED"),
                    (-3, "LACACHE_ERR_HIP"), (-4, "LACACHE_ERR_ALLOC"), (-5, "LACACHE_ERR_CAPTURE")]:
        assert L.lacache_status_string(s).decode() == name


def test_ws_variant_checks_workspace(L):
    f = Fake()
    p = [f() for _ in range(8)]
    args = [None] + p[:7] + [32, 4096, 12288, 128]
    need = L.lacache_ffn_workspace_bytes(32, 4096, 12288, 128)
    assert L.lacache_ffn_fp8_ws(*args, None, need) == INVALID
    assert L.lacache_ffn_fp8_ws(*args, f(), need - 1) == INVALID
    assert L.lacache_ffn_fp8_ws(*args, f() + 16, need) == INVALID  # not 256-byte aligned
    assert L.lacache_ffn_fp8_ws(*args, p[0], need) == INVALID      # overlaps x
    args0 = [None] + p[:7] + [0, 4096, 12288, 128]
    assert L.lacache_ffn_fp8_ws(*args0, None, 0) == OK             # M == 0: nothing to do


def test_noalloc_validation(L):
    """The allocation-free FFN call validates like lacache_ffn_fp8 and refuses,
    before any HIP call, a shape whose workspace exceeds its fixed array."""
    f = Fake()
    p = [f() for _ in range(8)]
    call = lambda M, H=4096, I=12288, g=128, ps=p: L.lacache_ffn_fp8_noalloc(None, *ps[:7], M, H, I, g)
    assert call(32, g=64) == UNSUP
    assert call(32, H=4000) == INVALID
    assert call(0) == OK
    assert call(32, ps=[None] + p[1:]) == INVALID
    assert L.lacache_ffn_workspace_bytes(8192, 4096, 12288, 128) > (64 << 20)
    assert call(8192) == UNSUP  # 129 MiB of workspace > the 64 MiB array
    assert all(L.lacache_ffn_workspace_bytes(M, 4096, 12288, 128) <= (64 << 20) for M in range(1, 1025))


def test_binding_refuses_host_tensors():
    import torch
    import paper_2607_16339_amd as lc
    x = torch.zeros(4, 256, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        lc.lacache_rmsnorm_quant(x, torch.zeros(256, dtype=torch.bfloat16), torch.zeros(4, 256, dtype=torch.uint8),
                                 torch.zeros(2, 4), stream=0)


def test_ctypes_signatures_cover_header():
    assert set(_declared_symbols()) == set(_lib.SIGNATURES)
    assert ctypes.sizeof(ctypes.c_void_p) == 8


def test_granularity_validation(L):
    f = Fake()
    w, wq, ws, wr = f(), f(), f(), f()
    # unknown granularity; null row scales; misaligned pointers; overlap
    assert L.lacache_quant_weights_g(None, w, wq, ws, wr, 256, 256, 3) == INVALID
    assert L.lacache_quant_weights_g(None, w, wq, ws, None, 256, 256, 1) == INVALID
    assert L.lacache_quant_weights_g(None, w, wq, ws, wr + 4, 256, 256, 2) == INVALID
    assert L.lacache_quant_weights_g(None, w, w, ws, wr, 256, 256, 1) == INVALID
    assert L.lacache_quant_weights_g(None, w, wq, ws, wr, 200, 256, 1) == INVALID
    # the group granularity is lacache_quant_weights (its own checks)
    assert L.lacache_quant_weights_g(None, w, wq, ws, None, 256, 200, 0) == INVALID
    # fp32 row quantization
    v, q, sk, sr = f(), f(), f(), f()
    assert L.lacache_quant_rows_g(None, v, q, sk, sr, 4, 256, -1) == INVALID
    assert L.lacache_quant_rows_g(None, v, q, sk, None, 4, 256, 2) == INVALID
    assert L.lacache_quant_rows_g(None, v, q, sk, sr, 4, 100, 1) == INVALID
    assert L.lacache_quant_rows_g(None, v, v, sk, sr, 4, 256, 1) == INVALID
    assert L.lacache_quant_rows_g(None, v, q, sk, sr, 0, 256, 1) == OK
    # the norm alone
    x, nw, y = f(), f(), f()
    assert L.lacache_rmsnorm_f32(None, x, nw, x, 4, 256) == INVALID
    assert L.lacache_rmsnorm_f32(None, x, nw, y, 4, 200) == INVALID
    assert L.lacache_rmsnorm_f32(None, x, nw, y, 0, 256) == OK
    # gate/up without re-quantization and down with row scales
    xq, xs, gq, gs, gr, h = f(), f(), f(), f(), f(), f()
    assert L.lacache_gateup_swiglu_f32(None, xq, xs, gq, gs, gr, h, 4, 256, 384, 64) == UNSUP
    assert L.lacache_gateup_swiglu_f32(None, xq, xs, gq, gs, gr, xq, 4, 256, 384, 128) == INVALID
    assert L.lacache_gateup_swiglu_f32(None, xq, xs, gq, gs, gr + 4, h, 4, 256, 384, 128) == INVALID
    assert L.lacache_gateup_swiglu_f32(None, xq, xs, gq, gs, None, h, 0, 256, 384, 128) == OK
    hq, hs, dq, ds, dr, out = f(), f(), f(), f(), f(), f()
    assert L.lacache_down_proj_g(None, hq, hs, dq, ds, dr, hq, None, 4, 256, 384, 128) == INVALID
    assert L.lacache_down_proj_g(None, hq, hs, dq, ds, dr + 8, out, None, 4, 256, 384, 128) == INVALID
    assert L.lacache_down_proj_g(None, hq, hs, dq, ds, None, out, None, 0, 256, 384, 128) == OK
    # the whole FFN at a granularity
    a = [f() for _ in range(10)]
    assert L.lacache_ffn_fp8_g(None, *a, 32, 256, 384, 5) == INVALID
    assert L.lacache_ffn_fp8_g(None, a[0], a[1], a[2], a[3], None, a[5], a[6], a[7], a[8], 32, 256, 384, 1) == INVALID
    assert L.lacache_ffn_fp8_g(None, a[0], a[1], a[2], a[3], a[4], a[5], a[6], a[7], a[0], 32, 256, 384, 2) == INVALID
    assert L.lacache_ffn_fp8_g(None, *a[:9], 0, 256, 384, 1) == OK
    assert L.lacache_ffn_g_workspace_bytes(32, 256, 384) > 0
    assert L.lacache_ffn_g_workspace_bytes(32, 200, 384) == 0


def test_first_layer_validation(L):
    f = Fake()
    ids, rows, emb, nw, cache, y = f(), f(), f(), f(), f(), f()
    assert L.lacache_embed_rmsnorm(None, ids, rows, -1, emb, 100, nw, cache, 64, y, 256) == INVALID
    assert L.lacache_embed_rmsnorm(None, ids, rows, 4, emb, 0, nw, cache, 64, y, 256) == INVALID
    assert L.lacache_embed_rmsnorm(None, ids, rows, 4, emb, 100, nw, cache, 64, y, 200) == INVALID
    assert L.lacache_embed_rmsnorm(None, ids, rows, 4, emb, 100, nw, emb, 64, y, 256) == INVALID
    assert L.lacache_embed_rmsnorm(None, ids + 4, rows, 4, emb, 100, nw, cache, 64, y, 256) == INVALID
    assert L.lacache_embed_rmsnorm(None, ids, rows, 0, emb, 100, nw, cache, 64, y, 256) == OK
    a, w, out = f(), f(), f()
    assert L.lacache_linear_bf16(None, a, w, out, None, 4, 384, 200) == INVALID
    assert L.lacache_linear_bf16(None, a, w, a, None, 4, 384, 256) == INVALID
    assert L.lacache_linear_bf16(None, a, w, out, out + 4, 4, 384, 256) == INVALID
    assert L.lacache_linear_bf16(None, a, w, out, None, 0, 384, 256) == OK
    qkv, cs, sn, q, k, v = f(), f(), f(), f(), f(), f()
    assert L.lacache_rope_scatter(None, qkv, rows, 4, cs, sn, q, k, v, 0, 64) == INVALID
    assert L.lacache_rope_scatter(None, qkv, rows, 4, cs, sn, q, q, v, 2, 64) == INVALID
    assert L.lacache_rope_scatter(None, qkv, rows, 4, cs, sn, q, k, v, 5000, 64) == UNSUP
    assert L.lacache_rope_scatter(None, qkv, rows, 0, cs, sn, q, k, v, 2, 64) == OK
    wq = f()
    assert L.lacache_first_layer_tokens(None, ids, rows, 4, emb, 100, nw, wq, cs, sn, cache, q, k, v, 2, 64, 200) \
        == INVALID
    assert L.lacache_first_layer_tokens(None, ids, rows, 4, emb, 100, nw, wq, cs, sn, q, q, k, v, 2, 64, 256) \
        == INVALID
    assert L.lacache_first_layer_tokens(None, ids, rows, 0, emb, 100, nw, wq, cs, sn, cache, q, k, v, 2, 64, 256) == OK
    assert L.lacache_first_layer_workspace_bytes(32, 32, 4096) > 0


def test_weight_tile_layout_helpers():
    """weight_codes_rowmajor / weight_codes_tiled against positions of the
    tile layout worked out by hand, and as inverses of each other."""
    import numpy as np
    import paper_2607_16339_amd as lc
    N, K = 48, 384  # 3 slabs of 16 rows x 3 K-groups
    rm = np.arange(N * K, dtype=np.int64).reshape(N, K)
    codes = (rm % 251).astype(np.uint8)
    t = lc.weight_codes_tiled(codes).reshape(-1)
    # W[0, 0..63] is the first 64 bytes; W[1, 0] follows them; W[0, 64] opens
    # the tile's second kilobyte; W[0, 128] opens the next tile (same slab)
    assert np.array_equal(t[:64], codes[0, :64])
    assert t[64] == codes[1, 0] and t[15 * 64 + 63] == codes[15, 63]
    assert t[1024] == codes[0, 64] and t[1024 + 64 * 3 + 5] == codes[3, 69]
    assert t[2048] == codes[0, 128] and t[2 * 2048 + 1024 + 7] == codes[0, 256 + 64 + 7]
    # the second slab starts at byte 16 K, as in a row-major matrix
    assert t[16 * K] == codes[16, 0] and t[16 * K + 64 * 15 + 1] == codes[31, 1]
    # every position: the formula of include/lacache.h
    n, k = np.meshgrid(np.arange(N), np.arange(K), indexing="ij")
    off = ((n // 16) * (K // 128) + k // 128) * 2048 + ((k // 64) % 2) * 1024 + (n % 16) * 64 + k % 64
    assert np.array_equal(t[off], codes)
    assert np.array_equal(lc.weight_codes_rowmajor(t.reshape(N, K)), codes)
