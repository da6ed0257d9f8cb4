"""MI355X (gfx950) per-group FP8 FFN of LaCache (arxiv 2607.16339, Sec. 3.4).

The Python functions carry the names of the C ABI (include/lacache.h) and take
torch device tensors; they check dtypes, devices and shapes, derive the sizes,
pass raw pointers and the current HIP stream, and raise ``LacacheError`` on a
non-OK status. Every step of the FFN runs in the library's HIP kernels.
"""

import numpy as np
import torch

from ._lib import (LACACHE_ERR_ALLOC, LACACHE_ERR_CAPTURE, LACACHE_ERR_HIP, LACACHE_ERR_INVALID_ARG,  # noqa: F401
                   LACACHE_ERR_UNSUPPORTED, LACACHE_GRAN_GROUP, LACACHE_GRAN_TENSOR, LACACHE_GRAN_TOKEN, LACACHE_OK,
                   LacacheError, check, lib, status_string)

GROUP = 128
_U8 = (torch.uint8, torch.float8_e4m3fn)
_BF16 = (torch.bfloat16, torch.int16, torch.uint16)


def _stream(stream, *tensors):
    if stream is not None:
        return int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)
    dev = tensors[0].device if tensors else None
    return int(torch.cuda.current_stream(dev).cuda_stream)


def _ptr(t, dtypes, name, shape=None, optional=False):
    if t is None:
        if optional:
            return None
        raise ValueError("%s is required" % name)
    if t.device.type != "cuda":
        raise ValueError("%s must be a device tensor" % name)
    if t.dtype not in dtypes:
        raise ValueError("%s: dtype %s not in %s" % (name, t.dtype, dtypes))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("%s: shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))
    return t.data_ptr()


def lacache_quant_weights(w, w_q, w_s, group=GROUP, stream=None):
    """128x128 block quantization: w [N, K] bf16 -> w_q [N, K] e4m3, w_s [N/128, K/128] fp32."""
    N, K = w.shape
    check(lib().lacache_quant_weights(
        _stream(stream, w), _ptr(w, _BF16, "w"), _ptr(w_q, _U8, "w_q", (N, K)),
        _ptr(w_s, (torch.float32,), "w_s", (N // group, K // group)), N, K, group), "lacache_quant_weights")


def lacache_pack_weights(w_q_rowmajor, w_q, stream=None):
    """Row-major e4m3 codes [N, K] -> w_q [N, K] in the library's weight tile layout (on the device)."""
    N, K = w_q_rowmajor.shape
    check(lib().lacache_pack_weights(_stream(stream, w_q_rowmajor), _ptr(w_q_rowmajor, _U8, "w_q_rowmajor"),
                                     _ptr(w_q, _U8, "w_q", (N, K)), N, K), "lacache_pack_weights")


def lacache_rmsnorm_quant(x, norm_w, xq, xs, group=GROUP, stream=None):
    """x [M, H] bf16, norm_w [H] -> xq [M, H] e4m3, xs [H/128, M] fp32."""
    M, H = x.shape
    check(lib().lacache_rmsnorm_quant(
        _stream(stream, x), _ptr(x, _BF16, "x"), _ptr(norm_w, _BF16, "norm_w", (H,)), _ptr(xq, _U8, "xq", (M, H)),
        _ptr(xs, (torch.float32,), "xs", (H // group, M)), M, H, group), "lacache_rmsnorm_quant")


def lacache_add_rmsnorm_quant(resid, y, norm_w, xq, xs, group=GROUP, stream=None):
    """resid [M, H] bf16 += y (in place, nearest-even), then the norm + quantization of resid."""
    M, H = resid.shape
    check(lib().lacache_add_rmsnorm_quant(
        _stream(stream, resid), _ptr(resid, _BF16, "resid"), _ptr(y, _BF16, "y", (M, H)),
        _ptr(norm_w, _BF16, "norm_w", (H,)), _ptr(xq, _U8, "xq", (M, H)),
        _ptr(xs, (torch.float32,), "xs", (H // group, M)), M, H, group), "lacache_add_rmsnorm_quant")


def lacache_gateup_swiglu_quant(xq, xs, wgu_q, wgu_s, hq, hs, h_tap=None, group=GROUP, stream=None):
    """xq [M, H], wgu_q [2I, H] -> hq [M, I] e4m3, hs [I/128, M] fp32 (h_tap [M, I] fp32 optional)."""
    M, H = xq.shape
    I = wgu_q.shape[0] // 2
    check(lib().lacache_gateup_swiglu_quant(
        _stream(stream, xq), _ptr(xq, _U8, "xq"), _ptr(xs, (torch.float32,), "xs", (H // group, M)),
        _ptr(wgu_q, _U8, "wgu_q", (2 * I, H)), _ptr(wgu_s, (torch.float32,), "wgu_s", (2 * I // group, H // group)),
        _ptr(hq, _U8, "hq", (M, I)), _ptr(hs, (torch.float32,), "hs", (I // group, M)),
        _ptr(h_tap, (torch.float32,), "h_tap", (M, I), optional=True), M, H, I, group),
        "lacache_gateup_swiglu_quant")


def lacache_down_proj(hq, hs, wd_q, wd_s, out, out_tap=None, group=GROUP, stream=None):
    """hq [M, I], wd_q [H, I] -> out [M, H] bf16 (out_tap [M, H] fp32 optional)."""
    M, I = hq.shape
    H = wd_q.shape[0]
    check(lib().lacache_down_proj(
        _stream(stream, hq), _ptr(hq, _U8, "hq"), _ptr(hs, (torch.float32,), "hs", (I // group, M)),
        _ptr(wd_q, _U8, "wd_q", (H, I)), _ptr(wd_s, (torch.float32,), "wd_s", (H // group, I // group)),
        _ptr(out, _BF16, "out", (M, H)), _ptr(out_tap, (torch.float32,), "out_tap", (M, H), optional=True),
        M, H, I, group), "lacache_down_proj")


def _ffn_args(x, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, group):
    M, H = x.shape
    I = wd_q.shape[1]
    return [_ptr(x, _BF16, "x"), _ptr(norm_w, _BF16, "norm_w", (H,)), _ptr(wgu_q, _U8, "wgu_q", (2 * I, H)),
            _ptr(wgu_s, (torch.float32,), "wgu_s", (2 * I // group, H // group)), _ptr(wd_q, _U8, "wd_q", (H, I)),
            _ptr(wd_s, (torch.float32,), "wd_s", (H // group, I // group)), _ptr(out, _BF16, "out", (M, H)),
            M, H, I, group]


def lacache_ffn_fp8(x, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, group=GROUP, stream=None):
    """The whole FP8 FFN of one layer: x [M, H] bf16 -> out [M, H] bf16."""
    check(lib().lacache_ffn_fp8(_stream(stream, x), *_ffn_args(x, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, group)),
          "lacache_ffn_fp8")


def lacache_ffn_fp8_noalloc(x, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, group=GROUP, stream=None):
    """lacache_ffn_fp8 with its workspace in the library's fixed device array: allocates nothing."""
    check(lib().lacache_ffn_fp8_noalloc(_stream(stream, x),
                                        *_ffn_args(x, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, group)),
          "lacache_ffn_fp8_noalloc")


def lacache_ffn_fp8_addnorm(resid, y, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, group=GROUP, stream=None):
    """resid += y (in place), then out = the FP8 FFN of resid."""
    args = _ffn_args(resid, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, group)
    check(lib().lacache_ffn_fp8_addnorm(_stream(stream, resid), args[0], _ptr(y, _BF16, "y", tuple(resid.shape)),
                                        *args[1:]), "lacache_ffn_fp8_addnorm")


def lacache_ffn_workspace_bytes(M, H, I, group=GROUP):
    return int(lib().lacache_ffn_workspace_bytes(M, H, I, group))


def lacache_ffn_fp8_ws(x, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, workspace, group=GROUP, stream=None):
    """lacache_ffn_fp8 with a caller-owned uint8 workspace tensor."""
    check(lib().lacache_ffn_fp8_ws(_stream(stream, x), *_ffn_args(x, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, group),
                                   _ptr(workspace, (torch.uint8,), "workspace"), workspace.numel()),
          "lacache_ffn_fp8_ws")


def lacache_add_bf16(x_inout, y, stream=None):
    """x_inout += y in bf16 (fp32 add, nearest-even rounding)."""
    check(lib().lacache_add_bf16(_stream(stream, x_inout), _ptr(x_inout, _BF16, "x_inout"),
                                 _ptr(y, _BF16, "y", tuple(x_inout.shape)), x_inout.numel()), "lacache_add_bf16")


def lacache_encode_e4m3(v, codes, stream=None):
    """Device e4m3 encoder (test hook): codes = E(v), elementwise."""
    check(lib().lacache_encode_e4m3(_stream(stream, v), _ptr(v, (torch.float32,), "v"),
                                    _ptr(codes, _U8, "codes", tuple(v.shape)), v.numel()), "lacache_encode_e4m3")


def lacache_facache_attention(q, k, v, o, lse=None, cache_m=None, cache_l=None, cache_o=None, c_begin=0, c_end=0,
                              mode=2, stream=None):
    """q, k, v, o: [heads, N, d] bf16; lse [heads, N] fp32 or None; cache_m,
    cache_l [heads, N] and cache_o [heads, N, d] fp32 (modes 0 populate and
    1 resume; unused in mode 2)."""
    heads, N, d = q.shape
    cache = mode in (0, 1)
    f32 = (torch.float32,)
    check(lib().lacache_facache_attention(
        _stream(stream, q), _ptr(q, _BF16, "q"), _ptr(k, _BF16, "k", (heads, N, d)), _ptr(v, _BF16, "v", (heads, N, d)),
        _ptr(o, _BF16, "o", (heads, N, d)), _ptr(lse, f32, "lse", (heads, N), optional=True),
        _ptr(cache_m, f32, "cache_m", (heads, N), optional=not cache),
        _ptr(cache_l, f32, "cache_l", (heads, N), optional=not cache),
        _ptr(cache_o, f32, "cache_o", (heads, N, d), optional=not cache), heads, N, d, c_begin, c_end, mode),
        "lacache_facache_attention")


# ---- coarse quantization granularities (per token, per tensor) ------------

_F32 = (torch.float32,)


def lacache_quant_weights_g(w, w_q, w_s, w_row_s, granularity, stream=None):
    """Weight quantization at a granularity: w [N, K] bf16 -> w_q [N, K], w_s
    [N/128, K/128] (1.0 for token/tensor), w_row_s [N] (token/tensor)."""
    N, K = w.shape
    check(lib().lacache_quant_weights_g(
        _stream(stream, w), _ptr(w, _BF16, "w"), _ptr(w_q, _U8, "w_q", (N, K)),
        _ptr(w_s, _F32, "w_s", (N // GROUP, K // GROUP)),
        _ptr(w_row_s, _F32, "w_row_s", (N,), optional=granularity == LACACHE_GRAN_GROUP), N, K, granularity),
        "lacache_quant_weights_g")


def lacache_rmsnorm_f32(x, norm_w, y, stream=None):
    """y [M, H] fp32 = RMSNorm(x) with the fused quantizer's arithmetic."""
    M, H = x.shape
    check(lib().lacache_rmsnorm_f32(_stream(stream, x), _ptr(x, _BF16, "x"), _ptr(norm_w, _BF16, "norm_w", (H,)),
                                    _ptr(y, _F32, "y", (M, H)), M, H), "lacache_rmsnorm_f32")


def lacache_quant_rows_g(v, q, s_kgm, s_rows, granularity, stream=None):
    """fp32 rows v [M, K] -> codes q [M, K], scales s_kgm [K/128, M], row scales s_rows [M]."""
    M, K = v.shape
    check(lib().lacache_quant_rows_g(
        _stream(stream, v), _ptr(v, _F32, "v"), _ptr(q, _U8, "q", (M, K)), _ptr(s_kgm, _F32, "s_kgm", (K // GROUP, M)),
        _ptr(s_rows, _F32, "s_rows", (M,), optional=granularity == LACACHE_GRAN_GROUP), M, K, granularity),
        "lacache_quant_rows_g")


def lacache_gateup_swiglu_f32(xq, xs, wgu_q, wgu_s, wgu_row_s, h, group=GROUP, stream=None):
    """h [M, I] fp32 = SiLU(g) u without re-quantization; wgu_row_s [2I] or None."""
    M, H = xq.shape
    I = h.shape[1]
    check(lib().lacache_gateup_swiglu_f32(
        _stream(stream, xq), _ptr(xq, _U8, "xq"), _ptr(xs, _F32, "xs", (H // group, M)),
        _ptr(wgu_q, _U8, "wgu_q", (2 * I, H)), _ptr(wgu_s, _F32, "wgu_s", (2 * I // group, H // group)),
        _ptr(wgu_row_s, _F32, "wgu_row_s", (2 * I,), optional=True), _ptr(h, _F32, "h", (M, I)), M, H, I, group),
        "lacache_gateup_swiglu_f32")


def lacache_down_proj_g(hq, hs, wd_q, wd_s, wd_row_s, out, out_tap=None, group=GROUP, stream=None):
    """lacache_down_proj with per-column weight scales wd_row_s [H] (or None)."""
    M, I = hq.shape
    H = out.shape[1]
    check(lib().lacache_down_proj_g(
        _stream(stream, hq), _ptr(hq, _U8, "hq"), _ptr(hs, _F32, "hs", (I // group, M)),
        _ptr(wd_q, _U8, "wd_q", (H, I)), _ptr(wd_s, _F32, "wd_s", (H // group, I // group)),
        _ptr(wd_row_s, _F32, "wd_row_s", (H,), optional=True), _ptr(out, _BF16, "out", (M, H)),
        _ptr(out_tap, _F32, "out_tap", (M, H), optional=True), M, H, I, group), "lacache_down_proj_g")


def lacache_ffn_fp8_g(x, norm_w, wgu_q, wgu_s, wgu_row_s, wd_q, wd_s, wd_row_s, out, granularity, stream=None):
    """The whole FFN at a granularity (weights from lacache_quant_weights_g)."""
    M, H = x.shape
    I = wd_q.shape[1]
    opt = granularity == LACACHE_GRAN_GROUP
    check(lib().lacache_ffn_fp8_g(
        _stream(stream, x), _ptr(x, _BF16, "x"), _ptr(norm_w, _BF16, "norm_w", (H,)),
        _ptr(wgu_q, _U8, "wgu_q", (2 * I, H)), _ptr(wgu_s, _F32, "wgu_s", (2 * I // GROUP, H // GROUP)),
        _ptr(wgu_row_s, _F32, "wgu_row_s", (2 * I,), optional=opt), _ptr(wd_q, _U8, "wd_q", (H, I)),
        _ptr(wd_s, _F32, "wd_s", (H // GROUP, I // GROUP)), _ptr(wd_row_s, _F32, "wd_row_s", (H,), optional=opt),
        _ptr(out, _BF16, "out", (M, H)), M, H, I, granularity), "lacache_ffn_fp8_g")


def lacache_ffn_g_workspace_bytes(M, H, I):
    return int(lib().lacache_ffn_g_workspace_bytes(M, H, I))


def quantize_weights_g(w, granularity, stream=None):
    """Returns (w_q, w_s, w_row_s) for a bf16 weight at a granularity (w_row_s None for GROUP);
    w_q is in the tile layout (weight_codes_rowmajor)."""
    N, K = w.shape
    w_q = torch.empty((N, K), dtype=torch.uint8, device=w.device)
    w_s = torch.empty((N // GROUP, K // GROUP), dtype=torch.float32, device=w.device)
    w_row_s = None if granularity == LACACHE_GRAN_GROUP else torch.empty((N,), dtype=torch.float32, device=w.device)
    lacache_quant_weights_g(w, w_q, w_s, w_row_s, granularity, stream)
    return w_q, w_s, w_row_s


# ---- token-wise first layer (EmbedCache, RoPECache) -------------------------

_I32 = (torch.int32,)


def lacache_embed_rmsnorm(token_ids, rows, embed, norm_w, embed_cache, y, stream=None):
    """token_ids, rows [R] int32; embed [vocab, H] bf16 -> embed_cache rows, y [R, H] bf16."""
    R = token_ids.shape[0]
    vocab, H = embed.shape
    N = embed_cache.shape[0]
    check(lib().lacache_embed_rmsnorm(
        _stream(stream, embed), _ptr(token_ids, _I32, "token_ids", (R,)), _ptr(rows, _I32, "rows", (R,)), R,
        _ptr(embed, _BF16, "embed"), vocab, _ptr(norm_w, _BF16, "norm_w", (H,)),
        _ptr(embed_cache, _BF16, "embed_cache", (N, H)), N, _ptr(y, _BF16, "y", (R, H)), H), "lacache_embed_rmsnorm")


def lacache_linear_bf16(a, w, out, out_tap=None, stream=None):
    """out [M, N] bf16 = a [M, K] w[N, K]^T (fp32 accumulation)."""
    M, K = a.shape
    N = w.shape[0]
    check(lib().lacache_linear_bf16(
        _stream(stream, a), _ptr(a, _BF16, "a"), _ptr(w, _BF16, "w", (N, K)), _ptr(out, _BF16, "out", (M, N)),
        _ptr(out_tap, _F32, "out_tap", (M, N), optional=True), M, N, K), "lacache_linear_bf16")


def lacache_rope_scatter(qkv, rows, rope_cos, rope_sin, q, k, v, stream=None):
    """qkv [R, 3 heads 128] bf16 -> RoPE(Q, K) and V scattered to rows of q, k, v [heads, N, 128]."""
    R = qkv.shape[0]
    heads, N, d = q.shape
    check(lib().lacache_rope_scatter(
        _stream(stream, qkv), _ptr(qkv, _BF16, "qkv", (R, 3 * heads * d)), _ptr(rows, _I32, "rows", (R,)), R,
        _ptr(rope_cos, _F32, "rope_cos", (N, 64)), _ptr(rope_sin, _F32, "rope_sin", (N, 64)),
        _ptr(q, _BF16, "q"), _ptr(k, _BF16, "k", (heads, N, d)), _ptr(v, _BF16, "v", (heads, N, d)), heads, N),
        "lacache_rope_scatter")


def lacache_first_layer_tokens(token_ids, rows, embed, norm_w, w_qkv, rope_cos, rope_sin, embed_cache, q, k, v,
                               stream=None):
    """The token-wise first layer for the given rows: embedding + norm, QKV projection, RoPE + scatter."""
    R = token_ids.shape[0]
    vocab, H = embed.shape
    heads, N, d = q.shape
    check(lib().lacache_first_layer_tokens(
        _stream(stream, embed), _ptr(token_ids, _I32, "token_ids", (R,)), _ptr(rows, _I32, "rows", (R,)), R,
        _ptr(embed, _BF16, "embed"), vocab, _ptr(norm_w, _BF16, "norm_w", (H,)),
        _ptr(w_qkv, _BF16, "w_qkv", (3 * heads * d, H)), _ptr(rope_cos, _F32, "rope_cos", (N, 64)),
        _ptr(rope_sin, _F32, "rope_sin", (N, 64)), _ptr(embed_cache, _BF16, "embed_cache", (N, H)),
        _ptr(q, _BF16, "q"), _ptr(k, _BF16, "k", (heads, N, d)), _ptr(v, _BF16, "v", (heads, N, d)), heads, N, H),
        "lacache_first_layer_tokens")


def lacache_set_path_policy(policy):
    """0 = automatic, 1 = skinny kernels (M <= 64), 2 = tiled kernels. Returns the previous policy."""
    r = lib().lacache_set_path_policy(int(policy))
    if r < 0:
        raise LacacheError(r, "lacache_set_path_policy")
    return r


def lacache_status_string(status):
    return status_string(status)


def lacache_release_workspace():
    lib().lacache_release_workspace()


# ---- allocation conveniences (torch allocates; the library computes) -------

def weight_codes_rowmajor(w_q):
    """Host copy of FP8 weight codes in row-major order: a numpy uint8 [N, K]
    array whose element (n, k) is the code of W[n, k].

    The library stores the codes of W [N x K] in 16-row x 128-column tiles of
    2 KB (the layout its kernels stream, described with lacache_quant_weights
    in include/lacache.h): tile (n/16, k/128) at byte
    ((n/16)(K/128) + k/128) 2048, columns 0..63 of its 16 rows in the first
    1 KB (64 bytes per row), columns 64..127 in the second. A host-side
    reordering for inspection; the kernels never need it.
    """
    a = w_q.cpu().numpy() if torch.is_tensor(w_q) else np.asarray(w_q)
    a = a.view(np.uint8) if a.dtype != np.uint8 else a
    N, K = a.shape
    return np.ascontiguousarray(a.reshape(N // 16, K // 128, 2, 16, 64).transpose(0, 3, 1, 2, 4).reshape(N, K))


def weight_codes_tiled(codes):
    """The inverse of weight_codes_rowmajor: row-major codes [N, K] -> the
    library's tile layout (a numpy uint8 array of the same shape)."""
    a = np.asarray(codes, dtype=np.uint8)
    N, K = a.shape
    return np.ascontiguousarray(a.reshape(N // 16, 16, K // 128, 2, 64).transpose(0, 2, 3, 1, 4).reshape(N, K))


def pack_weights(w_q_rowmajor, stream=None):
    """Returns the tile-layout copy of row-major e4m3 weight codes [N, K] (a new device tensor)."""
    w_q = torch.empty(tuple(w_q_rowmajor.shape), dtype=torch.uint8, device=w_q_rowmajor.device)
    lacache_pack_weights(w_q_rowmajor, w_q, stream)
    return w_q


def quantize_weights(w, group=GROUP, stream=None):
    """Returns (w_q uint8 [N, K] in the tile layout, w_s fp32 [N/128, K/128]) for a bf16 weight."""
    N, K = w.shape
    w_q = torch.empty((N, K), dtype=torch.uint8, device=w.device)
    w_s = torch.empty((N // group, K // group), dtype=torch.float32, device=w.device)
    lacache_quant_weights(w, w_q, w_s, group, stream)
    return w_q, w_s


def ffn_fp8(x, norm_w, wgu_q, wgu_s, wd_q, wd_s, group=GROUP, stream=None):
    """Allocates out and runs lacache_ffn_fp8."""
    out = torch.empty(x.shape, dtype=torch.bfloat16, device=x.device)
    lacache_ffn_fp8(x, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, group, stream)
    return out
