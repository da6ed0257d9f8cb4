/*
 * lacache.h -- C ABI of the MI355X (gfx950) per-group FP8 FFN.
 *
 * The library implements the mixed-precision FFN that LaCache (arxiv
 * 2607.16339) applies to every transformer layer except the first (Sec. 3.4):
 *
 *   x (bf16) -> RMSNorm fused with 1x128 e4m3 quantization     (Sec. 3.4, "AddNorm")
 *            -> FP8 gate/up GEMM with per-group dequantization  (Sec. 3.4, Eqs. 7-8)
 *            -> SwiGLU fused with 1x128 e4m3 re-quantization    (Sec. 3.4, "Swiglu")
 *            -> FP8 down GEMM with per-group dequantization -> out (bf16)
 *
 * Activations are quantized in groups of 128 consecutive elements of a row
 * and weights in 128x128 blocks (Sec. 3.4): scale = max|x| / 448 (Eq. 8),
 * code = e4m3(x / scale) with clipping to +-448 (Eq. 7). FP8 is OCP e4m3fn
 * (bias 7, max 448, no infinities); rounding is to nearest, ties to even; the
 * scale is an fp32 value rounded once from amax / 448 and x / scale is a
 * correctly rounded fp32 division. A group whose scale is 0 gets codes 0x00.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers are device pointers on the current HIP device, unless stated.
 *   bf16 values are passed as uint16_t bit patterns, e4m3 codes as uint8_t,
 *   scales as fp32. Row-major, last index contiguous.
 * - stream is a hipStream_t passed as void*; NULL means the null stream.
 *   Every call is asynchronous on that stream: it returns after enqueueing,
 *   with no host or device synchronization.
 * - group must be 128 (the paper fixes 1x128 and 128x128); any other value
 *   returns LACACHE_ERR_UNSUPPORTED. Dimensions H, I (and N, K) must be
 *   positive multiples of 128; M >= 0. M == 0 (n == 0) returns LACACHE_OK after
 *   the shape checks, launches nothing and does not look at the pointers.
 *   Size limits: H <= 16384, I <= 65536, M <= 2^24.
 * - Every argument is checked on the host before anything is launched; on
 *   error nothing is launched and no output is written. Pointers must be
 *   non-NULL (except the optional *_tap outputs) and 16-byte aligned.
 *   Outputs must not overlap inputs.
 * - The caller owns every buffer it passes. The library owns only its
 *   workspace: the intermediates of lacache_ffn_fp8 and the fp32 scratch of
 *   the GEMM stage calls (see lacache_ffn_fp8). The workspace is one buffer
 *   per device, allocated on first use and grown (by at least half) when a
 *   larger call needs it. A superseded buffer is not freed until
 *   lacache_release_workspace(), so work queued on any stream, and HIP graphs
 *   captured earlier, keep valid memory; growth never synchronizes.
 * - Stream capture (HIP graphs): a call whose stream is being captured must
 *   not need a larger library workspace than earlier calls have made the
 *   library allocate; it then returns LACACHE_ERR_CAPTURE and enqueues
 *   nothing (the capture stays valid). Call the largest shape once outside
 *   capture first, or use lacache_ffn_fp8_ws with a caller-owned workspace.
 *   Graphs that hold library-workspace calls become invalid at
 *   lacache_release_workspace().
 * - Results are deterministic: the same inputs give the same output bytes
 *   (no floating-point atomics).
 * - A failed HIP launch or allocation returns LACACHE_ERR_HIP or
 *   LACACHE_ERR_ALLOC; lacache_status_string() names any status.
 */
#ifndef LACACHE_H
#define LACACHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LACACHE_OK = 0,
  LACACHE_ERR_INVALID_ARG = -1, /* null/misaligned pointer, bad shape, overlap */
  LACACHE_ERR_UNSUPPORTED = -2, /* group != 128, or a size above the limits */
  LACACHE_ERR_HIP = -3,         /* a HIP runtime call or kernel launch failed */
  LACACHE_ERR_ALLOC = -4,       /* the library could not allocate its workspace */
  LACACHE_ERR_CAPTURE = -5      /* the library workspace would have to grow while the
                                   stream is being captured (see the conventions) */
} lacache_status;

/*
 * 128x128 block quantization of a bf16 weight (Sec. 3.4, Eqs. 7-8).
 *   w   [N x K] bf16               (input)
 *   w_q N*K e4m3 codes             (output) in the weight tile layout below
 *   w_s [N/128 x K/128] fp32       (output) block (nb, kb) covers rows
 *                                  nb*128.. and columns kb*128..
 * For the FFN, the gate/up weight is the row concatenation [W_gate; W_up]
 * ([2I x H], gate rows first) and the down weight is W_down [H x I].
 *
 * Weight tile layout (every e4m3 weight argument of this library): the code
 * of W[n, k] sits at byte
 *   ((n/16) (K/128) + k/128) 2048 + ((k/64) mod 2) 1024 + (n mod 16) 64 + k mod 64,
 * i.e. 16-row x 128-column tiles of 2 KB, a 16-row slab's tiles in K order
 * (the slab starts at byte 16 (n/16) K, as in a row-major matrix), and in a
 * tile first columns 0..63 of its 16 rows (64 bytes per row), then columns
 * 64..127. The MFMA operand of a slab and K-group is then two contiguous
 * 1 KB runs, so the weight-streaming kernels load 1 KB per instruction.
 * The codes themselves are those of the row-major statement of Eqs. 7-8.
 */
int lacache_quant_weights(void* stream, const uint16_t* w, uint8_t* w_q, float* w_s,
                          int64_t N, int64_t K, int group);

/*
 * Repack of e4m3 weight codes from row-major order into the weight tile
 * layout above, for weights quantized by another producer (the codes of
 * Eqs. 7-8 in the row-major [N x K] order of Sec. 3.4's statement; the block
 * scales [N/128 x K/128] need no repack).
 *   w_q_rowmajor [N x K] e4m3, row-major   (input)
 *   w_q          N*K e4m3, tile layout     (output), must not overlap the input
 * N and K must be positive multiples of 128 (N, K <= 131072). Every weight
 * code argument of the FFN calls below must be in the tile layout: row-major
 * codes passed there directly are the same size, so the library cannot tell
 * them apart, and give wrong results.
 */
int lacache_pack_weights(void* stream, const uint8_t* w_q_rowmajor, uint8_t* w_q, int64_t N, int64_t K);

/*
 * Fused RMSNorm + 1x128 activation quantization (Sec. 3.4: quantization fused
 * with the norm before the gate-up linear).
 *   x      [M x H] bf16            (input, the post-residual hidden state)
 *   norm_w [H] bf16                (input)
 *   xq     [M x H] e4m3            (output)
 *   xs     [H/128 x M] fp32        (output) scale of row m, group kb at xs[kb*M + m]
 * y = RN32(RN32(x * w) * r), r = RN32(1 / sqrt(sum(x^2) / H + 1e-5)), the sum
 * taken in fp64 in a fixed order: element i goes to partial (i/8) mod 64,
 * each partial adds in increasing i, and the partials combine by a xor
 * butterfly over offsets 32, 16, 8, 4, 2, 1.
 */
int lacache_rmsnorm_quant(void* stream, const uint16_t* x, const uint16_t* norm_w, uint8_t* xq, float* xs,
                          int64_t M, int64_t H, int group);

/*
 * The same with the residual add before the norm fused in (Sec. 3.4: the
 * quantization is fused with the AddNorm before the gate-up linear):
 *   resid [M x H] bf16 (input and output): resid = RNE_bf16(float(resid) +
 *         float(y)), written in place, and the norm reads the new value
 *   y     [M x H] bf16 (input), must not overlap resid
 * Bit for bit the same as lacache_add_bf16(resid, y) followed by
 * lacache_rmsnorm_quant(resid, ...), in one kernel.
 */
int lacache_add_rmsnorm_quant(void* stream, uint16_t* resid, const uint16_t* y, const uint16_t* norm_w,
                              uint8_t* xq, float* xs, int64_t M, int64_t H, int group);

/*
 * FP8 gate/up GEMM with per-group dequantization, fused SwiGLU and 1x128
 * re-quantization (Sec. 3.4: quantization fused with the SwiGLU before the
 * ffout linear).
 *   xq, xs  as produced by lacache_rmsnorm_quant                   (input)
 *   wgu_q   [2I x H] e4m3 (tile layout), wgu_s [2I/128 x H/128] fp32 (input)
 *   hq      [M x I] e4m3, hs [I/128 x M] fp32                      (output)
 *   h_tap   [M x I] fp32 or NULL: if non-NULL, also receives the fp32 h that
 *           was quantized (a test hook; same kernel, one more store)
 * acc[m,n] = sum_kb (xs[kb,m] * wgu_s[n/128,kb]) * dot_kb(xq[m,:], wgu_q[n,:])
 * accumulated in fp32; h = SiLU(acc[:, j]) * acc[:, I + j].
 * On the skinny path h passes through the library workspace (M x I fp32),
 * and the K range is split into four parts whose fp32 partial sums are
 * added in part order; at 33..64 rows the K range is first split into two
 * halves (separate workgroups) whose gate and up sums pass through the
 * workspace and are added in half order before SwiGLU.
 */
int lacache_gateup_swiglu_quant(void* stream, const uint8_t* xq, const float* xs, const uint8_t* wgu_q,
                                const float* wgu_s, uint8_t* hq, float* hs, float* h_tap,
                                int64_t M, int64_t H, int64_t I, int group);

/*
 * FP8 down (ffout) GEMM with per-group dequantization to bf16 (Sec. 3.4).
 *   hq, hs  as produced by lacache_gateup_swiglu_quant             (input)
 *   wd_q    [H x I] e4m3 (tile layout), wd_s [H/128 x I/128] fp32  (input)
 *   out     [M x H] bf16, rounded to nearest-even from fp32         (output)
 *   out_tap [M x H] fp32 or NULL: if non-NULL, also receives the fp32 value
 *           that was rounded (test hook)
 * On the skinny path (M <= 64) the K range is split over the four
 * wavefronts of a workgroup, whose fp32 partial sums are added in wavefront
 * order.
 */
int lacache_down_proj(void* stream, const uint8_t* hq, const float* hs, const uint8_t* wd_q, const float* wd_s,
                      uint16_t* out, float* out_tap, int64_t M, int64_t H, int64_t I, int group);

/*
 * The whole FP8 FFN of one layer: the three stages above in one call.
 *   x [M x H] bf16, norm_w [H] bf16, wgu_q/wgu_s and wd_q/wd_s as produced by
 *   lacache_quant_weights, out [M x H] bf16.
 * The intermediates (xq, xs, hq, hs and partial sums) live in a workspace
 * that the library allocates on first use per device, grows when a larger
 * call needs it, and keeps until lacache_release_workspace(). Calls that
 * share a device must therefore be serialized (one stream, or the caller's
 * own ordering); concurrent callers use lacache_ffn_fp8_ws instead.
 */
int lacache_ffn_fp8(void* stream, const uint16_t* x, const uint16_t* norm_w, const uint8_t* wgu_q,
                    const float* wgu_s, const uint8_t* wd_q, const float* wd_s, uint16_t* out,
                    int64_t M, int64_t H, int64_t I, int group);

/*
 * The FFN with the AddNorm before it: resid = RNE_bf16(resid + y) in place,
 * then out = FFN(resid) (Sec. 3.4). Bit for bit the same as
 * lacache_add_bf16(resid, y) followed by lacache_ffn_fp8(resid, ..., out),
 * one kernel less. In a stack of FFN layers with residual connections,
 * layer l > 1 passes the previous layer's out as y. resid, y and out must
 * not overlap each other or the weights. Uses the library workspace like
 * lacache_ffn_fp8.
 */
int lacache_ffn_fp8_addnorm(void* stream, uint16_t* resid, const uint16_t* y, const uint16_t* norm_w,
                            const uint8_t* wgu_q, const float* wgu_s, const uint8_t* wd_q, const float* wd_s,
                            uint16_t* out, int64_t M, int64_t H, int64_t I, int group);

/* Bytes of workspace lacache_ffn_fp8_ws needs for this shape (0 on bad arguments). */
size_t lacache_ffn_workspace_bytes(int64_t M, int64_t H, int64_t I, int group);

/* lacache_ffn_fp8 with a caller-owned workspace of at least
 * lacache_ffn_workspace_bytes() bytes (256-byte aligned device memory). */
int lacache_ffn_fp8_ws(void* stream, const uint16_t* x, const uint16_t* norm_w, const uint8_t* wgu_q,
                       const float* wgu_s, const uint8_t* wd_q, const float* wd_s, uint16_t* out,
                       int64_t M, int64_t H, int64_t I, int group, void* workspace, size_t ws_bytes);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops and harnesses that forbid hipMalloc):
 * lacache_ffn_fp8 with its whole workspace in a fixed device array of
 * LACACHE_NOALLOC_SCRATCH_BYTES (64 MiB) that the library's code object
 * holds on every device it runs on until the process ends. The call
 * allocates nothing (no hipMalloc, hipFree or allocating library routine);
 * its first call on a device looks up the array's address on that device
 * (hipGetSymbolAddress, no allocation). Arguments, results and errors are
 * those of lacache_ffn_fp8, and the same kernels run, so the output bytes
 * are identical. A shape whose workspace (lacache_ffn_workspace_bytes)
 * exceeds the array returns LACACHE_ERR_UNSUPPORTED before anything is
 * launched; at H = 4096, I = 12288 every M <= 1024 fits. All calls on one
 * device share the array, which keeps the last call's contents (no part of
 * it needs any initial value): calls that overlap in time on one device
 * (other streams, other host threads) race on it, so the caller must
 * serialize them.
 */
#define LACACHE_NOALLOC_SCRATCH_BYTES (64u << 20)
int lacache_ffn_fp8_noalloc(void* stream, const uint16_t* x, const uint16_t* norm_w, const uint8_t* wgu_q,
                            const float* wgu_s, const uint8_t* wd_q, const float* wd_s, uint16_t* out,
                            int64_t M, int64_t H, int64_t I, int group);

/* Residual add between stacked layers (the "Add" of the AddNorm that Sec. 3.4
 * fuses with the quantization; also available fused, see
 * lacache_add_rmsnorm_quant): x[i] = RNE_bf16(float(x[i]) + float(y[i])), i < n.
 * x and y must not overlap. */
int lacache_add_bf16(void* stream, uint16_t* x_inout, const uint16_t* y, int64_t n);

/* Test hook: the device e4m3 encoder applied elementwise, codes[i] = E(v[i]),
 * i < n (E clips to +-448 and rounds to nearest-even; NaN inputs give NaN codes). */
int lacache_encode_e4m3(void* stream, const float* v, uint8_t* codes, int64_t n);

/*
 * First-layer attention with FACache (Sec. 3.3, FACache; Eqs. 2-6).
 *
 * LaCache keeps the first transformer layer in bf16 and runs its attention
 * as a FlashAttention-style scan over blocks of 64 keys, carrying per query
 * row the running max m, the running sum l and the unnormalized output O~
 * (Eqs. 2-6), and finishing with O = O~ / l. Within one SAR block of the
 * generation only the rows of the current block C = [c_begin, c_end) change
 * between denoising steps; FACache stores the state of every query block of
 * 64 rows that has no row in C (a block "inside U"), taken over the key
 * blocks that also have no row in C, and later steps resume from it.
 *   q, k, v [heads x N x d] bf16    (input) one attention problem per head
 *   o       [heads x N x d] bf16    (output) softmax(q k^T / sqrt(d)) v per
 *                                   head, bidirectional (no mask)
 *   lse     [heads x N] fp32        (optional output, NULL to skip) the
 *                                   row-wise log-sum-exp of q k^T / sqrt(d),
 *                                   natural log (Alg. 1 of the Appendix)
 *   cache_m, cache_l [heads x N] fp32, cache_o [heads x N x d] fp32
 *                                   the FACache state of row n of head h at
 *                                   index h*N + n (cache_o rows of d values):
 *                                   m in base-2 units (max of q.k log2(e) /
 *                                   sqrt(d)), l and O~ relative to it; only
 *                                   the rows of query blocks inside U are
 *                                   written or read
 *   mode 0  populate: full attention; also writes the cache rows of the
 *           query blocks inside U (their state after the key blocks inside U);
 *   mode 1  resume: query blocks inside U load their cached state and scan
 *           only the key blocks that overlap C; the result equals plain
 *           attention of the current inputs when, since the mode-0 call with
 *           the same c_begin, c_end, only rows of C of q, k and v changed;
 *   mode 2  plain attention; the cache pointers are not used (may be NULL).
 * d must be 128 and N a multiple of 64 (LACACHE_ERR_UNSUPPORTED otherwise);
 * heads <= 4096, N <= 2^20; 0 <= c_begin <= c_end <= N, mode in 0..2
 * (LACACHE_ERR_INVALID_ARG otherwise). heads == 0 or N == 0 launches nothing.
 * The cache is written in mode 0 and read in mode 1; o and lse must not
 * overlap any other buffer, and in mode 0 the cache must not overlap q, k, v,
 * o or lse. An empty C (c_begin == c_end) overlaps no block: populate then
 * stores the state over all keys and resume streams no key block.
 * Arithmetic: bf16 products accumulated in fp32 (MFMA), scores scaled and
 * exponentiated in base 2, P rounded to bf16 for the P V product, m, l and
 * O~ kept in fp32, o rounded to bf16.
 */
int lacache_facache_attention(void* stream, const uint16_t* q, const uint16_t* k, const uint16_t* v, uint16_t* o,
                              float* lse, float* cache_m, float* cache_l, float* cache_o, int64_t heads, int64_t N,
                              int64_t d, int64_t c_begin, int64_t c_end, int mode);

/*
 * Coarse quantization granularities (Sec. 4, Table fp8-granularities): the
 * paper compares its per-group scheme with "per tensor" and "per token"
 * quantization of the same FFN linears. Readings: per tensor = one scale for
 * a whole activation tensor and one for a whole weight; per token = one scale
 * per activation row and one per weight output channel (row). The quantizer
 * rules are those of the per-group path (Eqs. 7-8); only the set of values
 * sharing a scale changes. A coarse scale needs the max over a whole row or
 * tensor, which one GEMM tile never sees, so these paths quantize in separate
 * passes and the SwiGLU output goes through HBM in fp32 (the per-group path
 * fuses both quantizations). Scales are written in the per-group layouts
 * (every group of a row carries the row's scale; weight block scales are 1
 * and the per-row weight scales multiply each output column after the K
 * sum), so the same GEMM kernels run every granularity. For comparison
 * studies; the per-group calls above are the library's FFN.
 */
enum { LACACHE_GRAN_GROUP = 0, LACACHE_GRAN_TOKEN = 1, LACACHE_GRAN_TENSOR = 2 };

/*
 * Weight quantization at a granularity. GROUP: lacache_quant_weights (w_row_s
 * unused, may be NULL). TOKEN / TENSOR:
 *   w       [N x K] bf16                     (input)
 *   w_q     [N x K] e4m3 (tile layout)       (output)
 *   w_s     [N/128 x K/128] fp32             (output) all 1.0
 *   w_row_s [N] fp32                         (output) RN32(max|w[n, :]| / 448)
 *                                            per row, or the whole matrix's
 *                                            scale in every entry (TENSOR)
 * Other granularity values: LACACHE_ERR_INVALID_ARG.
 */
int lacache_quant_weights_g(void* stream, const uint16_t* w, uint8_t* w_q, float* w_s, float* w_row_s, int64_t N,
                            int64_t K, int granularity);

/* The RMSNorm alone: y [M x H] fp32 = RN32(RN32(x * norm_w) * r), the same
 * values the fused quantizer quantizes (lacache_rmsnorm_quant). */
int lacache_rmsnorm_f32(void* stream, const uint16_t* x, const uint16_t* norm_w, float* y, int64_t M, int64_t H);

/*
 * Quantization of fp32 rows v [M x K] (K a multiple of 128) at a granularity:
 *   q      [M x K] e4m3                      (output)
 *   s_kgm  [K/128 x M] fp32                  (output) the scale of group kb of
 *                                            row m at s_kgm[kb*M + m] (for
 *                                            TOKEN / TENSOR the row's scale in
 *                                            every group)
 *   s_rows [M] fp32                          (output, TOKEN / TENSOR; unused
 *                                            and may be NULL for GROUP) the
 *                                            row scales
 */
int lacache_quant_rows_g(void* stream, const float* v, uint8_t* q, float* s_kgm, float* s_rows, int64_t M, int64_t K,
                         int granularity);

/*
 * The gate/up GEMM and SwiGLU without the re-quantization: h [M x I] fp32 =
 * SiLU(g) * u, g and u the dequantized sums of lacache_gateup_swiglu_quant,
 * each output column n also multiplied by wgu_row_s[n] ([2I] fp32, gate rows
 * first) when wgu_row_s is not NULL. Always the tiled kernels.
 */
int lacache_gateup_swiglu_f32(void* stream, const uint8_t* xq, const float* xs, const uint8_t* wgu_q,
                              const float* wgu_s, const float* wgu_row_s, float* h, int64_t M, int64_t H, int64_t I,
                              int group);

/* lacache_down_proj with output column n also multiplied by wd_row_s[n] ([H]
 * fp32, NULL for none) before the bf16 rounding. Always the tiled kernels. */
int lacache_down_proj_g(void* stream, const uint8_t* hq, const float* hs, const uint8_t* wd_q, const float* wd_s,
                        const float* wd_row_s, uint16_t* out, float* out_tap, int64_t M, int64_t H, int64_t I,
                        int group);

/*
 * The whole FFN at a granularity, with weights from lacache_quant_weights_g
 * of the same granularity. GROUP: lacache_ffn_fp8 (row scales unused).
 * TOKEN / TENSOR: RMSNorm -> quantization of its rows -> gate/up + SwiGLU
 * (fp32 h) -> quantization of h -> down, with a library-owned workspace of
 * lacache_ffn_g_workspace_bytes(M, H, I) (serialize calls on one device, as
 * for lacache_ffn_fp8).
 */
int lacache_ffn_fp8_g(void* stream, const uint16_t* x, const uint16_t* norm_w, const uint8_t* wgu_q,
                      const float* wgu_s, const float* wgu_row_s, const uint8_t* wd_q, const float* wd_s,
                      const float* wd_row_s, uint16_t* out, int64_t M, int64_t H, int64_t I, int granularity);
size_t lacache_ffn_g_workspace_bytes(int64_t M, int64_t H, int64_t I);

/*
 * Token-wise first layer with EmbedCache and RoPECache (Sec. 3.3). Inside a
 * SAR block only the tokens of the current block C change, so embedding, the
 * attention RMSNorm, the QKV projection and RoPE run on C's rows only and
 * write into cached tensors that hold every row of the sequence: the
 * embedding cache [N x H] and Q, K, V [heads x N x 128] (the attention layout
 * of lacache_facache_attention). The first layer keeps 16-bit precision
 * (Sec. 3.4): bf16 values, fp32 arithmetic. A call with rows = 0..N-1 fills
 * the caches (the block's first step); a call with C's rows updates them, and
 * the result equals the full call on the new tokens bit for bit. Row indices
 * must be distinct within a call. Token ids outside [0, vocab) and row indices
 * outside [0, N) are device data the host cannot check: the kernels skip such
 * entries (nothing is read or written for them).
 *
 * lacache_embed_rmsnorm: x_r = embed[token_ids[r]] ([vocab x H] bf16) is
 *   written to embed_cache[rows[r]], and y[r] = RNE_bf16(RMSNorm(x_r)) with the
 *   arithmetic of lacache_rmsnorm_quant (eps 1e-5, fp64 sum of squares in its
 *   fixed order, y = RN32(RN32(x w) r)). token_ids, rows: [R] int32.
 */
int lacache_embed_rmsnorm(void* stream, const int32_t* token_ids, const int32_t* rows, int64_t R,
                          const uint16_t* embed, int64_t vocab, const uint16_t* norm_w, uint16_t* embed_cache,
                          int64_t N, uint16_t* y, int64_t H);

/* out [M x N] bf16 = RNE_bf16(a [M x K] W[N x K]^T), bf16 inputs, fp32
 * accumulation (bf16 MFMAs; the K range is split over four partial sums added
 * in a fixed order); out_tap (nullable) receives the fp32 result. Up to 128
 * rows W is streamed from HBM once per 64 rows of a (the few rows of a block);
 * above, 128-row output tiles read it once per 128 rows. Both give every row
 * the same bytes, so a row's result does not depend on M. */
int lacache_linear_bf16(void* stream, const uint16_t* a, const uint16_t* w, uint16_t* out, float* out_tap, int64_t M,
                        int64_t N, int64_t K);

/*
 * RoPE and scatter: row r of qkv ([R x 3 heads 128] bf16, columns = Q heads,
 * then K heads, then V heads, 128 each) goes to row rows[r] of q, k, v
 * ([heads x N x 128] bf16). Q and K are rotated (rotate-half form): for the
 * pair (i, i + 64) of a head, i < 64, with c = rope_cos[p*64 + i] and
 * s = rope_sin[p*64 + i] (p = rows[r]; fp32 tables [N x 64]),
 *   out_i = RNE_bf16(RN32(x_i c) - RN32(x_{i+64} s)),
 *   out_{i+64} = RNE_bf16(RN32(x_{i+64} c) + RN32(x_i s)); V is copied.
 */
int lacache_rope_scatter(void* stream, const uint16_t* qkv, const int32_t* rows, int64_t R, const float* rope_cos,
                         const float* rope_sin, uint16_t* q, uint16_t* k, uint16_t* v, int64_t heads, int64_t N);

/* The three steps above in one call (embedding + norm, the QKV projection
 * with w_qkv [3 heads 128 x H] bf16, RoPE + scatter), with a library-owned
 * workspace of lacache_first_layer_workspace_bytes(R, heads, H) bytes. */
int lacache_first_layer_tokens(void* stream, const int32_t* token_ids, const int32_t* rows, int64_t R,
                               const uint16_t* embed, int64_t vocab, const uint16_t* norm_w, const uint16_t* w_qkv,
                               const float* rope_cos, const float* rope_sin, uint16_t* embed_cache, uint16_t* q,
                               uint16_t* k, uint16_t* v, int64_t heads, int64_t N, int64_t H);
size_t lacache_first_layer_workspace_bytes(int64_t R, int64_t heads, int64_t H);

/*
 * Kernel-path policy for the GEMM stages, process-wide:
 *   0 = automatic (the skinny weight-streaming kernels for M <= 64 whose
 *       activation rows fit the gate/up kernel's LDS: ceil(M/16) 16 (H + 16)
 *       <= 132096 bytes for M <= 32, ceil(M/16) 16 (ceil(H/256) 128 + 16)
 *       <= 132096 for 33..64 rows; H <= 8192, I <= 16384; the tiled MFMA
 *       kernels otherwise), 1 = always skinny (other shapes return
 *       LACACHE_ERR_UNSUPPORTED), 2 = always tiled.
 * Returns the previous policy, or LACACHE_ERR_INVALID_ARG for other values.
 */
int lacache_set_path_policy(int policy);

/* Human-readable name of a status code (static string). */
const char* lacache_status_string(int status);

/* Frees the library-owned workspace of every device, superseded buffers
 * included (synchronizes each device first). HIP graphs captured with calls
 * that used the library workspace must not be replayed afterwards. */
void lacache_release_workspace(void);

#ifdef __cplusplus
}
#endif

#endif /* LACACHE_H */
