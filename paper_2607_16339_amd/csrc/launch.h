// Internal kernel launchers (C++ linkage). Arguments are validated by the
// C ABI layer before any of these is called; each returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace lacache {

hipError_t launch_quant_weights(hipStream_t st, const uint16_t* w, uint8_t* wq, float* ws, int64_t N, int64_t K);
// Row-major e4m3 codes [N x K] (N % 16 == 0, K % 128 == 0) -> tile layout.
hipError_t launch_pack_weights(hipStream_t st, const uint8_t* w, uint8_t* wt, int64_t N, int64_t K);
// With y non-null: x = RNE_bf16(x + y) in place first (the fused AddNorm).
hipError_t launch_rmsnorm_quant(hipStream_t st, uint16_t* x, const uint16_t* nw, uint8_t* xq, float* xs, int64_t M,
                                int64_t H, const uint16_t* y = nullptr);
// The RMSNorm alone, y = RN32(RN32(x * w) * r) in fp32 [M x H] (same
// arithmetic as the fused quantizer).
hipError_t launch_rmsnorm_f32(hipStream_t st, const uint16_t* x, const uint16_t* nw, float* y, int64_t M, int64_t H);
hipError_t launch_add_bf16(hipStream_t st, uint16_t* x, const uint16_t* y, int64_t n);

// Coarse granularities: per-row (or, with per_tensor, one) scales of fp32
// rows [M x K] into s_rows [M], the codes, and (kgm non-null) the scales in
// the K-group-major [K/128 x M] layout of the GEMMs.
hipError_t launch_quant_rows_f32(hipStream_t st, const float* v, uint8_t* codes, float* kgm, float* s_rows, int64_t M,
                                 int64_t K, bool per_tensor);
// The same for a bf16 weight [N x K]: row scales w_rows [N], block scales
// w_blocks [N/128 x K/128] set to 1 (the row scales act in the GEMM epilogue).
hipError_t launch_quant_weights_rows(hipStream_t st, const uint16_t* w, uint8_t* wq, float* w_blocks, float* w_rows,
                                     int64_t N, int64_t K, bool per_tensor);
// The 1x128 group quantizer of fp32 rows [M x K] (codes, scales [K/128 x M]).
hipError_t launch_quant_groups_f32(hipStream_t st, const float* v, uint8_t* codes, float* scales, int64_t M, int64_t K);
hipError_t launch_encode_e4m3(hipStream_t st, const float* v, uint8_t* codes, int64_t n);

// Compute units of the current device, cached per device (256 when the
// runtime cannot tell).
int device_cu_count();

// Tile (row r, column c) of workgroup `bid` in an R x C grid of output tiles.
// Workgroups are handed out round-robin over the 8 XCDs, each with its own
// L2, so XCD x runs workgroups x, x + 8, ... Each XCD gets a contiguous range
// of tiles in grouped order (kTileGroupRows row tiles by all columns, row
// tile fastest): the workgroups an XCD runs at the same time cover a few
// weight tiles and a few activation tiles, which its L2 then serves to all of
// them. A bijection of [0, R*C) for any R, C.
constexpr int64_t kXcds = 8;
// 4 row tiles: measured 2.5 % faster than 8 at M = 512 and no slower at M = 8192
constexpr int64_t kTileGroupRows = 4;
__host__ __device__ inline void xcd_grouped_tile(int64_t bid, int64_t R, int64_t C, int64_t& r, int64_t& c) {
  const int64_t T = R * C;
  const int64_t x = bid % kXcds, slot = bid / kXcds;
  const int64_t per = T / kXcds, rem = T % kXcds;
  const int64_t t = (x < rem ? x * (per + 1) : rem * (per + 1) + (x - rem) * per) + slot;
  const int64_t g = t / (kTileGroupRows * C);
  const int64_t first = g * kTileGroupRows;
  const int64_t rows = R - first < kTileGroupRows ? R - first : kTileGroupRows;
  const int64_t w = t - g * kTileGroupRows * C;
  r = first + w % rows;
  c = w / rows;
}

// Tiled MFMA GEMMs (any M). col_s (nullable): a scale per weight row that
// multiplies that output column after the K sum (per-channel weights); with
// hq == nullptr the gate/up writes only the fp32 h to h_tap (no quantization).
hipError_t launch_gateup_tiled(hipStream_t st, const uint8_t* xq, const float* xs, const uint8_t* wq,
                               const float* ws, uint8_t* hq, float* hs, float* h_tap, int64_t M, int64_t H,
                               int64_t I, const float* col_s = nullptr);
// The down GEMM splits K over several workgroups when there are too few
// output tiles to fill the chip; it then needs an fp32 scratch buffer of
// tiled_down_ws_bytes() (0 when it does not split).
size_t tiled_down_ws_bytes(int64_t M, int64_t H, int64_t I);
hipError_t launch_down_tiled(hipStream_t st, const uint8_t* hq, const float* hs, const uint8_t* wq, const float* ws,
                             uint16_t* out, float* out_tap, int64_t M, int64_t H, int64_t I, void* ws_buf,
                             const float* col_s = nullptr);

// Skinny weight-streaming GEMMs (M <= kSkinnyMaxM; skinny_supported() also
// checks that the activation rows fit the gate/up kernel's LDS).
// The gate/up stage needs an fp32 scratch buffer of skinny_gateup_ws_bytes()
// (no initial contents) for h; the down stage needs none.
constexpr int64_t kSkinnyMaxM = 64;
bool skinny_supported(int64_t M, int64_t H, int64_t I);
size_t skinny_gateup_ws_bytes(int64_t M, int64_t I);
hipError_t launch_gateup_skinny(hipStream_t st, const uint8_t* xq, const float* xs, const uint8_t* wq,
                                const float* ws, uint8_t* hq, float* hs, float* h_tap, int64_t M, int64_t H,
                                int64_t I, void* ws_buf);
hipError_t launch_down_skinny(hipStream_t st, const uint8_t* hq, const float* hs, const uint8_t* wq, const float* ws,
                              uint16_t* out, float* out_tap, int64_t M, int64_t H, int64_t I);

// Token-wise first layer (EmbedCache / RoPECache). Ids outside [0, vocab)
// and rows outside [0, N) are skipped on the device.
hipError_t launch_embed_rmsnorm(hipStream_t st, const int32_t* ids, const int32_t* rows, int64_t R,
                                const uint16_t* embed, int64_t vocab, const uint16_t* nw, uint16_t* cache, int64_t N,
                                uint16_t* y, int64_t H);
hipError_t launch_linear_bf16(hipStream_t st, const uint16_t* a, const uint16_t* w, uint16_t* out, float* out_tap,
                              int64_t M, int64_t N, int64_t K);
hipError_t launch_rope_scatter(hipStream_t st, const uint16_t* qkv, const int32_t* rows, int64_t R, const float* cs,
                               const float* sn, uint16_t* q, uint16_t* k, uint16_t* v, int64_t heads, int64_t N);

// First-layer attention with FACache: heads x N x 128 bf16, N % 64 == 0;
// mode 0 populate, 1 resume, 2 plain (cache pointers unused).
hipError_t launch_facache_attention(hipStream_t st, const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                    uint16_t* o, float* cm, float* cl, float* co, float* lse, int64_t heads, int64_t N,
                                    int64_t c0, int64_t c1, int mode);

}  // namespace lacache
