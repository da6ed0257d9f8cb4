// Tiled FP8 MFMA GEMMs with per-group dequantization (Sec. 3.4):
//   gate/up: x[M x H] . Wgu[2I x H]^T, fused SwiGLU and 1x128 re-quantization
//   down:    h[M x I] . Wd[H x I]^T -> bf16
//
// A workgroup (4 wavefronts) computes a 128-row x 256-weight-row tile and
// walks K one 128-wide group at a time: the group's fp8 tiles are staged in
// LDS, every 16x16 output sub-tile gets one 16x16x128 FP8 MFMA (exactly one
// K-group), and its fp32 result is added to the accumulator times
// RN32(x_scale[row] * w_scale[block]).
//
// For gate/up the tile's 256 weight rows are the 128 gate rows and the 128
// matching up rows of one h-group, so each lane holds gate and up values of
// the same (row, column) and the whole 128-wide h-group of a row lives in
// one workgroup: SwiGLU, the row amax and the e4m3 encoding happen before
// anything is written; h never reaches memory in 16 or 32 bits.
#include "device.h"
#include "launch.h"

namespace lacache {
namespace {

constexpr int BM = 128;   // activation rows per workgroup
constexpr int BNR = 256;  // weight rows per workgroup
constexpr int kThreads = 256;

// LDS tiles are [rows][128 bytes]; the eight 16-byte chunks of a row are
// permuted by an xor with a row hash so that 16 consecutive rows read at the
// same logical chunk fall into distinct banks.
__device__ __forceinline__ int lds_off(int row, int chunk) {
  return row * 128 + ((chunk ^ ((row ^ (row >> 3)) & 7)) << 4);
}

// MFMA operand for one 16-row slab: lane (q = l/16, r = l%16) takes row
// base + r, logical chunks q and 4 + q (the same K placement for A and B).
__device__ __forceinline__ v8i load_frag(const uint8_t* tile, int row, int q) {
  const uint4 lo = *reinterpret_cast<const uint4*>(tile + lds_off(row, q));
  const uint4 hi = *reinterpret_cast<const uint4*>(tile + lds_off(row, 4 + q));
  v8i f;
  f[0] = static_cast<int>(lo.x); f[1] = static_cast<int>(lo.y); f[2] = static_cast<int>(lo.z); f[3] = static_cast<int>(lo.w);
  f[4] = static_cast<int>(hi.x); f[5] = static_cast<int>(hi.y); f[6] = static_cast<int>(hi.z); f[7] = static_cast<int>(hi.w);
  return f;
}

template <bool kGateUp>
__global__ __launch_bounds__(kThreads) void gemm_tiled_kernel(
    const uint8_t* __restrict__ aq, const float* __restrict__ as,  // [M x K] codes, [K/128 x M] scales
    const uint8_t* __restrict__ bq, const float* __restrict__ bs,  // [N x K] codes, [N/128 x K/128] scales
    uint8_t* __restrict__ hq, float* __restrict__ hs, float* __restrict__ h_tap,
    uint16_t* __restrict__ out, float* __restrict__ out_tap, int64_t M, int64_t K, int64_t N, int64_t I) {
  __shared__ __align__(16) uint8_t sA[BM * 128];
  __shared__ __align__(16) uint8_t sB[BNR * 128];
  __shared__ __align__(16) float sXs[BM];
  __shared__ float sRed[2][BM];

  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int q = lane >> 4, lr = lane & 15;
  const int64_t m0 = static_cast<int64_t>(blockIdx.x) * BM;
  const int64_t by = blockIdx.y;  // gate/up: h-group; down: 256-column tile
  const int64_t KB = K / 128;

  // ---- global -> register mapping: thread t loads tile rows (t/8) + 32u, chunk t%8
  const int lrow = t >> 3, lch = t & 7;
  const int64_t stride32 = 32 * K;
  const uint8_t* a_base = aq + (m0 + lrow) * K + lch * 16;
  const uint8_t* b_base;
  const uint8_t* b_base_hi;  // gate/up: up rows; down: unused
  int64_t n0 = 0;
  if (kGateUp) {
    b_base = bq + (by * 128 + lrow) * K + lch * 16;
    b_base_hi = b_base + I * K;
  } else {
    n0 = by * BNR;
    b_base = bq + (n0 + lrow) * K + lch * 16;
    b_base_hi = b_base;
  }
  uint4 ra[4], rb[8];
  float rxs = 0.0f;
  const uint4 z4 = make_uint4(0u, 0u, 0u, 0u);

  auto gload = [&](int64_t kb) {
    const int64_t ko = kb * 128;
#pragma unroll
    for (int u = 0; u < 4; ++u)
      ra[u] = (m0 + lrow + 32 * u < M) ? *reinterpret_cast<const uint4*>(a_base + u * stride32 + ko) : z4;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (kGateUp) {
        const uint8_t* p = (u < 4 ? b_base + u * stride32 : b_base_hi + (u - 4) * stride32) + ko;
        rb[u] = *reinterpret_cast<const uint4*>(p);
      } else {
        rb[u] = (n0 + lrow + 32 * u < N) ? *reinterpret_cast<const uint4*>(b_base + u * stride32 + ko) : z4;
      }
    }
    if (t < BM) rxs = (m0 + t < M) ? as[kb * M + m0 + t] : 0.0f;
  };
  auto sstore = [&]() {
#pragma unroll
    for (int u = 0; u < 4; ++u) *reinterpret_cast<uint4*>(sA + lds_off(lrow + 32 * u, lch)) = ra[u];
#pragma unroll
    for (int u = 0; u < 8; ++u) *reinterpret_cast<uint4*>(sB + lds_off(lrow + 32 * u, lch)) = rb[u];
    if (t < BM) sXs[t] = rxs;
  };

  // weight-block scale rows used by this wavefront
  int64_t nb0, nb1;
  bool nb_ok = true;
  if (kGateUp) {
    nb0 = by;             // gate block
    nb1 = I / 128 + by;   // up block
  } else {
    nb0 = (n0 + 128 * wn) / 128;
    nb1 = nb0;
    nb_ok = n0 + 128 * wn < N;
  }
  auto brow = [&](int j) -> int {
    if (kGateUp) return j < 4 ? 64 * wn + 16 * j : 128 + 64 * wn + 16 * (j - 4);
    return 128 * wn + 16 * j;
  };

  float acc[4][8][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[i][j][r] = 0.0f;

  gload(0);
  sstore();
  __syncthreads();
  for (int64_t kb = 0; kb < KB; ++kb) {
    if (kb + 1 < KB) gload(kb + 1);
    const float w0 = nb_ok ? bs[nb0 * KB + kb] : 0.0f;
    const float w1 = nb_ok ? bs[nb1 * KB + kb] : 0.0f;
    v8i af[4];
    float sc0[4][4], sc1[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      af[i] = load_frag(sA, 64 * wm + 16 * i + lr, q);
      const float4 xv = *reinterpret_cast<const float4*>(sXs + 64 * wm + 16 * i + 4 * q);
      const float xa[4] = {xv.x, xv.y, xv.z, xv.w};
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        sc0[i][r] = xa[r] * w0;  // RN32(x_scale * w_scale)
        sc1[i][r] = xa[r] * w1;
      }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const v8i bf = load_frag(sB, brow(j) + lr, q);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const v4f zero = {0.0f, 0.0f, 0.0f, 0.0f};
        const v4f p = mfma_fp8_16x16x128(af[i], bf, zero);
#pragma unroll
        for (int r = 0; r < 4; ++r)
          acc[i][j][r] = __builtin_fmaf(p[r], (kGateUp && j >= 4) ? sc1[i][r] : sc0[i][r], acc[i][j][r]);
      }
    }
    __syncthreads();
    if (kb + 1 < KB) {
      sstore();
      __syncthreads();
    }
  }

  if (kGateUp) {
    // ---- SwiGLU: h = SiLU(g) * u, lanes hold matching gate (j) and up (j + 4) values
    float h[4][4][4];
    float am[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float a = 0.0f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float g = acc[i][j][r], u = acc[i][j + 4][r];
          const float v = g / (1.0f + expf(-g)) * u;
          h[i][j][r] = v;
          a = __builtin_fmaxf(a, __builtin_fabsf(v));
        }
        am[i][r] = max_xor<16>(a);  // over the 16 columns of the same rows
      }
    if (lr == 0) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) sRed[wn][64 * wm + 16 * i + 4 * q + r] = am[i][r];
    }
    __syncthreads();
    // ---- 1x128 quantization of each row's h-group; codes go through LDS for coalesced stores
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 64 * wm + 16 * i + 4 * q + r;
        const float s = __builtin_fmaxf(sRed[0][row], sRed[1][row]) / kE4M3Max;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int col = 64 * wn + 16 * j + lr;
          sA[row * 128 + col] = s == 0.0f ? 0 : static_cast<uint8_t>(enc1_e4m3(qdiv(h[i][j][r], s)));
          if (h_tap != nullptr && m0 + row < M) h_tap[(m0 + row) * I + by * 128 + col] = h[i][j][r];
        }
      }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int row = lrow + 32 * u;
      if (m0 + row < M)
        *reinterpret_cast<uint4*>(hq + (m0 + row) * I + by * 128 + lch * 16) =
            *reinterpret_cast<const uint4*>(sA + row * 128 + lch * 16);
    }
    if (t < BM && m0 + t < M) hs[by * M + m0 + t] = __builtin_fmaxf(sRed[0][t], sRed[1][t]) / kE4M3Max;
  } else {
    // ---- bf16 output, nearest-even from the fp32 accumulator
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = m0 + 64 * wm + 16 * i + 4 * q + r;
        if (row >= M) continue;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int64_t col = n0 + 128 * wn + 16 * j + lr;
          if (col < N) {
            out[row * N + col] = static_cast<uint16_t>(f32_to_bf16(acc[i][j][r]));
            if (out_tap != nullptr) out_tap[row * N + col] = acc[i][j][r];
          }
        }
      }
  }
}

}  // namespace

hipError_t launch_gateup_tiled(hipStream_t st, const uint8_t* xq, const float* xs, const uint8_t* wq,
                               const float* ws, uint8_t* hq, float* hs, float* h_tap, int64_t M, int64_t H,
                               int64_t I) {
  dim3 grid(static_cast<unsigned>((M + BM - 1) / BM), static_cast<unsigned>(I / 128));
  hipLaunchKernelGGL(gemm_tiled_kernel<true>, grid, dim3(kThreads), 0, st, xq, xs, wq, ws, hq, hs, h_tap,
                     static_cast<uint16_t*>(nullptr), static_cast<float*>(nullptr), M, H, 2 * I, I);
  return hipGetLastError();
}

hipError_t launch_down_tiled(hipStream_t st, const uint8_t* hq, const float* hs, const uint8_t* wq, const float* ws,
                             uint16_t* out, float* out_tap, int64_t M, int64_t H, int64_t I) {
  dim3 grid(static_cast<unsigned>((M + BM - 1) / BM), static_cast<unsigned>((H + BNR - 1) / BNR));
  hipLaunchKernelGGL(gemm_tiled_kernel<false>, grid, dim3(kThreads), 0, st, hq, hs, wq, ws,
                     static_cast<uint8_t*>(nullptr), static_cast<float*>(nullptr), static_cast<float*>(nullptr),
                     out, out_tap, M, I, H, I);
  return hipGetLastError();
}

}  // namespace lacache
