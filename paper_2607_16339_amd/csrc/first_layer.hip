// Token-wise first-layer operators with EmbedCache and RoPECache (Sec. 3.3):
// inside a SAR block only the rows of the current block C change, so the
// embedding, the attention RMSNorm, the QKV projection and RoPE run on those
// rows only and write their results into the cached tensors (the embedding
// cache [N x H] and Q, K, V [heads x N x 128] in the attention layout). The
// first layer keeps 16-bit precision (Sec. 3.4): bf16 storage, fp32
// arithmetic.
//
//   embed_rmsnorm_kernel  one wavefront per row: gather the token's embedding
//                         row, write it to the embedding cache, RMSNorm (the
//                         fused FFN quantizer's arithmetic: fp64 sum of squares
//                         in the same fixed order) rounded to bf16;
//   linear_bf16_kernel    out = a W^T for a few rows: 16 or 48 weight rows per
//                         workgroup streamed from HBM once per 64 activation
//                         rows, K split over the 4 wavefronts (private
//                         direct-to-LDS rings), bf16 MFMAs into fp32, the four
//                         partials added in wavefront order, bf16 out;
//   linear_bf16_tiled_kernel  the same result for many rows, from 128 x 128
//                         or 128 x 192 output tiles (W read once per 128 rows);
//   rope_scatter_kernel   rotate-half RoPE of the Q and K heads from fp32 cos /
//                         sin tables, V unrotated, scattered to each row's
//                         position in Q, K, V.
// Token ids outside [0, vocab) and row indices outside [0, N) are skipped on
// the device (no access is made for them).
#include "device.h"
#include "launch.h"

namespace lacache {
namespace {

typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

template <int T>
__global__ __launch_bounds__(256) void embed_rmsnorm_kernel(const int32_t* __restrict__ ids,
                                                            const int32_t* __restrict__ rows, int64_t R,
                                                            const uint16_t* __restrict__ embed, int64_t vocab,
                                                            const uint16_t* __restrict__ nw,
                                                            uint16_t* __restrict__ cache, int64_t N,
                                                            uint16_t* __restrict__ y, int H) {
  const int lane = threadIdx.x & 63;
  const int64_t r = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (r >= R) return;  // uniform per wavefront
  const int64_t id = ids[r], pos = rows[r];
  if (id < 0 || id >= vocab || pos < 0 || pos >= N) return;
  const int nchunk = H >> 3;
  const uint4* xr = reinterpret_cast<const uint4*>(embed + id * H);
  const uint4* wr = reinterpret_cast<const uint4*>(nw);
  uint4 xv[T], wv[T];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int c = t * 64 + lane;
    const int cc = c < nchunk ? c : nchunk - 1;
    xv[t] = xr[cc];
    wv[t] = wr[cc];
  }
  uint4* cw = reinterpret_cast<uint4*>(cache + pos * H);  // EmbedCache row
#pragma unroll
  for (int t = 0; t < T; ++t) {
    if (t * 64 + lane < nchunk)
      cw[t * 64 + lane] = xv[t];
    else
      xv[t] = make_uint4(0u, 0u, 0u, 0u);
  }
  // fp64 sum of squares: per-lane partials in increasing element index, then
  // a xor butterfly over offsets 32..1 (every lane ends with the same bits)
  double p = 0.0;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const uint32_t q[4] = {xv[t].x, xv[t].y, xv[t].z, xv[t].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const double a = bf16lo(q[e]), b = bf16hi(q[e]);
      p = p + a * a;
      p = p + b * b;
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) p = p + __shfl_xor(p, o, 64);
  const float rs = static_cast<float>(1.0 / __builtin_sqrt(p / static_cast<double>(H) + 1e-5));
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int c = t * 64 + lane;
    if (c >= nchunk) continue;
    const uint32_t q[4] = {xv[t].x, xv[t].y, xv[t].z, xv[t].w};
    const uint32_t g[4] = {wv[t].x, wv[t].y, wv[t].z, wv[t].w};
    uint32_t o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      o[e] = pack_bf16x2((bf16lo(q[e]) * bf16lo(g[e])) * rs, (bf16hi(q[e]) * bf16hi(g[e])) * rs);
    reinterpret_cast<uint4*>(y + r * H)[c] = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

// out [M x N] = a [M x K] W[N x K]^T, bf16 in and out, fp32 accumulation.
// Workgroup (blockIdx.x, blockIdx.y): weight rows 16 NJ x .. (NJ slabs of
// 16), activation rows 64 y .. + 63 (MT slabs of 16 rows). Its 4 wavefronts
// take a quarter of the K range each; a K-step is 64 elements (128 bytes of a
// row), staged global -> LDS as [rows][128 B] with the 16-byte chunk c of
// row r at c ^ (r mod 8); each 16x16 tile gets two 16x16x32 bf16 MFMAs per
// K-step (the lanes' chunks q and 4 + q). Several weight slabs per workgroup
// share each staged activation row, so the activations (re-read from L2 by
// every workgroup) cost less of the CU's copy bandwidth than the weights.
constexpr int kLinSplit = 4;

template <int MT, int NJ>
struct LinCfg {
  static constexpr int RA = MT * 16;
  static constexpr int kA = RA * 128;
  static constexpr int kSlot = kA + NJ * 16 * 128;
  static constexpr int AI = RA / 8;  // 1 KB copies of activations per slot
  static constexpr int PER = AI + 2 * NJ;
  static constexpr int D0 = 160000 / (kLinSplit * kSlot);  // ring depth that fits the LDS
  static constexpr int D = D0 > 8 ? 8 : D0;
  static_assert(D >= 2, "ring depth");
};

__device__ __forceinline__ void lin_frag(const uint8_t* rows, int lr, int q, bf8& lo, bf8& hi) {
  const uint8_t* row = rows + lr * 128;
  lo = *reinterpret_cast<const bf8*>(row + ((q ^ (lr & 7)) << 4));
  hi = *reinterpret_cast<const bf8*>(row + (((4 + q) ^ (lr & 7)) << 4));
}

template <int MT, int NJ>
__global__ __launch_bounds__(kLinSplit * 64) void linear_bf16_kernel(const uint16_t* __restrict__ a,
                                                                     const uint16_t* __restrict__ w,
                                                                     uint16_t* __restrict__ out,
                                                                     float* __restrict__ out_tap, int64_t M,
                                                                     int64_t N, int64_t K) {
  using C = LinCfg<MT, NJ>;
  constexpr int D = C::D, RA = C::RA, NC = 16 * NJ;
  __shared__ __align__(16) uint8_t ring[kLinSplit][D * C::kSlot];
  const int t = threadIdx.x, lane = t & 63;
  const int wave = wave_uniform(t >> 6);
  const int q = lane >> 4, lr = lane & 15;
  const int64_t n0 = static_cast<int64_t>(blockIdx.x) * NC;
  const int64_t m0 = static_cast<int64_t>(blockIdx.y) * 64;
  const int64_t KS = K / 64;  // K-steps
  const int64_t ks0 = wave * KS / kLinSplit, ks1 = (wave + 1) * KS / kLinSplit;
  const int nks = static_cast<int>(ks1 - ks0);
  uint8_t* my = ring[wave];
  const uint8_t* ab = reinterpret_cast<const uint8_t*>(a);
  const uint8_t* wb = reinterpret_cast<const uint8_t*>(w);

  // copy plan: instruction u fills slot rows 8u..8u+7; lane l fills row
  // 8u + l/8, physical chunk l%8 (logical chunk (l%8) ^ (row & 7))
  const int crow = lane >> 3, pch = lane & 7;
  int64_t a_off[C::AI];
#pragma unroll
  for (int u = 0; u < C::AI; ++u) {
    const int row = 8 * u + crow;
    const int64_t gr = m0 + row < M ? m0 + row : M - 1;
    a_off[u] = gr * K * 2 + ((pch ^ (row & 7)) << 4);
  }
  int64_t w_off[2 * NJ];
#pragma unroll
  for (int u = 0; u < 2 * NJ; ++u) {
    const int row = 8 * u + crow;
    w_off[u] = (n0 + row) * K * 2 + ((pch ^ (row & 7)) << 4);
  }
  auto issue = [&](int s, int slot) {
    const int64_t kb = (ks0 + (s < nks ? s : nks - 1)) * 128;  // byte offset of the K-step
    const uint32_t base = lds_u32(my + slot * C::kSlot);
#pragma unroll
    for (int u = 0; u < C::AI; ++u) dma16(ab + a_off[u] + kb, wave_uniform(static_cast<int>(base) + u * 1024));
#pragma unroll
    for (int u = 0; u < 2 * NJ; ++u)
      dma16(wb + w_off[u] + kb, wave_uniform(static_cast<int>(base) + C::kA + u * 1024));
  };
  if (nks > 0) {
#pragma unroll
    for (int s = 0; s < D - 1; ++s) issue(s, s);
  }
  v4f acc[MT][NJ];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
  for (int s = 0; s < nks; ++s) {
    wait_vm_lds<(D - 2) * C::PER>();  // step s has landed; slot (s-1) % D is read
    issue(s + D - 1, (s + D - 1) % D);
    const uint8_t* slot = my + (s % D) * C::kSlot;
    bf8 alo[MT], ahi[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) lin_frag(slot + i * 16 * 128, lr, q, alo[i], ahi[i]);
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      bf8 blo, bhi;
      lin_frag(slot + C::kA + j * 16 * 128, lr, q, blo, bhi);
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo[i], blo, acc[i][j], 0, 0, 0);
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi[i], bhi, acc[i][j], 0, 0, 0);
      }
    }
  }
  wait_vm<0>();
  __syncthreads();  // every ring is idle: reuse it for the partials
  float* red = reinterpret_cast<float*>(&ring[0][0]);
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[(wave * RA + 16 * i + 4 * q + r) * NC + 16 * j + lr] = acc[i][j][r];
  __syncthreads();
  for (int e = t; e < RA * NC; e += kLinSplit * 64) {
    const int row = e / NC, col = e - row * NC;
    if (m0 + row >= M) continue;
    float sum = red[row * NC + col];
#pragma unroll
    for (int wv = 1; wv < kLinSplit; ++wv) sum += red[(wv * RA + row) * NC + col];
    out[(m0 + row) * N + n0 + col] = static_cast<uint16_t>(f32_to_bf16(sum));
    if (out_tap != nullptr) out_tap[(m0 + row) * N + n0 + col] = sum;
  }
}

// out = a W^T for many rows: BM x BN output tiles, 8 wavefronts (4 bands of
// BM/4 activation rows x 2 bands of BN/2 weight rows), one direct-to-LDS ring
// of 3 stages shared by the workgroup (K-steps of 64 elements: BM activation
// rows and BN weight rows a stage), so a staged activation row serves BN
// weight rows and a staged weight row BM activation rows; with BM = 128, W
// is read once per 128 rows instead of once per 64. Every output element gets exactly the
// arithmetic of linear_bf16_kernel: the same four K quarters, each a chain of
// the same 16x16x32 bf16 MFMAs on the same operand halves (K-step by K-step)
// started from zero, and the quarter sums added in quarter order. So a row's
// result does not depend on which of the two kernels computed it, and a
// block update of the caches still equals a full recompute bit for bit.
constexpr int kLtWaves = 8, kLtS = 3;
#ifndef LACACHE_LIN_TILED_MIN_M
#define LACACHE_LIN_TILED_MIN_M 128
#endif
constexpr int64_t kLinTiledMinM = LACACHE_LIN_TILED_MIN_M;  // rows above which the tiled kernel runs

// BM x BN output tile; wavefront (wm, wn) of 4 x 2 owns BM/4 rows x BN/2
// columns (MT x NT 16x16 tiles)
template <int BM, int BN>
__global__ __launch_bounds__(kLtWaves * 64) void linear_bf16_tiled_kernel(const uint16_t* __restrict__ a,
                                                                        const uint16_t* __restrict__ w,
                                                                        uint16_t* __restrict__ out,
                                                                        float* __restrict__ out_tap, int64_t M,
                                                                        int64_t N, int64_t K) {
  constexpr int kStage = (BM + BN) * 128;             // bytes per stage
  constexpr int kPer = (BM + BN) / 8 / kLtWaves;      // 1 KB copies per wavefront per stage
  constexpr int MT = BM / 64, NT = BN / 32, WRr = BM / 4, WCc = BN / 2;
  static_assert((BM + BN) % (8 * kLtWaves) == 0 && BM % 64 == 0 && BN % 32 == 0, "tile shape");
  __shared__ __align__(16) uint8_t ring[kLtS][kStage];
  const int t = threadIdx.x, lane = t & 63;
  const int wave = wave_uniform(t >> 6);
  const int q = lane >> 4, lr = lane & 15;
  const int wm = wave >> 1, wn = wave & 1;
  // row tiles along x (up to 2^24 / 128 of them; gridDim.y is limited to
  // 65536), column tiles along y
  const int64_t m0 = static_cast<int64_t>(blockIdx.x) * BM;
  const int64_t n0 = static_cast<int64_t>(blockIdx.y) * BN;
  const int KS = static_cast<int>(K / 64);
  const uint8_t* ab = reinterpret_cast<const uint8_t*>(a);
  const uint8_t* wb = reinterpret_cast<const uint8_t*>(w);

  // copy plan: copy u of wavefront v fills stage rows 8 g .. 8 g + 7, g = v + 8 u
  // (rows 0..BM-1 activations, then BN weight rows); lane l fills row 8 g + l/8,
  // physical chunk l%8, i.e. logical chunk (l%8) ^ (row & 7)
  const int crow = lane >> 3, pch = lane & 7;
  int64_t src[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int row = 8 * (wave + kLtWaves * u) + crow;
    const int chunk = (pch ^ (row & 7)) << 4;
    if (row < BM) {
      const int64_t gr = m0 + row < M ? m0 + row : M - 1;
      src[u] = gr * K * 2 + chunk;
    } else {
      src[u] = (n0 + row - BM) * K * 2 + chunk;
    }
  }
  auto issue = [&](int ks, int st) {
    const uint32_t base = lds_u32(&ring[st][0]);
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int g = wave + kLtWaves * u;
      const uint8_t* b = (8 * g < BM ? ab : wb) + src[u] + static_cast<int64_t>(ks) * 128;
      dma16(b, wave_uniform(static_cast<int>(base) + g * 1024));
    }
  };

  v4f acc[MT][NT], tot[MT][NT];
  const v4f zero = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) tot[i][j] = zero;
#pragma unroll
  for (int s = 0; s < kLtS - 1; ++s)
    if (s < KS) issue(s, s);
  int ks = 0;
  for (int qq = 0; qq < kLinSplit; ++qq) {
    const int k1 = (qq + 1) * KS / kLinSplit;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NT; ++j) acc[i][j] = zero;
    for (; ks < k1; ++ks) {
      // this wavefront's copies of step ks have landed (later ones may fly) ...
      if (ks + kLtS - 2 < KS)
        wait_vm<(kLtS - 2) * kPer>();
      else
        wait_vm<0>();
      bar();  // ... and every wavefront's; the stage refilled next is read by no one
      if (ks + kLtS - 1 < KS) issue(ks + kLtS - 1, (ks + kLtS - 1) % kLtS);
      const uint8_t* st = &ring[ks % kLtS][0];
      bf8 alo[MT], ahi[MT];
#pragma unroll
      for (int i = 0; i < MT; ++i) lin_frag(st + (WRr * wm + 16 * i) * 128, lr, q, alo[i], ahi[i]);
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        bf8 blo, bhi;
        lin_frag(st + (BM + WCc * wn + 16 * j) * 128, lr, q, blo, bhi);
#pragma unroll
        for (int i = 0; i < MT; ++i) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo[i], blo, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi[i], bhi, acc[i][j], 0, 0, 0);
        }
      }
    }
    // the quarter's sum joins the total in quarter order (the first is a copy)
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) tot[i][j][r] = qq == 0 ? acc[i][j][r] : tot[i][j][r] + acc[i][j][r];
  }
  wait_vm<0>();
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t row = m0 + WRr * wm + 16 * i + 4 * q + r;
      if (row >= M) continue;
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        const int64_t col = n0 + WCc * wn + 16 * j + lr;
        out[row * N + col] = static_cast<uint16_t>(f32_to_bf16(tot[i][j][r]));
        if (out_tap != nullptr) out_tap[row * N + col] = tot[i][j][r];
      }
    }
}

// One thread per (row r, Q/K/V part, head, pair i < 64): the pair (i, i + 64)
// of the head's 128 values; Q and K rotated by the angle of the row's position.
__global__ __launch_bounds__(256) void rope_scatter_kernel(const uint16_t* __restrict__ qkv,
                                                           const int32_t* __restrict__ rows, int64_t R,
                                                           const float* __restrict__ cs, const float* __restrict__ sn,
                                                           uint16_t* __restrict__ q, uint16_t* __restrict__ k,
                                                           uint16_t* __restrict__ v, int64_t heads, int64_t N) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t per_row = 3 * heads * 64;
  if (e >= R * per_row) return;
  const int64_t r = e / per_row;
  const int64_t rem = e - r * per_row;
  const int part = static_cast<int>(rem / (heads * 64));
  const int64_t h = (rem / 64) % heads;
  const int i = static_cast<int>(rem & 63);
  const int64_t pos = rows[r];
  if (pos < 0 || pos >= N) return;
  const uint16_t* src = qkv + r * 3 * heads * 128 + (part * heads + h) * 128;
  uint16_t* dst = (part == 0 ? q : (part == 1 ? k : v)) + (h * N + pos) * 128;
  const uint16_t x1 = src[i], x2 = src[64 + i];
  if (part == 2) {
    dst[i] = x1;
    dst[64 + i] = x2;
    return;
  }
  const float a = bf16lo(x1), b = bf16lo(x2), c = cs[pos * 64 + i], s = sn[pos * 64 + i];
  dst[i] = static_cast<uint16_t>(f32_to_bf16(a * c - b * s));
  dst[64 + i] = static_cast<uint16_t>(f32_to_bf16(b * c + a * s));
}

}  // namespace

hipError_t launch_embed_rmsnorm(hipStream_t st, const int32_t* ids, const int32_t* rows, int64_t R,
                                const uint16_t* embed, int64_t vocab, const uint16_t* nw, uint16_t* cache, int64_t N,
                                uint16_t* y, int64_t H) {
  const int T = static_cast<int>((H + 511) / 512);
  const dim3 grid(static_cast<unsigned>((R + 3) / 4)), block(256);
  const int h = static_cast<int>(H);
#define ER(T_) \
  hipLaunchKernelGGL(embed_rmsnorm_kernel<T_>, grid, block, 0, st, ids, rows, R, embed, vocab, nw, cache, N, y, h)
  if (T <= 1) ER(1);
  else if (T <= 2) ER(2);
  else if (T <= 4) ER(4);
  else if (T <= 8) ER(8);
  else if (T <= 16) ER(16);
  else ER(32);
#undef ER
  return hipGetLastError();
}

hipError_t launch_linear_bf16(hipStream_t st, const uint16_t* a, const uint16_t* w, uint16_t* out, float* out_tap,
                              int64_t M, int64_t N, int64_t K) {
  if (M > kLinTiledMinM) {
    // many rows: 128-row tiles (N % 128 == 0), W read once per 128 rows
    // 128 x 192 tiles when they need fewer rounds of one workgroup per CU
    // than 128 x 128 (measured at N = 12288, K = 4096: 52 against 72 us at
    // M = 512, 122 against 132 us at M = 1024; at M = 256, with one round
    // either way, 128 x 128 leaves fewer CUs idle: 39 against 47 us)
    const int64_t rt = (M + 127) / 128, cus = device_cu_count();
    const bool wide = N % 192 == 0 && (rt * (N / 192) + cus - 1) / cus < (rt * (N / 128) + cus - 1) / cus;
    const dim3 block(kLtWaves * 64);
    if (wide)
      hipLaunchKernelGGL((linear_bf16_tiled_kernel<128, 192>), dim3(static_cast<unsigned>(rt), static_cast<unsigned>(N / 192)),
                         block, 0, st, a, w, out, out_tap, M, N, K);
    else
      hipLaunchKernelGGL((linear_bf16_tiled_kernel<128, 128>), dim3(static_cast<unsigned>(rt), static_cast<unsigned>(N / 128)),
                         block, 0, st, a, w, out, out_tap, M, N, K);
    return hipGetLastError();
  }
  // up to 64 rows per pass; the last pass may hold fewer slabs. Three weight
  // slabs per workgroup when that still gives a workgroup per CU (few rows),
  // else one.
  const unsigned passes = static_cast<unsigned>((M + 63) / 64);
  const int mt = static_cast<int>(M >= 64 ? 4 : (M + 15) / 16);
  const bool wide = mt <= 2 && N % 48 == 0 && N / 48 >= 256;
  const dim3 grid(static_cast<unsigned>(N / (wide ? 48 : 16)), passes), block(kLinSplit * 64);
#define LB(MT_, NJ_) hipLaunchKernelGGL((linear_bf16_kernel<MT_, NJ_>), grid, block, 0, st, a, w, out, out_tap, M, N, K)
  if (wide) {
    if (mt <= 1) LB(1, 3);
    else LB(2, 3);
  } else if (mt <= 1) LB(1, 1);
  else if (mt == 2) LB(2, 1);
  else if (mt == 3) LB(3, 1);
  else LB(4, 1);
#undef LB
  return hipGetLastError();
}

hipError_t launch_rope_scatter(hipStream_t st, const uint16_t* qkv, const int32_t* rows, int64_t R, const float* cs,
                               const float* sn, uint16_t* q, uint16_t* k, uint16_t* v, int64_t heads, int64_t N) {
  const int64_t threads = R * 3 * heads * 64;
  hipLaunchKernelGGL(rope_scatter_kernel, dim3(static_cast<unsigned>((threads + 255) / 256)), dim3(256), 0, st, qkv,
                     rows, R, cs, sn, q, k, v, heads, N);
  return hipGetLastError();
}

}  // namespace lacache
