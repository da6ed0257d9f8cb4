// Quantization kernels: 128x128 weight blocks, the fused RMSNorm + 1x128
// activation quantizer, the residual add and the encoder test hook.
// Paper: LaCache (arxiv 2607.16339), Sec. 3.4, Eqs. 7-8.
#include "device.h"
#include "launch.h"

namespace lacache {

// ---------------------------------------------------------------------------
// 128x128 block weight quantization. One workgroup (256 threads) per block:
// thread t owns row t/2 of the block, 64 consecutive elements (128 bytes of
// bf16); its 64 codes are one row's half of a 16 x 128 tile (wtile_off).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void quant_weights_kernel(const uint16_t* __restrict__ w, uint8_t* __restrict__ wq,
                                                            float* __restrict__ ws, int64_t K) {
  __shared__ float red[4];
  const int t = threadIdx.x;
  const int64_t kb = blockIdx.x, nb = blockIdx.y;
  const int64_t row = nb * kGroup + (t >> 1);
  const int64_t col = kb * kGroup + (t & 1) * 64;
  const uint4* src = reinterpret_cast<const uint4*>(w + row * K + col);
  uint4 v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = src[i];
  float amax = 0.0f;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t q[4] = {v[i].x, v[i].y, v[i].z, v[i].w};
#pragma unroll
    for (int e = 0; e < 4; ++e)
      amax = __builtin_fmaxf(amax, __builtin_fmaxf(__builtin_fabsf(bf16lo(q[e])), __builtin_fabsf(bf16hi(q[e]))));
  }
  amax = max_xor<64>(amax);
  if ((t & 63) == 0) red[t >> 6] = amax;
  __syncthreads();
  amax = __builtin_fmaxf(__builtin_fmaxf(red[0], red[1]), __builtin_fmaxf(red[2], red[3]));
  const float s = amax / kE4M3Max;  // Eq. 8, rounded once to fp32
  uint32_t out[16];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t q[4] = {v[i].x, v[i].y, v[i].z, v[i].w};
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if (s == 0.0f) {
        out[2 * i + h] = 0u;
      } else {
        out[2 * i + h] = enc4_e4m3(qdiv(bf16lo(q[2 * h]), s), qdiv(bf16hi(q[2 * h]), s),
                                   qdiv(bf16lo(q[2 * h + 1]), s), qdiv(bf16hi(q[2 * h + 1]), s));
      }
    }
  }
  uint4* dst = reinterpret_cast<uint4*>(wq + wtile_off(row, col, K));
#pragma unroll
  for (int i = 0; i < 4; ++i) dst[i] = make_uint4(out[4 * i], out[4 * i + 1], out[4 * i + 2], out[4 * i + 3]);
  if (t == 0) ws[nb * (K / kGroup) + kb] = s;
}

hipError_t launch_quant_weights(hipStream_t st, const uint16_t* w, uint8_t* wq, float* ws, int64_t N, int64_t K) {
  dim3 grid(static_cast<unsigned>(K / kGroup), static_cast<unsigned>(N / kGroup));
  hipLaunchKernelGGL(quant_weights_kernel, grid, dim3(256), 0, st, w, wq, ws, K);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Row-major e4m3 codes [N x K] -> the weight tile layout (wtile_off). A
// 16-byte run of a row (k a multiple of 16) stays contiguous in the tile
// layout (it lies inside one 64-column half of a tile), so each thread moves
// one run: loads are contiguous across the wavefront, stores are 64-byte
// segments.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void pack_weights_kernel(const uint8_t* __restrict__ w, uint8_t* __restrict__ wt,
                                                           int64_t N, int64_t K) {
  const int64_t runs = K / 16;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= N * runs) return;
  const int64_t n = i / runs, k = (i - n * runs) * 16;
  *reinterpret_cast<uint4*>(wt + wtile_off(n, k, K)) = *reinterpret_cast<const uint4*>(w + n * K + k);
}

hipError_t launch_pack_weights(hipStream_t st, const uint8_t* w, uint8_t* wt, int64_t N, int64_t K) {
  const int64_t threads = N * (K / 16);
  hipLaunchKernelGGL(pack_weights_kernel, dim3(static_cast<unsigned>((threads + 255) / 256)), dim3(256), 0, st, w, wt,
                     N, K);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Fused RMSNorm + 1x128 quantization. A row belongs to 1 << wpr_log2
// wavefronts; lane l of each holds chunks c = 64 t + l (8 bf16 each) for
// t < T, so a 128-wide group is the 16 lanes 16g'..16g'+15 of one pass. The
// fp64 sum of squares follows the fixed order: per-lane partials in
// increasing element index, then a xor butterfly over offsets 32..1 (every
// lane ends with the same bits); each wavefront of the row computes it, and
// quantizes the passes t with t mod (1 << wpr_log2) equal to its index in the
// row (several wavefronts per row shorten the path of a small-M call).
// With y (the fused AddNorm), the row is first x = RNE_bf16(float(x) +
// float(y)), written back in place: each wavefront of the row writes its own
// passes, after a workgroup barrier that follows every wavefront's reads of
// the old row. With kF32Out the normalized row goes to
// yf (fp32) instead of being quantized (the coarse-granularity paths).
// ---------------------------------------------------------------------------
template <int T, bool kF32Out = false, bool kAdd = false>
__global__ __launch_bounds__(256, T <= 8 && !kAdd ? 4 : 1) void rmsnorm_quant_kernel(uint16_t* x, const uint16_t* __restrict__ y,
                                                            const uint16_t* __restrict__ nw,
                                                            uint8_t* __restrict__ xq, float* __restrict__ xs,
                                                            int64_t M, int H, int wpr_log2, float* __restrict__ yf) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int part = wave & ((1 << wpr_log2) - 1);
  const int64_t row = (static_cast<int64_t>(blockIdx.x) * (blockDim.x >> 6) + wave) >> wpr_log2;
  // uniform per wavefront, and per workgroup when a row has several
  // wavefronts (the workgroup is then that row): the AddNorm barrier below is
  // reached by every wavefront of the workgroup or by none
  if (row >= M) return;
  const int nchunk = H >> 3;
  const uint4* xr = reinterpret_cast<const uint4*>(x + row * H);  // (read before any write of the row)
  const uint4* wr = reinterpret_cast<const uint4*>(nw);
  // every load of the row and of the norm weight is issued before any is
  // used (clamped indices keep them unconditional), so the wavefront waits
  // for memory once
  uint4 xv[T], wv[T], yv[kAdd ? T : 1];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int c = t * 64 + lane;
    const int cc = c < nchunk ? c : nchunk - 1;
    xv[t] = xr[cc];
    wv[t] = wr[cc];
    if constexpr (kAdd) yv[t] = reinterpret_cast<const uint4*>(y + row * H)[cc];
  }
  if constexpr (kAdd) {  // the residual add, in registers (written back below)
#pragma unroll
    for (int t = 0; t < T; ++t) {
      uint32_t* a = reinterpret_cast<uint32_t*>(&xv[t]);
      const uint32_t* b = reinterpret_cast<const uint32_t*>(&yv[t]);
#pragma unroll
      for (int e = 0; e < 4; ++e) a[e] = pack_bf16x2(bf16lo(a[e]) + bf16lo(b[e]), bf16hi(a[e]) + bf16hi(b[e]));
    }
  }
#pragma unroll
  for (int t = 0; t < T; ++t)
    if (t * 64 + lane >= nchunk) xv[t] = make_uint4(0u, 0u, 0u, 0u);
  double p = 0.0;
#pragma unroll
  for (int t = 0; t < T; ++t) p = sumsq8(p, xv[t]);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) p = p + __shfl_xor(p, o, 64);
  const float r = rms_inv(p, H);
  if constexpr (kAdd) {
    // every wavefront of the row has used all of the old row (the sum above)
    // before any writes its passes of the new one; the row's wavefronts are
    // one workgroup (wpr_log2 > 0) or a single wavefront
    if (wpr_log2 > 0) __syncthreads();
    uint4* xw = reinterpret_cast<uint4*>(x + row * H);
#pragma unroll
    for (int t = 0; t < T; ++t)
      if ((t & ((1 << wpr_log2) - 1)) == part && t * 64 + lane < nchunk) xw[t * 64 + lane] = xv[t];
  }
#pragma unroll
  for (int t = 0; t < T; ++t) {
    if ((t & ((1 << wpr_log2) - 1)) != part) continue;  // uniform
    const int c = t * 64 + lane;
    const bool valid = c < nchunk;  // whole 16-lane groups share validity (H % 128 == 0)
    float y[8];
    norm8(xv[t], wv[t], r, y);
    if (kF32Out) {
      if (valid) {
        float4* d = reinterpret_cast<float4*>(yf + row * H + 8 * c);
        d[0] = make_float4(y[0], y[1], y[2], y[3]);
        d[1] = make_float4(y[4], y[5], y[6], y[7]);
      }
      continue;
    }
    uint32_t lo, hi;
    const float s = quant8_group(y, lo, hi);
    if (valid) {
      *reinterpret_cast<uint2*>(xq + row * H + 8 * c) = make_uint2(lo, hi);
      if ((lane & 15) == 0) xs[static_cast<int64_t>(c >> 4) * M + row] = s;
    }
  }
}

hipError_t launch_rmsnorm_quant(hipStream_t st, uint16_t* x, const uint16_t* nw, uint8_t* xq, float* xs, int64_t M,
                                int64_t H, const uint16_t* y) {
  const int T = static_cast<int>((H + 511) / 512);
  // small M: up to 4 wavefronts per row (one row per workgroup); large M:
  // one wavefront per row, 4 rows per workgroup
  int wl = 0;
  if (M <= 1024) wl = T >= 4 ? 2 : (T >= 2 ? 1 : 0);
  const int64_t waves = M << wl;
  const int per_block = wl > 0 ? (1 << wl) : 4;
  dim3 grid(static_cast<unsigned>((waves + per_block - 1) / per_block)), block(64 * per_block);
  const int h = static_cast<int>(H);
#define NQ(T_)                                                                                                    \
  do {                                                                                                            \
    if (y != nullptr)                                                                                             \
      hipLaunchKernelGGL((rmsnorm_quant_kernel<T_, false, true>), grid, block, 0, st, x, y, nw, xq, xs, M, h, wl,  \
                         nullptr);                                                                                \
    else                                                                                                          \
      hipLaunchKernelGGL((rmsnorm_quant_kernel<T_, false, false>), grid, block, 0, st, x, y, nw, xq, xs, M, h, wl, \
                         nullptr);                                                                                \
  } while (0)
  if (T <= 1) NQ(1);
  else if (T <= 2) NQ(2);
  else if (T <= 4) NQ(4);
  else if (T <= 8) NQ(8);
  else if (T <= 16) NQ(16);
  else NQ(32);
#undef NQ
  return hipGetLastError();
}

hipError_t launch_rmsnorm_f32(hipStream_t st, const uint16_t* x, const uint16_t* nw, float* yf, int64_t M, int64_t H) {
  const int T = static_cast<int>((H + 511) / 512);
  const dim3 grid(static_cast<unsigned>((M + 3) / 4)), block(256);  // one wavefront per row
  uint16_t* xr = const_cast<uint16_t*>(x);                            // only read (no residual)
  const int h = static_cast<int>(H);
#define NF(T_)                                                                                                  \
  hipLaunchKernelGGL((rmsnorm_quant_kernel<T_, true>), grid, block, 0, st, xr, nullptr, nw, nullptr, nullptr, M, h, \
                     0, yf)
  if (T <= 1) NF(1);
  else if (T <= 2) NF(2);
  else if (T <= 4) NF(4);
  else if (T <= 8) NF(8);
  else if (T <= 16) NF(16);
  else NF(32);
#undef NF
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Residual add: x = RNE_bf16(float(x) + float(y)). 8 elements per thread.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void add_bf16_kernel(uint16_t* __restrict__ x, const uint16_t* __restrict__ y,
                                                       int64_t n) {
  const int64_t i8 = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 8;
  if (i8 + 8 <= n) {
    uint4 a = *reinterpret_cast<const uint4*>(x + i8);
    const uint4 b = *reinterpret_cast<const uint4*>(y + i8);
    uint32_t* pa = reinterpret_cast<uint32_t*>(&a);
    const uint32_t* pb = reinterpret_cast<const uint32_t*>(&b);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      pa[e] = pack_bf16x2(bf16lo(pa[e]) + bf16lo(pb[e]), bf16hi(pa[e]) + bf16hi(pb[e]));
    *reinterpret_cast<uint4*>(x + i8) = a;
  } else {
    for (int64_t i = i8; i < n; ++i)
      x[i] = static_cast<uint16_t>(f32_to_bf16(bf16lo(x[i]) + bf16lo(y[i])));
  }
}

hipError_t launch_add_bf16(hipStream_t st, uint16_t* x, const uint16_t* y, int64_t n) {
  const int64_t threads = (n + 7) / 8;
  hipLaunchKernelGGL(add_bf16_kernel, dim3(static_cast<unsigned>((threads + 255) / 256)), dim3(256), 0, st, x, y, n);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Encoder test hook: codes[i] = E(v[i]).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void encode_kernel(const float* __restrict__ v, uint8_t* __restrict__ codes,
                                                     int64_t n) {
  const int64_t i4 = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 4;
  if (i4 + 4 <= n) {
    const float4 f = *reinterpret_cast<const float4*>(v + i4);
    *reinterpret_cast<uint32_t*>(codes + i4) = enc4_e4m3(f.x, f.y, f.z, f.w);
  } else {
    for (int64_t i = i4; i < n; ++i) codes[i] = static_cast<uint8_t>(enc1_e4m3(v[i]));
  }
}

hipError_t launch_encode_e4m3(hipStream_t st, const float* v, uint8_t* codes, int64_t n) {
  const int64_t threads = (n + 3) / 4;
  hipLaunchKernelGGL(encode_kernel, dim3(static_cast<unsigned>((threads + 255) / 256)), dim3(256), 0, st, v, codes, n);
  return hipGetLastError();
}

}  // namespace lacache
