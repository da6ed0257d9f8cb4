// Coarse quantization granularities of the FFN (Sec. 4, Table
// fp8-granularities): one scale per row (per token for activations, per
// output channel for weights) or one scale per tensor, against the library's
// 1x128 / 128x128 groups. The quantizer itself is the same (Eqs. 7-8):
// scale = RN32(max|v| / 448), code = E(RN32(v / scale)), an all-zero set gets
// scale 0 and codes 0x00; only the set of values sharing a scale changes.
//
// A coarse scale needs the max over a whole row (or tensor), which no GEMM
// tile sees, so these paths quantize in separate passes over an fp32 (or
// bf16) source: the row maxima, then the scales (a reduction over the rows
// for a tensor), then the codes. The scales are also written in the GEMMs'
// K-group-major layout (every K-group of row m carries row m's scale), so the
// tiled GEMMs run unchanged; a weight's per-row scales are applied in the
// GEMM epilogue to each output column.
#include "device.h"
#include "launch.h"

namespace lacache {
namespace {

template <typename T>
struct Load8;
// eight consecutive values as fp32
template <>
struct Load8<float> {
  static __device__ __forceinline__ void run(const float* p, float (&v)[8]) {
    const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
};
template <>
struct Load8<uint16_t> {
  static __device__ __forceinline__ void run(const uint16_t* p, float (&v)[8]) {
    const uint4 a = *reinterpret_cast<const uint4*>(p);
    v[0] = bf16lo(a.x); v[1] = bf16hi(a.x); v[2] = bf16lo(a.y); v[3] = bf16hi(a.y);
    v[4] = bf16lo(a.z); v[5] = bf16hi(a.z); v[6] = bf16lo(a.w); v[7] = bf16hi(a.w);
  }
};

// amax[row] = max |v[row, :]| (exact); one workgroup of 256 threads per row.
template <typename T>
__global__ __launch_bounds__(256) void row_amax_kernel(const T* __restrict__ v, float* __restrict__ amax, int64_t K) {
  __shared__ float red[4];
  const int64_t row = blockIdx.x;
  float a = 0.0f;
  for (int64_t k = static_cast<int64_t>(threadIdx.x) * 8; k < K; k += 256 * 8) {
    float x[8];
    Load8<T>::run(v + row * K + k, x);
#pragma unroll
    for (int e = 0; e < 8; ++e) a = __builtin_fmaxf(a, __builtin_fabsf(x[e]));
  }
  a = max_xor<64>(a);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = a;
  __syncthreads();
  if (threadIdx.x == 0) amax[row] = __builtin_fmaxf(__builtin_fmaxf(red[0], red[1]), __builtin_fmaxf(red[2], red[3]));
}

// In place: s[m] = RN32(amax[m] / 448) (per row), or RN32(max_m amax[m] / 448)
// for every m (per tensor). One workgroup of 1024 threads.
__global__ __launch_bounds__(1024) void row_scales_kernel(float* __restrict__ s, int64_t M, int per_tensor) {
  __shared__ float red[16];
  if (per_tensor) {
    float a = 0.0f;
    for (int64_t m = threadIdx.x; m < M; m += 1024) a = __builtin_fmaxf(a, s[m]);
    a = max_xor<64>(a);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = a;
    __syncthreads();  // every thread has read its amax values before any is overwritten
    float t = red[0];
#pragma unroll
    for (int w = 1; w < 16; ++w) t = __builtin_fmaxf(t, red[w]);
    const float sc = t / kE4M3Max;
    for (int64_t m = threadIdx.x; m < M; m += 1024) s[m] = sc;
  } else {
    for (int64_t m = threadIdx.x; m < M; m += 1024) s[m] = s[m] / kE4M3Max;
  }
}

// codes[m, k] = E(RN32(v[m, k] / s[m])) (0x00 for s == 0); eight values per
// thread; with kgm non-null every K-group's first thread of row m also writes
// kgm[kb * M + m] = s[m]. kTiled: the codes go to the weight tile layout
// (wtile_off) instead of row-major.
template <typename T, bool kTiled>
__global__ __launch_bounds__(256) void quant_rows_kernel(const T* __restrict__ v, const float* __restrict__ s,
                                                         uint8_t* __restrict__ codes, float* __restrict__ kgm,
                                                         int64_t M, int64_t K) {
  const int64_t e = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 8;
  if (e >= M * K) return;
  const int64_t row = e / K, col = e - row * K;
  float y[8];
  Load8<T>::run(v + e, y);
  const float sc = s[row];
  uint32_t lo = 0u, hi = 0u;
  if (sc != 0.0f && !(scale_is_fast(sc) && enc8_div_fast(y, fast_rcp(sc), lo, hi))) {
    lo = enc4_e4m3(qdiv(y[0], sc), qdiv(y[1], sc), qdiv(y[2], sc), qdiv(y[3], sc));
    hi = enc4_e4m3(qdiv(y[4], sc), qdiv(y[5], sc), qdiv(y[6], sc), qdiv(y[7], sc));
  }
  *reinterpret_cast<uint2*>(codes + (kTiled ? wtile_off(row, col, K) : e)) = make_uint2(lo, hi);
  if (kgm != nullptr && (col & (kGroup - 1)) == 0) kgm[(col / kGroup) * M + row] = sc;
}

__global__ __launch_bounds__(256) void fill_kernel(float* __restrict__ p, float v, int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) p[i] = v;
}

template <typename T, bool kTiled>
hipError_t quant_rows(hipStream_t st, const T* v, uint8_t* codes, float* kgm, float* s_rows, int64_t M, int64_t K,
                      int per_tensor) {
  hipLaunchKernelGGL(row_amax_kernel<T>, dim3(static_cast<unsigned>(M)), dim3(256), 0, st, v, s_rows, K);
  hipLaunchKernelGGL(row_scales_kernel, dim3(1), dim3(1024), 0, st, s_rows, M, per_tensor);
  const int64_t threads = M * K / 8;
  hipLaunchKernelGGL((quant_rows_kernel<T, kTiled>), dim3(static_cast<unsigned>((threads + 255) / 256)), dim3(256), 0, st, v,
                     s_rows, codes, kgm, M, K);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_quant_rows_f32(hipStream_t st, const float* v, uint8_t* codes, float* kgm, float* s_rows, int64_t M,
                                 int64_t K, bool per_tensor) {
  return quant_rows<float, false>(st, v, codes, kgm, s_rows, M, K, per_tensor ? 1 : 0);
}

hipError_t launch_quant_weights_rows(hipStream_t st, const uint16_t* w, uint8_t* wq, float* w_blocks, float* w_rows,
                                     int64_t N, int64_t K, bool per_tensor) {
  const hipError_t e = quant_rows<uint16_t, true>(st, w, wq, nullptr, w_rows, N, K, per_tensor ? 1 : 0);
  if (e != hipSuccess) return e;
  const int64_t nb = (N / kGroup) * (K / kGroup);
  hipLaunchKernelGGL(fill_kernel, dim3(static_cast<unsigned>((nb + 255) / 256)), dim3(256), 0, st, w_blocks, 1.0f, nb);
  return hipGetLastError();
}

}  // namespace lacache
