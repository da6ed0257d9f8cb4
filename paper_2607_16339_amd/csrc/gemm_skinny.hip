// Skinny-M (M <= 64) FP8 GEMMs for block-only calls: bound by streaming the
// fp8 weights from HBM once, so they are spread over many workgroups that
// each own a thin slice of weight rows and the whole K.
//
//   gate/up: workgroup c owns h-columns [16c, 16c+16): gate rows 16c.. and up
//            rows I+16c.. of Wgu. Its wavefronts split K by interleaved
//            K-groups, each K-group is one 16x16x128 FP8 MFMA per 16-row slab
//            of x, scaled by RN32(x_scale * w_scale) into fp32. The partial
//            sums meet in LDS (fixed order), SwiGLU gives h in fp32, and h is
//            parked in a small fp32 workspace. The 8 workgroups of one
//            128-wide h-group count themselves in; the last to arrive
//            quantizes the group (row amax, scale, e4m3 codes) and re-arms
//            the counter.
//   down:    workgroup c owns output columns [16c, 16c+16) of W_down, same
//            K split and LDS reduction, bf16 store.
#include "device.h"
#include "launch.h"

namespace lacache {
namespace {

constexpr int kCols = 16;                    // weight rows (output columns) per workgroup slice
constexpr int kSlicesPerGroup = kGroup / kCols;

__device__ __forceinline__ v8i load_frag_global(const uint8_t* p) {
  // lane q reads bytes [16q, 16q+16) and [64+16q, 64+16q+16) of the row's K-group
  const uint4 lo = *reinterpret_cast<const uint4*>(p);
  const uint4 hi = *reinterpret_cast<const uint4*>(p + 64);
  v8i f;
  f[0] = static_cast<int>(lo.x); f[1] = static_cast<int>(lo.y); f[2] = static_cast<int>(lo.z); f[3] = static_cast<int>(lo.w);
  f[4] = static_cast<int>(hi.x); f[5] = static_cast<int>(hi.y); f[6] = static_cast<int>(hi.z); f[7] = static_cast<int>(hi.w);
  return f;
}

template <int MT, int NB>
struct SkinnyOperands {
  v8i a[MT];
  v8i b[NB];
  float xs[MT][4];
  float ws[NB];
};

// Loads one K-group's operands: activation slabs (rows 16i + lr, zero past M),
// weight slices and the scales.
template <int MT, int NB>
__device__ __forceinline__ void skinny_load(SkinnyOperands<MT, NB>& o, const uint8_t* __restrict__ aq,
                                            const float* __restrict__ as, const uint8_t* const* wrow,
                                            const float* __restrict__ bs, const int64_t* nb, int64_t kb,
                                            int64_t KB, int64_t M, int64_t K, int q, int lr) {
  const v8i z = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    const int64_t row = 16 * i + lr;
    o.a[i] = row < M ? load_frag_global(aq + row * K + kb * 128 + 16 * q) : z;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t sr = 16 * i + 4 * q + r;
      o.xs[i][r] = sr < M ? as[kb * M + sr] : 0.0f;
    }
  }
#pragma unroll
  for (int n = 0; n < NB; ++n) {
    o.b[n] = load_frag_global(wrow[n] + kb * 128 + 16 * q);
    o.ws[n] = bs[nb[n] * KB + kb];
  }
}

template <int MT, int NB>
__device__ __forceinline__ void skinny_mma(float (&acc)[MT][NB][4], const SkinnyOperands<MT, NB>& o) {
#pragma unroll
  for (int n = 0; n < NB; ++n)
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const v4f zero = {0.0f, 0.0f, 0.0f, 0.0f};
      const v4f p = mfma_fp8_16x16x128(o.a[i], o.b[n], zero);
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[i][n][r] = __builtin_fmaf(p[r], o.xs[i][r] * o.ws[n], acc[i][n][r]);
    }
}

// K loop of one wavefront (K-groups wave, wave + NW, ...) with one K-group of
// operands in flight while the previous one is multiplied.
template <int MT, int NB, int NW>
__device__ __forceinline__ void skinny_kloop(float (&acc)[MT][NB][4], const uint8_t* __restrict__ aq,
                                             const float* __restrict__ as, const uint8_t* const* wrow,
                                             const float* __restrict__ bs, const int64_t* nb, int64_t KB,
                                             int64_t M, int64_t K, int wave, int q, int lr) {
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int n = 0; n < NB; ++n)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[i][n][r] = 0.0f;
  if (wave >= KB) return;
  SkinnyOperands<MT, NB> cur, nxt;
  skinny_load<MT, NB>(cur, aq, as, wrow, bs, nb, wave, KB, M, K, q, lr);
  for (int64_t kb = wave; kb < KB; kb += NW) {
    const bool more = kb + NW < KB;
    if (more) skinny_load<MT, NB>(nxt, aq, as, wrow, bs, nb, kb + NW, KB, M, K, q, lr);
    skinny_mma<MT, NB>(acc, cur);
    if (more) cur = nxt;
  }
}

// Fixed-order sum of the NW wavefronts' accumulators through LDS; wavefront 0
// ends with the totals.
template <int MT, int NB, int NW>
__device__ __forceinline__ void skinny_reduce(float (&acc)[MT][NB][4], float* red, int wave, int lane) {
  constexpr int E = MT * NB * 4;
  if (wave != 0) {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int n = 0; n < NB; ++n)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[((wave - 1) * E + (i * NB + n) * 4 + r) * 64 + lane] = acc[i][n][r];
  }
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int w = 1; w < NW; ++w)
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int n = 0; n < NB; ++n)
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[i][n][r] += red[((w - 1) * E + (i * NB + n) * 4 + r) * 64 + lane];
  }
}

template <int MT, int NW>
__global__ __launch_bounds__(NW * 64) void gateup_skinny_kernel(
    const uint8_t* __restrict__ xq, const float* __restrict__ xs, const uint8_t* __restrict__ wq,
    const float* __restrict__ ws, uint8_t* __restrict__ hq, float* __restrict__ hs, float* __restrict__ h_tap,
    float* __restrict__ hbuf, unsigned* __restrict__ counters, int64_t M, int64_t H, int64_t I) {
  __shared__ float red[(NW - 1) * MT * 2 * 4 * 64];
  __shared__ int last;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int q = lane >> 4, lr = lane & 15;
  const int64_t c = blockIdx.x;
  const int64_t hg = c / kSlicesPerGroup;
  const int64_t KB = H / 128;
  const uint8_t* wrow[2] = {wq + (c * kCols + lr) * H, wq + (I + c * kCols + lr) * H};
  const int64_t nb[2] = {hg, I / 128 + hg};

  float acc[MT][2][4];
  skinny_kloop<MT, 2, NW>(acc, xq, xs, wrow, ws, nb, KB, M, H, wave, q, lr);
  skinny_reduce<MT, 2, NW>(acc, red, wave, lane);

  if (wave == 0) {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = 16 * i + 4 * q + r;
        const float g = acc[i][0][r], u = acc[i][1][r];
        const float h = g / (1.0f + expf(-g)) * u;
        if (row < M) {
          hbuf[row * I + c * kCols + lr] = h;
          if (h_tap != nullptr) h_tap[row * I + c * kCols + lr] = h;
        }
      }
    __threadfence();  // release this slice's h before counting in
    if (lane == 0) last = (atomicAdd(counters + hg, 1u) == kSlicesPerGroup - 1);
  }
  __syncthreads();
  if (!last) return;  // uniform across the workgroup
  __threadfence();    // acquire the other slices' h

  // Last arrival: quantize the 128-wide h-group of every row. Four threads per
  // row, 32 consecutive values each.
  const int64_t row = t >> 2;
  const int part = t & 3;
  for (int64_t r0 = 0; r0 < M; r0 += (NW * 64) / 4) {
    const int64_t rr = r0 + row;
    const bool ok = rr < M;
    float v[32];
    const float4* src = reinterpret_cast<const float4*>(hbuf + rr * I + hg * 128 + part * 32);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float4 f = ok ? src[e] : make_float4(0.f, 0.f, 0.f, 0.f);
      v[4 * e] = f.x; v[4 * e + 1] = f.y; v[4 * e + 2] = f.z; v[4 * e + 3] = f.w;
    }
    float a = 0.0f;
#pragma unroll
    for (int e = 0; e < 32; ++e) a = __builtin_fmaxf(a, __builtin_fabsf(v[e]));
    a = max_xor<4>(a);
    const float s = a / kE4M3Max;
    uint32_t w[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
      w[e] = s == 0.0f ? 0u
                       : enc4_e4m3(qdiv(v[4 * e], s), qdiv(v[4 * e + 1], s), qdiv(v[4 * e + 2], s),
                                   qdiv(v[4 * e + 3], s));
    if (ok) {
      uint4* dst = reinterpret_cast<uint4*>(hq + rr * I + hg * 128 + part * 32);
      dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
      dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
      if (part == 0) hs[hg * M + rr] = s;
    }
  }
  if (t == 0) counters[hg] = 0u;  // re-arm for the next call on this stream
}

template <int MT, int NW>
__global__ __launch_bounds__(NW * 64) void down_skinny_kernel(
    const uint8_t* __restrict__ hq, const float* __restrict__ hs, const uint8_t* __restrict__ wq,
    const float* __restrict__ ws, uint16_t* __restrict__ out, float* __restrict__ out_tap, int64_t M, int64_t H,
    int64_t I) {
  __shared__ float red[(NW - 1) * MT * 1 * 4 * 64];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int q = lane >> 4, lr = lane & 15;
  const int64_t c = blockIdx.x;
  const int64_t KB = I / 128;
  const uint8_t* wrow[1] = {wq + (c * kCols + lr) * I};
  const int64_t nb[1] = {(c * kCols) / 128};

  float acc[MT][1][4];
  skinny_kloop<MT, 1, NW>(acc, hq, hs, wrow, ws, nb, KB, M, I, wave, q, lr);
  skinny_reduce<MT, 1, NW>(acc, red, wave, lane);
  if (wave == 0) {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = 16 * i + 4 * q + r;
        if (row < M) {
          out[row * H + c * kCols + lr] = static_cast<uint16_t>(f32_to_bf16(acc[i][0][r]));
          if (out_tap != nullptr) out_tap[row * H + c * kCols + lr] = acc[i][0][r];
        }
      }
  }
}

constexpr int kGateUpWaves = 4;
constexpr int kDownWaves = 8;

}  // namespace

size_t skinny_gateup_ws_bytes(int64_t M, int64_t I) {
  const size_t h = static_cast<size_t>(M) * static_cast<size_t>(I) * sizeof(float);
  return kSkinnyCounterBytes + ((h + 255) / 256) * 256;
}

// Workspace layout: [counters: kSkinnyCounterBytes][hbuf: M x I fp32]. The
// counters (I/128 words) must be zero when the kernel starts; the kernel
// leaves them zero again.
hipError_t launch_gateup_skinny(hipStream_t st, const uint8_t* xq, const float* xs, const uint8_t* wq,
                                const float* ws, uint8_t* hq, float* hs, float* h_tap, int64_t M, int64_t H,
                                int64_t I, void* ws_buf) {
  unsigned* counters = static_cast<unsigned*>(ws_buf);
  float* hbuf = reinterpret_cast<float*>(static_cast<char*>(ws_buf) + kSkinnyCounterBytes);
  dim3 grid(static_cast<unsigned>(I / kCols)), block(kGateUpWaves * 64);
  const int mt = static_cast<int>((M + 15) / 16);
#define LAUNCH_GU(MT_) \
  hipLaunchKernelGGL((gateup_skinny_kernel<MT_, kGateUpWaves>), grid, block, 0, st, xq, xs, wq, ws, hq, hs, h_tap, hbuf, counters, M, H, I)
  if (mt <= 1) LAUNCH_GU(1);
  else if (mt == 2) LAUNCH_GU(2);
  else if (mt == 3) LAUNCH_GU(3);
  else LAUNCH_GU(4);
#undef LAUNCH_GU
  return hipGetLastError();
}

hipError_t launch_down_skinny(hipStream_t st, const uint8_t* hq, const float* hs, const uint8_t* wq, const float* ws,
                              uint16_t* out, float* out_tap, int64_t M, int64_t H, int64_t I) {
  dim3 grid(static_cast<unsigned>(H / kCols)), block(kDownWaves * 64);
  const int mt = static_cast<int>((M + 15) / 16);
#define LAUNCH_DN(MT_) \
  hipLaunchKernelGGL((down_skinny_kernel<MT_, kDownWaves>), grid, block, 0, st, hq, hs, wq, ws, out, out_tap, M, H, I)
  if (mt <= 1) LAUNCH_DN(1);
  else if (mt == 2) LAUNCH_DN(2);
  else if (mt == 3) LAUNCH_DN(3);
  else LAUNCH_DN(4);
#undef LAUNCH_DN
  return hipGetLastError();
}

}  // namespace lacache
