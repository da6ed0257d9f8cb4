// Device helpers for the gfx950 FP8 FFN kernels: e4m3 encoding, bf16
// conversion, the FP8 MFMA and wavefront reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lacache {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kGroup = 128;      // quantization group (1x128 activations, 128x128 weights)
constexpr float kE4M3Max = 448.0f;

// ---------------------------------------------------------------------------
// Layout of FP8 weight codes W [N x K] (N a multiple of 16, K of 128): tiles
// of 16 rows x 128 columns (one K-group), 2 KB each, tile (n/16, k/128) at
// byte ((n/16) (K/128) + k/128) 2048, so a 16-row slab's K range is one
// contiguous run starting at byte 16 (n/16) K, as in a row-major matrix.
// Inside a tile the first 1 KB holds columns 0..63 of the 16 rows (64 bytes
// per row, row after row) and the second 1 KB columns 64..127. The 16x16x128
// MFMA operand of a slab then takes exactly the two 1 KB halves of a tile,
// one 16-byte load per lane each, so register loads of the weights read 1 KB
// contiguous per instruction.
// ---------------------------------------------------------------------------
__host__ __device__ inline int64_t wtile_off(int64_t n, int64_t k, int64_t K) {
  return ((n >> 4) * (K >> 7) + (k >> 7)) * 2048 + ((k >> 6) & 1) * 1024 + (n & 15) * 64 + (k & 63);
}

// ---------------------------------------------------------------------------
// e4m3fn encoding: clip to [-448, 448] (Eq. 7), then the hardware's
// round-to-nearest-even conversion. The conversion itself does not saturate
// (values above 464 become the NaN code), so the clip must come first. The
// clip keeps the sign of zero, so -0 encodes to 0x80.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float clip448(float v) {
  return __builtin_fminf(__builtin_fmaxf(v, -kE4M3Max), kE4M3Max);
}

// Four values -> four codes packed little-endian into one 32-bit word.
__device__ __forceinline__ uint32_t enc4_e4m3(float a, float b, float c, float d) {
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(clip448(a), clip448(b), 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(clip448(c), clip448(d), w, true);
  return static_cast<uint32_t>(w);
}

__device__ __forceinline__ uint32_t enc1_e4m3(float a) {
  return static_cast<uint32_t>(__builtin_amdgcn_cvt_pk_fp8_f32(clip448(a), 0.0f, 0, false)) & 0xFFu;
}

// Group quantizer step for one value: code = E(RN32(y / s)), s > 0. The
// division is IEEE-correctly rounded (the library is compiled with correctly
// rounded fp32 division).
__device__ __forceinline__ float qdiv(float y, float s) { return y / s; }

// The same code, E(RN32(y / s)), from the hardware reciprocal rs = rcp(s)
// (1 ulp): q0 = y * rs is within 2^-22 (relative) of y / s, so when the codes
// of q0 * (1 - 2^-20) and q0 * (1 + 2^-20) agree, that is the code of every
// value in between, RN32(y / s) included (the encoder is monotone). Otherwise
// the value sits at an e4m3 rounding boundary and the correctly rounded
// division decides. Requires s >= 2^-100 (see scale_is_fast).
__device__ __forceinline__ uint32_t enc1_div_fast(float y, float s, float rs) {
  const float q0 = y * rs;
  const float d = __builtin_fabsf(q0) * 0x1p-20f;
  const uint32_t w = static_cast<uint32_t>(__builtin_amdgcn_cvt_pk_fp8_f32(clip448(q0 - d), clip448(q0 + d), 0, false));
  if ((w & 0xFFu) == ((w >> 8) & 0xFFu)) return w & 0xFFu;
  return enc1_e4m3(y / s);
}
__device__ __forceinline__ bool scale_is_fast(float s) { return s >= 0x1p-100f; }

// Eight values at once, branch-free: the codes of q0 * (1 -+ 2^-20) for
// each value (q0 = y * rs), as in enc1_div_fast. Returns true when all eight
// pairs agree; the codes in lo/hi are then E(RN32(y / s)). Otherwise the
// caller redoes the eight with the correctly rounded division.
__device__ __forceinline__ bool enc8_div_fast(const float (&y)[8], float rs, uint32_t& lo, uint32_t& hi) {
  float m[8], p[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float q0 = y[e] * rs;
    const float d = __builtin_fabsf(q0) * 0x1p-20f;
    m[e] = q0 - d;
    p[e] = q0 + d;
  }
  lo = enc4_e4m3(m[0], m[1], m[2], m[3]);
  hi = enc4_e4m3(m[4], m[5], m[6], m[7]);
  const uint32_t lo2 = enc4_e4m3(p[0], p[1], p[2], p[3]);
  const uint32_t hi2 = enc4_e4m3(p[4], p[5], p[6], p[7]);
  return ((lo ^ lo2) | (hi ^ hi2)) == 0u;
}
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

// The bracket of enc1_div_fast with the factors folded into the reciprocal:
// rl = RN32(rcp(s) (1 - 2^-20)), rh = RN32(rcp(s) (1 + 2^-20)). For a group
// with amax = max|y| and s = RN32(amax / 448) >= 2^-100, and rcp within 2^-22
// of 1/s, every y of the group has
//   |y rl| < |RN32(y / s)| < |y rh|  (y != 0; both products have its sign),
// since (1 - 2^-20) (1 + 2^-22) (1 + 2^-24)^2 < 1 - 2^-21 < 1 - 2^-24, and
// likewise above; and |y rh| < 448 (1 + 2^-19) < 464, below the conversion's
// NaN threshold, so no clip is needed. Where the codes of y rl and y rh agree,
// that is E(RN32(y / s)) (the encoder is monotone).
struct FastQuant {
  float rl, rh;
};
__device__ __forceinline__ FastQuant fast_quant(float s) {
  const float rs = __builtin_amdgcn_rcpf(s);
  return {rs * (1.0f - 0x1p-20f), rs * (1.0f + 0x1p-20f)};
}
// Codes of four values by the bracket: returns the codes from y rl in lo and
// whether they equal the codes from y rh.
__device__ __forceinline__ bool enc4_bracket(float a, float b, float c, float d, FastQuant f, uint32_t& lo) {
  int w0 = __builtin_amdgcn_cvt_pk_fp8_f32(a * f.rl, b * f.rl, 0, false);
  w0 = __builtin_amdgcn_cvt_pk_fp8_f32(c * f.rl, d * f.rl, w0, true);
  int w1 = __builtin_amdgcn_cvt_pk_fp8_f32(a * f.rh, b * f.rh, 0, false);
  w1 = __builtin_amdgcn_cvt_pk_fp8_f32(c * f.rh, d * f.rh, w1, true);
  lo = static_cast<uint32_t>(w0);
  return w0 == w1;
}

// SiLU(g) * u in fp32 with the hardware exp2 and reciprocal (a few ulp).
__device__ __forceinline__ float swiglu_fast(float g, float u) {
  const float e = __builtin_amdgcn_exp2f(-g * 1.44269504088896341f);
  return g * fast_rcp(1.0f + e) * u;
}

// ---------------------------------------------------------------------------
// RMSNorm fused with the 1x128 quantizer, the arithmetic shared by every
// kernel that normalizes a row (the same operations in the same order, so
// the codes and scales are bit-identical wherever they are computed).
// A wavefront owns a row: lane l holds the 16-byte chunks c = 64 t + l (8
// bf16 each), so a 128-wide group is 16 consecutive lanes of one pass t.
// ---------------------------------------------------------------------------
// p + the squares of the chunk's 8 values in element order (each square of a
// bf16 value is exact in fp64).
__device__ __forceinline__ double sumsq8(double p, uint4 v);
// r = RN32(1 / sqrt(ss / H + 1e-5)) from the row's fp64 sum of squares (ss =
// the xor-butterfly total of the lanes' partials), every step in fp64.
__device__ __forceinline__ float rms_inv(double ss, int H) {
  return static_cast<float>(1.0 / __builtin_sqrt(ss / static_cast<double>(H) + 1e-5));
}
// y = RN32(RN32(x w) r) of a chunk's 8 values (x w is exact in fp32).
__device__ __forceinline__ void norm8(uint4 xv, uint4 wv, float r, float (&y)[8]);
// The 1x128 group quantizer of a chunk's 8 values y within its 16-lane group:
// returns the group scale s = RN32(max|y| / 448) and the codes E(RN32(y / s))
// (all 0x00 when s == 0). Every lane of the 16 must call it.
__device__ __forceinline__ float quant8_group(const float (&y)[8], uint32_t& lo, uint32_t& hi);

// ---------------------------------------------------------------------------
// bf16 <-> fp32
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Round to nearest, ties to even; NaN -> quiet NaN.
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return f32_to_bf16(lo) | (f32_to_bf16(hi) << 16);
}

// ---------------------------------------------------------------------------
// FP8 x FP8 -> fp32 MFMA, 16x16 output, 128-deep K (exactly one K-group).
// Operand layout (per lane l of the wavefront): A row l%16, B column l%16,
// 32 bytes of K each; A and B must place K identically. Output: lane l holds
// D[4*(l/16) + r][l%16] in element r. Zero scale operands select the
// unscaled FP8 (e4m3, format 0) instruction.
// ---------------------------------------------------------------------------
__device__ __forceinline__ v4f mfma_fp8_16x16x128(v8i a, v8i b, v4f c) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// An int the compiler can see is the same in every lane of the wavefront.
__device__ __forceinline__ int wave_uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// ---------------------------------------------------------------------------
// Direct-to-LDS streaming with explicit waits. The copies are inline asm, so
// the compiler neither waits for them nor moves memory accesses across them;
// the kernels wait with explicit vmcnt counts (loads retire in issue order).
// ---------------------------------------------------------------------------
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// LDS byte address of a pointer into __shared__ memory.
__device__ __forceinline__ uint32_t lds_u32(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) char*)(p)));
}
// 16 bytes per lane global -> LDS: lane l lands at lds + 16 l (lds wave-uniform).
__device__ __forceinline__ void dma16(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds) : "memory", "m0");
}
// The same with a wave-uniform 64-bit base in SGPRs and a 32-bit per-lane
// byte offset (the global instructions' scalar-base form): no 64-bit address
// arithmetic per lane.
__device__ __forceinline__ void dma16s(const void* sbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
}
__device__ __forceinline__ void dma4s(const void* sbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1" ::"v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// s_waitcnt vmcnt(n), n < 64, other counters untouched (gfx9 encoding: vmcnt
// in bits 3:0 and 15:14, expcnt 6:4 and lgkmcnt 11:8 at their maxima).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}
// s_waitcnt vmcnt(n) lgkmcnt(0): this wave's copies up to the n most recent
// have landed, and its LDS reads have returned.
template <int N>
__device__ __forceinline__ void wait_vm_lds() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0070 | (N & 15) | ((N >> 4) << 14));
}
// s_waitcnt lgkmcnt(0): this wave's LDS accesses are done (copies in flight
// are not waited for).
__device__ __forceinline__ void wait_lds() { __builtin_amdgcn_s_waitcnt(0xC07F); }
// Workgroup barrier without a memory fence (a fence would drain the copies in
// flight); the empty asm statements keep LDS accesses from moving across it.
__device__ __forceinline__ void bar() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// ---------------------------------------------------------------------------
// Wavefront reductions (max is exact, so order does not matter)
// ---------------------------------------------------------------------------
template <int kWidth>
__device__ __forceinline__ float max_xor(float v) {
#pragma unroll
  for (int o = kWidth / 2; o >= 1; o >>= 1) v = __builtin_fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// ---- definitions of the RMSNorm + quantizer helpers declared above

__device__ __forceinline__ double sumsq8(double p, uint4 v) {
  const uint32_t q[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    // the square of a bf16 value is exact in fp64, so the fused form rounds
    // once where the separate add does: the same sum, one instruction
    const double a = bf16lo(q[e]), b = bf16hi(q[e]);
    p = __builtin_fma(a, a, p);
    p = __builtin_fma(b, b, p);
  }
  return p;
}

__device__ __forceinline__ void norm8(uint4 xv, uint4 wv, float r, float (&y)[8]) {
  const uint32_t q[4] = {xv.x, xv.y, xv.z, xv.w};
  const uint32_t g[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    y[2 * e] = (bf16lo(q[e]) * bf16lo(g[e])) * r;  // x*w is exact in fp32; one rounding for *r
    y[2 * e + 1] = (bf16hi(q[e]) * bf16hi(g[e])) * r;
  }
}

__device__ __forceinline__ float quant8_group(const float (&y)[8], uint32_t& lo, uint32_t& hi) {
  float amax = 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) amax = __builtin_fmaxf(amax, __builtin_fabsf(y[e]));
  amax = max_xor<16>(amax);
  const float s = amax / kE4M3Max;
  lo = 0u;
  hi = 0u;
  if (s != 0.0f && !(scale_is_fast(s) && enc8_div_fast(y, fast_rcp(s), lo, hi))) {
    lo = enc4_e4m3(qdiv(y[0], s), qdiv(y[1], s), qdiv(y[2], s), qdiv(y[3], s));
    hi = enc4_e4m3(qdiv(y[4], s), qdiv(y[5], s), qdiv(y[6], s), qdiv(y[7], s));
  }
  return s;
}

}  // namespace lacache
