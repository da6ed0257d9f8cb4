// First-layer FlashAttention with FACache (Sec. 3.3, FACache; Eqs. 2-6).
//
// One workgroup per (head, block of 64 query rows); 4 wavefronts of 16 rows.
// Key/value blocks of 64 rows stream through LDS; per block every wavefront
//   * computes S^T = K Q^T with bf16 MFMAs (16x16x32): lane (g, r) of a 16x16
//     output tile holds keys 4g..4g+3 of query row r, so a query row's
//     softmax state lives in the 4 lanes r, r+16, r+32, r+48;
//   * updates the online-softmax state (m, l) in the log2 domain (Eqs. 2-5,
//     with exp2 and the scale folded into the scores);
//   * accumulates O~^T += V^T P^T (Eq. 6) with P in bf16; lane (g, r) of an
//     output tile holds dims 4g..4g+3 of query row r.
// V is stored transposed in LDS so that the key order of the P^T operand,
// which is fixed by the S^T output layout, can be matched by the V^T operand.
//
// FACache: a query block with no row in the current block C (inside U)
// streams the key blocks inside U first; in populate mode it then stores its
// state (m, l, O~) in the cache before streaming the blocks that overlap C.
// In resume mode it loads the cached state and streams only the blocks that
// overlap C. Query blocks overlapping C stream everything from scratch.
#include "device.h"
#include "launch.h"

namespace lacache {
namespace {

typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int kD = 128;         // head dimension
constexpr int kBlk = 64;        // query rows and key rows per block
constexpr int kVtStride = 68;   // V^T row stride in bf16 (136 B: conflict-free 8-byte reads)

__device__ __forceinline__ v4f mfma_bf16(bf8 a, bf8 b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ bf8 as_bf8(uint4 v) {
  const u4 w = {v.x, v.y, v.z, v.w};
  return __builtin_bit_cast(bf8, w);
}

template <int kMode>  // 0: populate the cache, 1: resume from it, 2: plain attention
__global__ __launch_bounds__(256) void facache_attention_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    uint16_t* __restrict__ o, float* __restrict__ cm, float* __restrict__ cl, float* __restrict__ co, int64_t N,
    int64_t c0, int64_t c1, float scale_log2) {
  __shared__ __align__(16) uint16_t Ks[kBlk * kD];         // [key][dim], 16-byte chunks xor-swizzled by key
  __shared__ __align__(16) uint16_t Vt[kD * kVtStride];    // [dim][key]

  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int g = lane >> 4, r = lane & 15;
  const int64_t nqb = N / kBlk;
  const int64_t h = blockIdx.x / nqb, qb = blockIdx.x % nqb;
  const int64_t hb = h * N * kD;
  const int64_t row = qb * kBlk + wave * 16 + r;  // this lane's query row

  bf8 qf[4];  // Q^T operands: query row r, dims 32 kk + 8 g ..
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) qf[kk] = as_bf8(*reinterpret_cast<const uint4*>(q + hb + row * kD + 32 * kk + 8 * g));

  const bool q_in_u = !(qb * kBlk < c1 && c0 < (qb + 1) * kBlk);  // no row of this block in C
  float m = -__builtin_inff(), l = 0.0f;
  float ot[8][4];  // O~^T tiles: dims 16 dt + 4 g + i of row r
#pragma unroll
  for (int dt = 0; dt < 8; ++dt)
#pragma unroll
    for (int i = 0; i < 4; ++i) ot[dt][i] = 0.0f;

  // one key/value block: stage it, then Eqs. 2-6 for this wave's 16 rows
  auto process = [&](int64_t kb) {
    __syncthreads();  // every wave is done with the previous block
    const int64_t kr0 = kb * kBlk;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = t + 256 * j;          // 16-byte chunk of the 64 x 128 tile
      const int key = c >> 4, ch = c & 15;
      const uint4 kv = *reinterpret_cast<const uint4*>(k + hb + (kr0 + key) * kD + 8 * ch);
      *reinterpret_cast<uint4*>(Ks + key * kD + 8 * (ch ^ (key & 15))) = kv;
      const uint4 vv = *reinterpret_cast<const uint4*>(v + hb + (kr0 + key) * kD + 8 * ch);
      const uint32_t w[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        Vt[(8 * ch + 2 * e) * kVtStride + key] = static_cast<uint16_t>(w[e] & 0xFFFFu);
        Vt[(8 * ch + 2 * e + 1) * kVtStride + key] = static_cast<uint16_t>(w[e] >> 16);
      }
    }
    __syncthreads();
    // S^T = K Q^T: 4 key tiles of 16, K-dim 128 in 4 steps
    float s[4][4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      const int key = 16 * kt + r;
      v4f acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const bf8 kf = as_bf8(*reinterpret_cast<const uint4*>(Ks + key * kD + 8 * ((4 * kk + g) ^ (key & 15))));
        acc = mfma_bf16(kf, qf[kk], acc);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) s[kt][i] = acc[i] * scale_log2;
    }
    // online softmax of row r (the 4 lanes r + 16 g share it)
    float mx = s[0][0];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) mx = __builtin_fmaxf(mx, s[kt][i]);
    mx = __builtin_fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = __builtin_fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = __builtin_fmaxf(m, mx);                 // Eq. 2
    const float alpha = __builtin_amdgcn_exp2f(m - m_new);      // Eq. 3
    float p[4][4], ps = 0.0f;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        p[kt][i] = __builtin_amdgcn_exp2f(s[kt][i] - m_new);   // Eq. 4
        ps += p[kt][i];
      }
    ps += __shfl_xor(ps, 16, 64);
    ps += __shfl_xor(ps, 32, 64);
    l = alpha * l + ps;                                         // Eq. 5
    m = m_new;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) ot[dt][i] *= alpha;
    // P^T operands: key step ks covers key tiles 2 ks (slots 8g..8g+3) and
    // 2 ks + 1 (slots 8g+4..8g+7), keys 4g..4g+3 of each
    bf8 pb[2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const uint4 pw = make_uint4(pack_bf16x2(p[2 * ks][0], p[2 * ks][1]), pack_bf16x2(p[2 * ks][2], p[2 * ks][3]),
                                  pack_bf16x2(p[2 * ks + 1][0], p[2 * ks + 1][1]),
                                  pack_bf16x2(p[2 * ks + 1][2], p[2 * ks + 1][3]));
      pb[ks] = as_bf8(pw);
    }
    // O~^T += V^T P^T (Eq. 6): V^T operand of dim 16 dt + r, the same key order
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      v4f acc = {ot[dt][0], ot[dt][1], ot[dt][2], ot[dt][3]};
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const uint16_t* vr = Vt + (16 * dt + r) * kVtStride + 32 * ks + 4 * g;
        const uint2 lo = *reinterpret_cast<const uint2*>(vr);
        const uint2 hi = *reinterpret_cast<const uint2*>(vr + 16);
        acc = mfma_bf16(as_bf8(make_uint4(lo.x, lo.y, hi.x, hi.y)), pb[ks], acc);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) ot[dt][i] = acc[i];
    }
  };

  // a block [a, a + 64) overlaps C = [c0, c1) when a < c1 and c0 < a + 64
  auto overlaps_c = [&](int64_t kb) { return kb * kBlk < c1 && c0 < (kb + 1) * kBlk; };
  const int64_t nkb = N / kBlk;
  const int64_t sb = h * N + row;  // state index of this row
  if (kMode == 1 && q_in_u) {
    m = cm[sb];
    l = cl[sb];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      const float4 c4 = *reinterpret_cast<const float4*>(co + sb * kD + 16 * dt + 4 * g);
      ot[dt][0] = c4.x; ot[dt][1] = c4.y; ot[dt][2] = c4.z; ot[dt][3] = c4.w;
    }
  } else {
    for (int64_t kb = 0; kb < nkb; ++kb)
      if (!overlaps_c(kb)) process(kb);  // the key blocks inside U
    if (kMode == 0 && q_in_u) {
      if (g == 0) {
        cm[sb] = m;
        cl[sb] = l;
      }
#pragma unroll
      for (int dt = 0; dt < 8; ++dt)
        *reinterpret_cast<float4*>(co + sb * kD + 16 * dt + 4 * g) = make_float4(ot[dt][0], ot[dt][1], ot[dt][2], ot[dt][3]);
    }
  }
  for (int64_t kb = 0; kb < nkb; ++kb)
    if (overlaps_c(kb)) process(kb);  // the key blocks overlapping C

  const float inv = 1.0f / l;
#pragma unroll
  for (int dt = 0; dt < 8; ++dt)
    *reinterpret_cast<uint2*>(o + hb + row * kD + 16 * dt + 4 * g) =
        make_uint2(pack_bf16x2(ot[dt][0] * inv, ot[dt][1] * inv), pack_bf16x2(ot[dt][2] * inv, ot[dt][3] * inv));
}

}  // namespace

hipError_t launch_facache_attention(hipStream_t st, const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                    uint16_t* o, float* cm, float* cl, float* co, int64_t heads, int64_t N, int64_t c0,
                                    int64_t c1, int mode) {
  const dim3 grid(static_cast<unsigned>(heads * (N / kBlk))), block(256);
  const float scale_log2 = 1.4426950408889634f / 11.313708498984761f;  // log2(e) / sqrt(128)
  if (mode == 0)
    hipLaunchKernelGGL(facache_attention_kernel<0>, grid, block, 0, st, q, k, v, o, cm, cl, co, N, c0, c1, scale_log2);
  else if (mode == 1)
    hipLaunchKernelGGL(facache_attention_kernel<1>, grid, block, 0, st, q, k, v, o, cm, cl, co, N, c0, c1, scale_log2);
  else
    hipLaunchKernelGGL(facache_attention_kernel<2>, grid, block, 0, st, q, k, v, o, cm, cl, co, N, c0, c1, scale_log2);
  return hipGetLastError();
}

}  // namespace lacache
