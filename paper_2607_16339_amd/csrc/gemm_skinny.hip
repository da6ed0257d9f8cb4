// Skinny-M (M <= 64) FP8 GEMMs for block-only calls (Sec. 3.4 linears at a
// decode block's 32 tokens). At this size the FFN is bound by streaming the
// fp8 weights from HBM once, so the kernels are built around that stream:
//
//   * a workgroup owns slabs of 16 weight rows and walks K in blocks of
//     K-groups;
//   * every block of weights and of the M activation rows goes global -> LDS
//     with direct-to-LDS copies into a ring of D slots, D - 1 blocks ahead of
//     the multiply, so D - 1 blocks per CU are always in flight;
//   * the copies are issued with inline asm and waited for with explicit
//     vmcnt counts (loads retire in issue order), so the compiler never adds
//     a wait that would drain the ring;
//   * in LDS, row r's 16-byte chunk c sits at chunk c ^ (r mod 16), so the
//     16 rows of an MFMA operand read hit 16 different bank groups, while each
//     copy instruction still reads 256 contiguous bytes of a row;
//   * each K-group of each 16 x 16 output tile is one 16x16x128 FP8 MFMA,
//     added to the fp32 accumulator times RN32(x_scale * w_scale).
//
// gate/up: 3 waves, each owning the gate rows 16p.. and the matching up rows
//          I + 16p.., all of K, in blocks of two K-groups (256 bytes of each
//          row) shared by the waves; SwiGLU in registers, h stored as fp32.
//          A second kernel quantizes h per 1x128 group (a group's columns
//          come from several workgroups, and stream order is the cheapest
//          way to make all of them visible: device-scope fences inside the
//          kernel cost more than the stream).
// down:    16 output columns per workgroup, its 4 waves take a quarter of K
//          each, one K-group per block, in private rings; the partials are
//          added in LDS in wave order.
#include "device.h"
#include "launch.h"

namespace lacache {
namespace {

constexpr int kRowBytes = 256;  // one block: two K-groups of a row
constexpr int kMaxNkb = 64;     // K-groups per workgroup (scales staged in LDS)
constexpr int kGuWaves = 3;     // gate/up: (gate, up) slab pairs per workgroup
#ifndef LACACHE_SKINNY_ROT
#define LACACHE_SKINNY_ROT 1
#endif
// Workgroups start their walk over K at different blocks (and wrap), so that
// at any moment the chip's copies spread over all memory channels instead of
// all reading the same K offset of rows that are a multiple of 4 KB apart.
constexpr bool kRotateK = LACACHE_SKINNY_ROT != 0;

// MFMA operand from a ring slot laid out [row][256 B] with the chunk xor:
// lane (q, lr) takes row base + lr, logical chunks kk*8 + q and kk*8 + 4 + q.
__device__ __forceinline__ v8i ring_frag(const uint8_t* slab, int lr, int q, int kk) {
  const uint8_t* row = slab + lr * kRowBytes;
  const uint4 lo = *reinterpret_cast<const uint4*>(row + (((kk * 8 + q) ^ lr) << 4));
  const uint4 hi = *reinterpret_cast<const uint4*>(row + (((kk * 8 + 4 + q) ^ lr) << 4));
  v8i f;
  f[0] = static_cast<int>(lo.x); f[1] = static_cast<int>(lo.y); f[2] = static_cast<int>(lo.z); f[3] = static_cast<int>(lo.w);
  f[4] = static_cast<int>(hi.x); f[5] = static_cast<int>(hi.y); f[6] = static_cast<int>(hi.z); f[7] = static_cast<int>(hi.w);
  return f;
}

template <int MT>
struct Cfg {
  static constexpr int NW = kGuWaves;
  static constexpr int NS = 2;                           // gate and up slab
  static constexpr int RA = MT * 16;                     // activation rows in a slot (padded)
  static constexpr int kA = RA * kRowBytes;              // activation bytes per slot
  static constexpr int kW = NW * NS * 16 * kRowBytes;    // weight bytes per slot
  static constexpr int kSlot = kA + kW;
  static constexpr int AI = RA / 4;                      // 1 KB copies of activations per block
  static constexpr int AIW = (AI + NW - 1) / NW;         // ... per wave (the last may repeat one)
  static constexpr int WI = NS * 4;                      // 1 KB copies of weights per wave per block
  static constexpr int PER = AIW + WI;                   // copies per wave per block
};

template <int MT, int D>
__global__ __launch_bounds__(kGuWaves * 64) void skinny_gateup_kernel(
    const uint8_t* __restrict__ aq, const float* __restrict__ as,  // activations [M x K], scales [K/128 x M]
    const uint8_t* __restrict__ wq, const float* __restrict__ ws,  // weights [2I x K], scales [2I/128 x K/128]
    float* __restrict__ h_tap, float* __restrict__ hbuf, int64_t M, int64_t K, int64_t I) {
  using C = Cfg<MT>;
  constexpr int NW = C::NW, NS = C::NS, RA = C::RA;
  __shared__ __align__(16) uint8_t ring[D * C::kSlot];
  __shared__ __align__(16) float sXs[kMaxNkb * RA];
  __shared__ float sWs[NW * NS * kMaxNkb];

  const int t = threadIdx.x, lane = t & 63;
  const int wave = wave_uniform(t >> 6);
  const int q = lane >> 4, lr = lane & 15;
  const int64_t KB = K / 128;

  // ---- work of this wavefront: h columns 16 pair .. 16 pair + 15
  const int64_t pair = static_cast<int64_t>(blockIdx.x) * NW + wave;
  const bool active = pair < I / 16;
  const int64_t p0 = active ? pair : 0;
  const int64_t slab_row[NS] = {16 * p0, I + 16 * p0};  // gate rows, up rows
  const int64_t kb0 = 0, kb1 = KB;
  const int nkb = static_cast<int>(kb1 - kb0);
  const int NB = (nkb + 1) / 2;
  // block visited at step b (steps past the end repeat the last visited block)
  const int rot = kRotateK ? static_cast<int>((blockIdx.x >> 3) % static_cast<unsigned>(NB)) : 0;
  auto block_at = [&](int b) {
    int bb = (b < NB ? b : NB - 1) + rot;
    return bb >= NB ? bb - NB : bb;
  };

  // ---- copy plan. Copy instruction u of a 16-row slab covers rows 4u..4u+3;
  // lane l fills slot chunk l%16 of row 4u + l/16 with logical chunk
  // (l%16) ^ row, i.e. K-group half (chunk / 8) and 16-byte piece chunk % 8.
  const int crow = lane >> 4;  // row within the copy's 4 rows
  const int pch = lane & 15;   // physical chunk in LDS
  // activations: wave copies instructions a = wave + NW j (clamped: repeats are identical writes)
  int64_t a_off[C::AIW];
  int a_dst[C::AIW];
  int a_half[C::AIW];
#pragma unroll
  for (int j = 0; j < C::AIW; ++j) {
    int a = wave + NW * j;
    if (a > C::AI - 1) a = C::AI - 1;
    const int row = 4 * a + crow;                        // slot row
    const int lch = pch ^ (row & 15);
    const int64_t gr = row < M ? row : M - 1;
    a_off[j] = gr * K + (lch & 7) * 16;
    a_half[j] = lch >> 3;
    a_dst[j] = a * 1024;
  }
  int64_t w_off[C::WI];
  int w_half[C::WI];
  int w_dst[C::WI];
#pragma unroll
  for (int n = 0; n < NS; ++n)
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int row = 4 * u + crow;
      const int lch = pch ^ row;
      w_off[n * 4 + u] = (slab_row[n] + row) * K + (lch & 7) * 16;
      w_half[n * 4 + u] = lch >> 3;
      w_dst[n * 4 + u] = C::kA + ((wave * NS + n) * 16 * kRowBytes) + u * 1024;
    }

  // Issues the copies of step b (the repeats past the end rewrite the last
  // block's own data into an idle slot).
  auto issue = [&](int b, int slot) {
    const int bb = block_at(b);
    const uint32_t base = lds_u32(ring + slot * C::kSlot);
#pragma unroll
    for (int j = 0; j < C::AIW; ++j) {
      int64_t kg = kb0 + 2 * bb + a_half[j];
      if (kg >= kb1) kg = kb1 - 1;
      dma16(aq + a_off[j] + kg * 128, wave_uniform(static_cast<int>(base) + a_dst[j]));
    }
#pragma unroll
    for (int i = 0; i < C::WI; ++i) {
      int64_t kg = kb0 + 2 * bb + w_half[i];
      if (kg >= kb1) kg = kb1 - 1;
      dma16(wq + w_off[i] + kg * 128, wave_uniform(static_cast<int>(base) + w_dst[i]));
    }
  };

  float acc[MT][NS][4];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int n = 0; n < NS; ++n)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[i][n][r] = 0.0f;

  // ---- the stream: D - 1 blocks ahead
#pragma unroll
  for (int b = 0; b < D - 1; ++b) issue(b, b);

  // ---- scales for the whole K range, staged in LDS. Loaded after the first
  // copies are on their way and all issued before any is stored, so the
  // staging costs one memory latency, overlapped with the copies'.
  {
    constexpr int XPT = (kMaxNkb * RA + NW * 64 - 1) / (NW * 64);
    constexpr int WPT = (NW * NS * kMaxNkb + NW * 64 - 1) / (NW * 64);
    float xv[XPT], wv[WPT];
#pragma unroll
    for (int j = 0; j < XPT; ++j) {
      const int i = t + j * NW * 64;
      const int kb = i / RA, m = i % RA;
      xv[j] = (i < nkb * RA && m < M) ? as[(kb0 + kb) * M + m] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < WPT; ++j) {
      const int i = t + j * NW * 64;
      const int w = i / (NS * nkb), n = (i / nkb) % NS, kb = i % nkb;
      const int64_t p = static_cast<int64_t>(blockIdx.x) * NW + w;
      const bool ok = i < NW * NS * nkb && p < I / 16;
      const int64_t r = n == 0 ? 16 * p : I + 16 * p;
      wv[j] = ok ? ws[(r / 128) * KB + kb0 + kb] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < XPT; ++j) {
      const int i = t + j * NW * 64;
      if (i < nkb * RA) sXs[i] = xv[j];
    }
#pragma unroll
    for (int j = 0; j < WPT; ++j) {
      const int i = t + j * NW * 64;
      if (i < NW * NS * nkb) sWs[i] = wv[j];
    }
  }
  __syncthreads();

  for (int b = 0; b < NB; ++b) {
    wait_vm_lds<(D - 2) * C::PER>();  // block b has landed (later blocks may still fly)
    bar();                            // ... for every wave; and slot (b-1) % D is free
    issue(b + D - 1, (b + D - 1) % D);
    const uint8_t* slot = ring + (b % D) * C::kSlot;
    const int bk = block_at(b);
    // the block's two K-groups (the second may lie past K when K/128 is odd):
    // all operands first, then every MFMA back to back (they are independent),
    // then the scale FMAs in K-group order, so the block's latency is one LDS
    // round trip plus the MFMA issue time rather than a chain of MFMA results
    const int nk = 2 * bk + 1 < nkb ? 2 : 1;
    v8i af[2][MT], bf[2][NS];
    float xa[2][MT][4], wv[2][NS];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int kb = 2 * bk + (kk < nk ? kk : 0);
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        af[kk][i] = ring_frag(slot + i * 16 * kRowBytes, lr, q, kk);
        const float4 xv = *reinterpret_cast<const float4*>(sXs + kb * RA + 16 * i + 4 * q);
        xa[kk][i][0] = xv.x; xa[kk][i][1] = xv.y; xa[kk][i][2] = xv.z; xa[kk][i][3] = xv.w;
      }
#pragma unroll
      for (int n = 0; n < NS; ++n) {
        bf[kk][n] = ring_frag(slot + C::kA + (wave * NS + n) * 16 * kRowBytes, lr, q, kk);
        wv[kk][n] = sWs[(wave * NS + n) * nkb + kb];
      }
    }
    v4f p[2][NS][MT];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int n = 0; n < NS; ++n)
#pragma unroll
        for (int i = 0; i < MT; ++i) {
          const v4f zero = {0.0f, 0.0f, 0.0f, 0.0f};
          p[kk][n][i] = mfma_fp8_16x16x128(af[kk][i], bf[kk][n], zero);
        }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      if (kk >= nk) break;
#pragma unroll
      for (int n = 0; n < NS; ++n)
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            acc[i][n][r] = __builtin_fmaf(p[kk][n][i][r], xa[kk][i][r] * wv[kk][n], acc[i][n][r]);
    }
  }
  wait_vm<0>();  // drain the trailing repeat copies

  if (!active) return;
  // ---- SwiGLU, h -> fp32 [M x I]
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t row = 16 * i + 4 * q + r;
      if (row < M) {
        const float h = swiglu_fast(acc[i][0][r], acc[i][1][r]);
        hbuf[row * I + 16 * pair + lr] = h;
        if (h_tap != nullptr) h_tap[row * I + 16 * pair + lr] = h;
      }
    }
}

// ---------------------------------------------------------------------------
// down, K split inside the workgroup: 16 output columns per workgroup, its 4
// wavefronts take a quarter of K each. A wavefront streams its own K range
// (the 16 weight rows and the M activation rows, one K-group per slot) into
// a private LDS ring, so the streaming needs no workgroup barrier; the four
// fp32 partials meet in LDS at the end and are added in wavefront order.
// ---------------------------------------------------------------------------
constexpr int kDnSplit = 4;       // wavefronts (K quarters) per workgroup
constexpr int kDnMaxNkbW = 32;    // K-groups per wavefront (scales staged in LDS)

template <int MT>
struct DnCfg {
  static constexpr int RA = MT * 16;        // activation rows in a slot (padded)
  static constexpr int kA = RA * 128;       // activation bytes per slot
  static constexpr int kSlot = kA + 16 * 128;
  static constexpr int AI = RA / 8;         // 1 KB copies of activations per slot
  static constexpr int PER = AI + 2;        // copies per slot (activations + 2 of weights)
  static constexpr int D = MT == 1 ? 8 : (MT == 2 ? 5 : (MT == 3 ? 4 : 3));  // ring depth that fits the LDS
};

// MFMA operand from a slot laid out [row][128 B], physical chunk = logical
// chunk ^ (row & 7): lane (q, lr) takes row lr, logical chunks q and 4 + q.
__device__ __forceinline__ v8i slot_frag(const uint8_t* rows, int lr, int q) {
  const uint8_t* row = rows + lr * 128;
  const uint4 lo = *reinterpret_cast<const uint4*>(row + ((q ^ (lr & 7)) << 4));
  const uint4 hi = *reinterpret_cast<const uint4*>(row + (((4 + q) ^ (lr & 7)) << 4));
  v8i f;
  f[0] = static_cast<int>(lo.x); f[1] = static_cast<int>(lo.y); f[2] = static_cast<int>(lo.z); f[3] = static_cast<int>(lo.w);
  f[4] = static_cast<int>(hi.x); f[5] = static_cast<int>(hi.y); f[6] = static_cast<int>(hi.z); f[7] = static_cast<int>(hi.w);
  return f;
}

template <int MT>
__global__ __launch_bounds__(kDnSplit * 64) void skinny_down_kernel(
    const uint8_t* __restrict__ aq, const float* __restrict__ as,  // h codes [M x K], scales [K/128 x M]
    const uint8_t* __restrict__ wq, const float* __restrict__ ws,  // W_down codes [N x K], scales [N/128 x K/128]
    uint16_t* __restrict__ out, float* __restrict__ out_tap, int64_t M, int64_t K, int64_t N) {
  using C = DnCfg<MT>;
  constexpr int D = C::D, RA = C::RA;
  __shared__ __align__(16) uint8_t ring[kDnSplit][D * C::kSlot];
  __shared__ __align__(16) float sXs[kDnSplit][kDnMaxNkbW * RA];
  __shared__ float sWs[kDnSplit][kDnMaxNkbW];

  const int t = threadIdx.x, lane = t & 63;
  const int wave = wave_uniform(t >> 6);
  const int q = lane >> 4, lr = lane & 15;
  const int64_t KB = K / 128;
  const int64_t n0 = static_cast<int64_t>(blockIdx.x) * 16;
  const int64_t kb0 = wave * KB / kDnSplit, kb1 = (wave + 1) * KB / kDnSplit;
  const int nkb = static_cast<int>(kb1 - kb0);  // 0 when K has fewer groups than wavefronts
  uint8_t* my = ring[wave];

  // copy plan: instruction u fills slot rows 8u..8u+7; lane l fills row
  // 8u + l/8, physical chunk l%8, i.e. logical chunk (l%8) ^ (row & 7)
  const int crow = lane >> 3, pch = lane & 7;
  int64_t a_off[C::AI];
#pragma unroll
  for (int u = 0; u < C::AI; ++u) {
    const int row = 8 * u + crow;
    const int64_t gr = row < M ? row : M - 1;
    a_off[u] = gr * K + ((pch ^ (row & 7)) << 4);
  }
  int64_t w_off[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int row = 8 * u + crow;
    w_off[u] = (n0 + row) * K + ((pch ^ (row & 7)) << 4);
  }
  auto issue = [&](int b, int slot) {
    const int64_t kg = kb0 + (b < nkb ? b : nkb - 1);  // past the end: the last K-group again
    const uint32_t base = lds_u32(my + slot * C::kSlot);
#pragma unroll
    for (int u = 0; u < C::AI; ++u) dma16(aq + a_off[u] + kg * 128, wave_uniform(static_cast<int>(base) + u * 1024));
#pragma unroll
    for (int u = 0; u < 2; ++u)
      dma16(wq + w_off[u] + kg * 128, wave_uniform(static_cast<int>(base) + C::kA + u * 1024));
  };
  if (nkb > 0) {
#pragma unroll
    for (int b = 0; b < D - 1; ++b) issue(b, b);
  }

  // ---- this wavefront's scales, staged in LDS (loaded after the first copies)
  {
    constexpr int XPT = kDnMaxNkbW * RA / 64;
    float xv[XPT];
#pragma unroll
    for (int j = 0; j < XPT; ++j) {
      const int i = lane + 64 * j, kb = i / RA, m = i % RA;
      xv[j] = (i < nkb * RA && m < M) ? as[(kb0 + kb) * M + m] : 0.0f;
    }
    const float wv = lane < nkb ? ws[(n0 / 128) * KB + kb0 + lane] : 0.0f;
#pragma unroll
    for (int j = 0; j < XPT; ++j) {
      const int i = lane + 64 * j;
      if (i < nkb * RA) sXs[wave][i] = xv[j];
    }
    if (lane < nkb) sWs[wave][lane] = wv;
  }

  float acc[MT][4];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[i][r] = 0.0f;
  for (int b = 0; b < nkb; ++b) {
    wait_vm_lds<(D - 2) * C::PER>();  // K-group b has landed; slot (b-1) % D is read
    issue(b + D - 1, (b + D - 1) % D);
    const uint8_t* slot = my + (b % D) * C::kSlot;
    const v8i bf = slot_frag(slot + C::kA, lr, q);
    const float w = sWs[wave][b];
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const v8i af = slot_frag(slot + i * 16 * 128, lr, q);
      const float4 x4 = *reinterpret_cast<const float4*>(&sXs[wave][b * RA + 16 * i + 4 * q]);
      const v4f zero = {0.0f, 0.0f, 0.0f, 0.0f};
      const v4f p = mfma_fp8_16x16x128(af, bf, zero);
      acc[i][0] = __builtin_fmaf(p[0], x4.x * w, acc[i][0]);
      acc[i][1] = __builtin_fmaf(p[1], x4.y * w, acc[i][1]);
      acc[i][2] = __builtin_fmaf(p[2], x4.z * w, acc[i][2]);
      acc[i][3] = __builtin_fmaf(p[3], x4.w * w, acc[i][3]);
    }
  }
  wait_vm<0>();  // the trailing repeat copies
  __syncthreads();  // every ring is idle: reuse the space for the partials

  // ---- partials [wave][RA][16] -> sum in wavefront order -> bf16
  float* red = reinterpret_cast<float*>(&ring[0][0]);
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) red[(wave * RA + 16 * i + 4 * q + r) * 16 + lr] = acc[i][r];
  __syncthreads();
  for (int e = t; e < M * 16; e += kDnSplit * 64) {
    const int row = e >> 4, col = e & 15;
    float sum = red[row * 16 + col];
#pragma unroll
    for (int w = 1; w < kDnSplit; ++w) sum += red[(w * RA + row) * 16 + col];
    out[row * N + n0 + col] = static_cast<uint16_t>(f32_to_bf16(sum));
    if (out_tap != nullptr) out_tap[row * N + n0 + col] = sum;
  }
}

// h [M x I] fp32 -> 1x128 e4m3 groups (Eq. 7): codes [M x I], scales
// [I/128 x M]. 16 lanes per group, 8 values per lane.
__global__ __launch_bounds__(256) void skinny_hquant_kernel(const float* __restrict__ h, uint8_t* __restrict__ hq,
                                                            float* __restrict__ hs, int64_t M, int64_t I) {
  const int64_t gi = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) >> 4;  // group index, row-major
  const int part = threadIdx.x & 15;
  const int64_t G = I / 128;
  const bool ok = gi < M * G;
  const int64_t row = ok ? gi / G : 0, g = ok ? gi % G : 0;
  float v[8];
  const float4* src = reinterpret_cast<const float4*>(h + row * I + g * 128 + part * 8);
  const float4 a = src[0], b = src[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  float m = 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) m = __builtin_fmaxf(m, __builtin_fabsf(v[e]));
  m = max_xor<16>(m);
  const float s = m / kE4M3Max;
  uint32_t lo = 0u, hi = 0u;
  if (s != 0.0f && !(scale_is_fast(s) && enc8_div_fast(v, fast_rcp(s), lo, hi))) {
    lo = enc4_e4m3(qdiv(v[0], s), qdiv(v[1], s), qdiv(v[2], s), qdiv(v[3], s));
    hi = enc4_e4m3(qdiv(v[4], s), qdiv(v[5], s), qdiv(v[6], s), qdiv(v[7], s));
  }
  if (!ok) return;
  *reinterpret_cast<uint2*>(hq + row * I + g * 128 + part * 8) = make_uint2(lo, hi);
  if (part == 0) hs[g * M + row] = s;
}

// Ring depth per M-tile count: the deepest ring that fits the LDS.
template <int MT>
constexpr int gateup_ring_depth() {
  return MT <= 2 ? 4 : 3;
}

template <int MT>
hipError_t launch_gateup(hipStream_t st, const uint8_t* aq, const float* as, const uint8_t* wq, const float* ws,
                         float* h_tap, float* hbuf, int64_t M, int64_t K, int64_t I, unsigned grid) {
  constexpr int D = gateup_ring_depth<MT>();
  hipLaunchKernelGGL((skinny_gateup_kernel<MT, D>), dim3(grid), dim3(kGuWaves * 64), 0, st, aq, as, wq, ws, h_tap,
                     hbuf, M, K, I);
  return hipGetLastError();
}

}  // namespace

bool skinny_supported(int64_t M, int64_t H, int64_t I) {
  return M >= 1 && M <= kSkinnyMaxM && H / 128 <= kMaxNkb && I / 128 <= kDnSplit * kDnMaxNkbW;
}

size_t skinny_gateup_ws_bytes(int64_t M, int64_t I) {
  const size_t h = static_cast<size_t>(M) * static_cast<size_t>(I) * sizeof(float);
  return ((h + 255) / 256) * 256;
}

// ws_buf: an fp32 buffer of skinny_gateup_ws_bytes() for h.
hipError_t launch_gateup_skinny(hipStream_t st, const uint8_t* xq, const float* xs, const uint8_t* wq,
                                const float* ws, uint8_t* hq, float* hs, float* h_tap, int64_t M, int64_t H,
                                int64_t I, void* ws_buf) {
  float* hbuf = static_cast<float*>(ws_buf);
  const unsigned grid = static_cast<unsigned>((I / 16 + kGuWaves - 1) / kGuWaves);
  const int mt = static_cast<int>((M + 15) / 16);
  hipError_t e;
#define GU(MT_) launch_gateup<MT_>(st, xq, xs, wq, ws, h_tap, hbuf, M, H, I, grid)
  if (mt <= 1) e = GU(1);
  else if (mt == 2) e = GU(2);
  else if (mt == 3) e = GU(3);
  else e = GU(4);
#undef GU
  if (e != hipSuccess) return e;
  const int64_t groups = M * (I / 128);
  hipLaunchKernelGGL(skinny_hquant_kernel, dim3(static_cast<unsigned>((groups + 15) / 16)), dim3(256), 0, st, hbuf, hq,
                     hs, M, I);
  return hipGetLastError();
}

hipError_t launch_quant_groups_f32(hipStream_t st, const float* v, uint8_t* codes, float* scales, int64_t M, int64_t K) {
  const int64_t groups = M * (K / 128);
  hipLaunchKernelGGL(skinny_hquant_kernel, dim3(static_cast<unsigned>((groups + 15) / 16)), dim3(256), 0, st, v, codes,
                     scales, M, K);
  return hipGetLastError();
}

hipError_t launch_down_skinny(hipStream_t st, const uint8_t* hq, const float* hs, const uint8_t* wq, const float* ws,
                              uint16_t* out, float* out_tap, int64_t M, int64_t H, int64_t I) {
  const dim3 grid(static_cast<unsigned>(H / 16)), block(kDnSplit * 64);
  const int mt = static_cast<int>((M + 15) / 16);
#define DN(MT_) hipLaunchKernelGGL(skinny_down_kernel<MT_>, grid, block, 0, st, hq, hs, wq, ws, out, out_tap, M, I, H)
  if (mt <= 1) DN(1);
  else if (mt == 2) DN(2);
  else if (mt == 3) DN(3);
  else DN(4);
#undef DN
  return hipGetLastError();
}

}  // namespace lacache
