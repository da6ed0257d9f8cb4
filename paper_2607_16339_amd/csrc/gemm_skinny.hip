// Skinny-M (M <= 64) FP8 GEMMs for block-only calls (Sec. 3.4 linears at a
// decode block's 32 tokens). At this size the FFN is bound by streaming the
// fp8 weights from HBM once, so the kernels are built around that stream.
// Each K-group of each 16 x 16 output tile is one 16x16x128 FP8 MFMA, added
// to the fp32 accumulator times RN32(x_scale * w_scale), and the K range of
// an output tile is split over several wavefronts of a workgroup, whose fp32
// partials are added in LDS in a fixed order.
//
// gate/up: a workgroup owns 3 (gate, up) slab pairs x 4 K parts (one
//          wavefront each), or at 33..64 rows 6 pairs x 2 parts. The
//          activation codes are copied into LDS once per workgroup (up to
//          32 rows over all of K; 33..64 rows over one half of K, the halves
//          in two workgroups); the weights go global -> VGPRs with non-temporal
//          16-byte loads straight into the MFMA operand layout, a ring of
//          K-groups per wavefront in straight-line code (the compiler waits
//          for one K-group's registers at a time). The weight tile layout
//          (wtile_off) makes each load read 1 KB contiguous; on a row-major
//          matrix the same operand layout reads 16 rows x 64 bytes per load,
//          which streams about 25 % slower on gfx950. SwiGLU after the
//          partials are added; h stored as fp32 (33..64 rows: the gate and
//          up sums of each K half, added by the second kernel before
//          SwiGLU). A second kernel quantizes h per 1x128 group (a group's columns come from several workgroups,
//          and stream order is the cheapest way to make all of them visible:
//          device-scope fences inside the kernel cost more than the stream).
// down:    16 output columns per workgroup, 8 K parts (up to 32 rows and 96
//          K-groups) or 4, direct-to-LDS copies of both operands (see the
//          kernel).
#include "device.h"
#include "launch.h"

namespace lacache {
namespace {

#ifndef LACACHE_SKINNY_ROT
#define LACACHE_SKINNY_ROT 1
#endif
// Workgroups walk their K parts from different starting K-groups (and
// wrap), so that at any moment the chip's loads spread over more memory
// pages instead of all reading one K offset.
constexpr bool kRotateK = LACACHE_SKINNY_ROT != 0;

// On gfx950 register loads of 1 KB runs stream the weights about 15 % faster
// than direct-to-LDS copies, and a CU pulls about twice as many bytes per
// second from L2 into registers as into LDS, so the activation operand
// (re-read by every workgroup) does not slow the weight stream either.
typedef unsigned int u4v __attribute__((ext_vector_type(4)));
// K-groups in flight per wavefront (the ring depth DR): gate/up runs 12
// wavefronts per CU (at most 168 VGPRs each) and keeps 2, i.e. 96 KB per CU.
constexpr int kVuDR = 2;

__device__ __forceinline__ u4v ld_nt(const uint8_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u4v*>(p));
}
__device__ __forceinline__ v8i cat_frag(u4v lo, u4v hi) {
  v8i f;
  f[0] = static_cast<int>(lo[0]); f[1] = static_cast<int>(lo[1]); f[2] = static_cast<int>(lo[2]); f[3] = static_cast<int>(lo[3]);
  f[4] = static_cast<int>(hi[0]); f[5] = static_cast<int>(hi[1]); f[6] = static_cast<int>(hi[2]); f[7] = static_cast<int>(hi[3]);
  return f;
}

// gate/up: a workgroup owns PAIRS (gate, up) slab pairs; each pair's K
// range is split into KQ parts, one wavefront each (PAIRS KQ = 12). The workgroup first
// loads the M activation rows (codes) of its K range into LDS, rows padded by
// 16 bytes so that the 16 rows of an operand read fall on 16 different bank
// groups; then every wavefront streams its 32 weight rows over its K part.
// The KQ fp32 partials meet in LDS and are added in part order.
// NH = 1: the workgroup covers all of K and applies SwiGLU (h to hbuf).
// NH = 2 (33..64 rows, whose codes over all of K do not fit the LDS): the
// workgroups of blockIdx.y = 0, 1 cover the two halves of K and store their
// gate and up sums to part[y] [M][2I]; the h-quantization kernel adds the two
// halves in that order and applies SwiGLU.
constexpr int kVuWaves = 12;
#ifndef LACACHE_NH2_PAIRS
#define LACACHE_NH2_PAIRS 6
#endif
constexpr int kNh2Pairs = LACACHE_NH2_PAIRS;  // slab pairs per workgroup at 33..64 rows
constexpr int kVuXBytes = 64 * (2048 + 16);  // activation rows x (K range + 16) bytes, at most
constexpr int kVuMaxNkb = 64;                 // K-groups of the whole K
constexpr int kVuScales = 2048;               // activation scales of a workgroup's K range, at most

template <int MT, int DR, int NH, int PAIRS, int KQ>
__global__ __launch_bounds__(kVuWaves * 64) void skinny_gateup_kernel(
    const uint8_t* __restrict__ aq, const float* __restrict__ as,  // activations [M x K], scales [K/128 x M]
    const uint8_t* __restrict__ wq, const float* __restrict__ ws,  // weights [2I x K], scales [2I/128 x K/128]
    float* __restrict__ h_tap, float* __restrict__ hbuf, int64_t M, int64_t K, int64_t I) {
  constexpr int R = MT * 16;  // activation rows (padded)
  static_assert(NH == 1 || NH == 2, "K pieces");
  static_assert(PAIRS * KQ == kVuWaves, "one wavefront per (pair, part)");
  constexpr int kMaxNkw = kVuMaxNkb / KQ;  // K-groups of one part
  __shared__ __align__(16) uint8_t sX[kVuXBytes];  // codes [R][Kw + 16]; later the partials
  __shared__ __align__(16) float sXs[kVuScales];   // activation scales [Kw/128][R]
  __shared__ float sWs[kVuWaves][2][kMaxNkw];    // each wavefront's (gate, up) block scales

  const int t = threadIdx.x, lane = t & 63;
  const int wave = wave_uniform(t >> 6);
  const int q = lane >> 4, lr = lane & 15;
  const int pw = wave % PAIRS, kq = wave / PAIRS;
  const int KB = static_cast<int>(K / 128);
  // this workgroup's K range [kbw, kbw + KBW) and its parts
  const int kh = NH == 1 ? 0 : static_cast<int>(blockIdx.y);
  const int kbw = kh * KB / NH, KBW = (kh + 1) * KB / NH - kbw;
  const int64_t Kw = static_cast<int64_t>(KBW) * 128;
  const int64_t stride = Kw + 16;
  const int64_t npair = I / 16;
  const int64_t pair = static_cast<int64_t>(blockIdx.x) * PAIRS + pw;
  const int64_t p0 = pair < npair ? pair : npair - 1;  // past the end: a valid pair, never stored
  const int kb0 = kbw + kq * KBW / KQ, kb1 = kbw + (kq + 1) * KBW / KQ;
  const int nkw = kb1 - kb0;

  // ---- 1. activation codes -> registers: 16-byte chunk c = t + 768 j of
  // the M rows' K range (row c / cpr, chunk c % cpr) goes to LDS byte
  // 16 (c + c / cpr) (rows padded by one chunk). Register loads take these
  // L2-resident bytes at about twice the per-CU rate of direct-to-LDS
  // copies, and this copy is the kernel's start-up. Rows M..R-1 of the LDS
  // stay unwritten: they only feed output rows that are never stored (an
  // MFMA output row depends on its own activation row alone).
  constexpr int XCH = (kVuXBytes / 16 + kVuWaves * 64 - 1) / (kVuWaves * 64);  // chunks per thread, at most
  const int cpr = KBW * 8;  // chunks per row
  const int nch = static_cast<int>(M) * cpr;
  // c / cpr for c < 2^14: the float estimate is off by at most one
  const float rcpr = 1.0f / static_cast<float>(cpr > 0 ? cpr : 1);
  auto row_of = [&](int c) {
    int r = static_cast<int>(static_cast<float>(c) * rcpr);
    r -= r * cpr > c ? 1 : 0;
    r += (r + 1) * cpr <= c ? 1 : 0;
    return r;
  };
  u4v xc[XCH];
#pragma unroll
  for (int j = 0; j < XCH; ++j) {
    const int c = t + j * kVuWaves * 64;
    if (c < nch) {
      // NH = 1: the rows are contiguous; NH = 2: row r's range starts at r K + kbw 128
      const uint32_t off = NH == 1 ? 16u * static_cast<uint32_t>(c)
                                   : static_cast<uint32_t>(row_of(c)) * static_cast<uint32_t>(K) +
                                         static_cast<uint32_t>(kbw) * 128u +
                                         16u * static_cast<uint32_t>(c - row_of(c) * cpr);
      xc[j] = *reinterpret_cast<const u4v*>(aq + off);
    }
  }
  // ---- 2. scales into registers
  constexpr int XPT = (kVuScales + kVuWaves * 64 - 1) / (kVuWaves * 64);
  float xv[XPT];
#pragma unroll
  for (int j = 0; j < XPT; ++j) {
    const int i = t + j * kVuWaves * 64;
    const int kb = i / R, m = i % R;
    xv[j] = (kb < KBW && m < M) ? as[static_cast<int64_t>(kbw + kb) * M + m] : 0.0f;
  }
  const int64_t wrow[2] = {16 * p0, I + 16 * p0};
  const int sn = lane >> 5, sj = lane & 31;
  const float wv = sj < nkw ? ws[(wrow[sn] / 128) * KB + kb0 + sj] : 0.0f;

  // ---- 3. the weight ring: K-group j of this wavefront's part in slot j % DR
  // (lane (q, lr) takes row lr, columns 16q.. and 64 + 16q.. of the K-group:
  // bytes 64 lr + 16 q of the two 1 KB halves of the slab's tile)
  const uint8_t* wg = wq + wtile_off(wrow[0] + lr, 16 * q, K);
  const uint8_t* wu = wq + wtile_off(wrow[1] + lr, 16 * q, K);
  // K-group of step j: the part is walked from a workgroup-dependent start
  // (and wraps); steps past the end repeat the last K-group walked
  const int rot = (kRotateK && nkw > 0) ? static_cast<int>(blockIdx.x % static_cast<unsigned>(nkw)) : 0;
  auto kg_at = [&](int j) {
    if (nkw <= 0) return kb0 < KB ? kb0 : KB - 1;
    const int jj = (j < nkw ? j : nkw - 1) + rot;
    return kb0 + (jj >= nkw ? jj - nkw : jj);
  };
  u4v wr[DR][4];  // gate lo, gate hi, up lo, up hi
  auto issue = [&](int j, int slot) {
    const int64_t o = static_cast<int64_t>(kg_at(j)) * 2048;
    wr[slot][0] = ld_nt(wg + o);
    wr[slot][1] = ld_nt(wg + o + 1024);
    wr[slot][2] = ld_nt(wu + o);
    wr[slot][3] = ld_nt(wu + o + 1024);
  };
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int u = 0; u < DR; ++u) issue(u, u);
  __builtin_amdgcn_sched_barrier(0);

#pragma unroll
  for (int j = 0; j < XCH; ++j) {
    const int c = t + j * kVuWaves * 64;
    if (c < nch) *reinterpret_cast<u4v*>(sX + 16 * (c + row_of(c))) = xc[j];
  }
#pragma unroll
  for (int j = 0; j < XPT; ++j) {
    const int i = t + j * kVuWaves * 64;
    if (i < KBW * R) sXs[i] = xv[j];
  }
  if (sj < kMaxNkw) sWs[wave][sn][sj] = wv;
  __syncthreads();  // the activation codes and the scales are in LDS

  float acc[MT][2][4];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int n = 0; n < 2; ++n)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[i][n][r] = 0.0f;

  // Rounds of DR K-groups, straight-line code (the compiler then waits for
  // each slot's loads alone): step j multiplies slot j % DR and refills it
  // with K-group j + DR; the last round refills nothing. Steps past the
  // part's end re-multiply its last K-group with a zero scale.
  auto step = [&](int j, int u) {
    const bool live = j < nkw;
    const int kg = kg_at(j);
    const int kl = kg - kbw;  // K-group within the workgroup's range
    const float w0 = live ? sWs[wave][0][kg - kb0] : 0.0f, w1 = live ? sWs[wave][1][kg - kb0] : 0.0f;
    const v8i bg = cat_frag(wr[u][0], wr[u][1]), bu = cat_frag(wr[u][2], wr[u][3]);
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const uint8_t* xr = sX + (16 * i + lr) * stride + kl * 128 + 16 * q;
      const v8i af = cat_frag(*reinterpret_cast<const u4v*>(xr), *reinterpret_cast<const u4v*>(xr + 64));
      const float4 x4 = *reinterpret_cast<const float4*>(sXs + kl * R + 16 * i + 4 * q);
      const v4f zero = {0.0f, 0.0f, 0.0f, 0.0f};
      const v4f pg = mfma_fp8_16x16x128(af, bg, zero);
      const v4f pu = mfma_fp8_16x16x128(af, bu, zero);
      const float xa[4] = {x4.x, x4.y, x4.z, x4.w};
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        acc[i][0][r] = __builtin_fmaf(pg[r], xa[r] * w0, acc[i][0][r]);
        acc[i][1][r] = __builtin_fmaf(pu[r], xa[r] * w1, acc[i][1][r]);
      }
    }
  };
  const int NR = (nkw + DR - 1) / DR;
  for (int rd = 0; rd + 1 < NR; ++rd) {
#pragma unroll
    for (int u = 0; u < DR; ++u) {
      step(rd * DR + u, u);
      issue(rd * DR + u + DR, u);
    }
  }
  if (NR > 0) {
#pragma unroll
    for (int u = 0; u < DR; ++u) step((NR - 1) * DR + u, u);
  }

  // ---- 4. partials [kq][pair][R][32] in LDS, added in part order; then
  // SwiGLU (NH = 1) or the gate and up sums of this K half (NH = 2)
  __syncthreads();  // every wavefront is done with the activation codes
  float* red = reinterpret_cast<float*>(sX);
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int n = 0; n < 2; ++n)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[((kq * PAIRS + pw) * R + 16 * i + 4 * q + r) * 32 + 16 * n + lr] = acc[i][n][r];
  __syncthreads();
  const int per_pair = static_cast<int>(M) * 16;
  for (int e = t; e < PAIRS * per_pair; e += kVuWaves * 64) {
    const int pp = e / per_pair, rem = e - pp * per_pair;
    const int row = rem >> 4, col = rem & 15;
    const int64_t pr = static_cast<int64_t>(blockIdx.x) * PAIRS + pp;
    if (pr >= npair) continue;
    float g = red[(pp * R + row) * 32 + col], u = red[(pp * R + row) * 32 + 16 + col];
#pragma unroll
    for (int k = 1; k < KQ; ++k) {
      g += red[((k * PAIRS + pp) * R + row) * 32 + col];
      u += red[((k * PAIRS + pp) * R + row) * 32 + 16 + col];
    }
    if (NH == 1) {
      const float h = swiglu_fast(g, u);
      hbuf[row * I + 16 * pr + col] = h;
      if (h_tap != nullptr) h_tap[row * I + 16 * pr + col] = h;
    } else {
      float* part = hbuf + static_cast<int64_t>(kh) * M * 2 * I + row * 2 * I;
      part[16 * pr + col] = g;
      part[I + 16 * pr + col] = u;
    }
  }
}

// down: 16 output columns per workgroup; its SPLIT wavefronts take a part
// of K each and stream their part of the h codes (the M rows) and the 16
// weight rows into a private LDS ring with direct-to-LDS copies, one K-group
// per slot, so the streaming needs no workgroup barrier; the fp32 partials
// meet in LDS at the end and are added in wavefront order. Every workgroup
// reads all of h, which at 256 workgroups is twice the weight bytes; those
// re-reads hit L2, and the copy path takes them at a better rate than
// register loads of 16 rows x 64 bytes each (the operand layout of
// row-major h).
//
// Slot layout: the h rows [R][128 B], chunk c of row r at c ^ (r mod 8);
// then the K-group's weight tile as two 1 KB halves of [16 rows][4 chunks],
// chunk c of row r at c ^ ((r / 4) mod 4). Either way the 16 rows of an
// operand read fall on different bank groups. A weight half is one copy
// instruction reading 1 KB contiguous of the tile.
//
// Up to 32 rows and 96 K-groups (I <= 12288) a workgroup runs 8 wavefronts of
// at most 12 K-groups each, with rings of 4 (16 rows) or 3 (32 rows) slots;
// otherwise 4 wavefronts of at most 32. The same bytes are in flight per CU
// either way, and the 8-wavefront form streams faster: at H = 4096,
// I = 12288 the whole FFN step took 37.75 against 38.56 us at 32 rows and
// 33.80 against 34.66 us at one row.
constexpr int kDnSplit = 4;     // wavefronts (K parts) per workgroup (the general case)
constexpr int kDnMaxNkbW = 32;  // ... and their K-groups each, at most (scales staged in LDS)

// SPLIT wavefronts of NKW K-groups each, at most; the ring as deep as the LDS allows
template <int MT, int SPLIT, int NKW>
struct DnCfg {
  static constexpr int RA = MT * 16;        // activation rows in a slot (padded)
  static constexpr int kA = RA * 128;       // activation bytes per slot
  static constexpr int kSlot = kA + 2048;
  static constexpr int AI = RA / 8;         // 1 KB copies of activations per slot
  static constexpr int PER = AI + 2;        // copies per slot (activations + the two weight halves)
  static constexpr int kFree = 163840 - SPLIT * NKW * (RA + 1) * 4;
  static constexpr int D0 = kFree / (SPLIT * kSlot);
  static constexpr int D = D0 > 8 ? 8 : D0;  // ring depth that fits the LDS
  static_assert(D >= 2, "ring depth");
};

template <int MT, int SPLIT, int NKW>
__global__ __launch_bounds__(SPLIT * 64) void skinny_down_kernel(
    const uint8_t* __restrict__ aq, const float* __restrict__ as,  // h codes [M x K], scales [K/128 x M]
    const uint8_t* __restrict__ wq, const float* __restrict__ ws,  // W_down codes (tile layout), scales [N/128 x K/128]
    uint16_t* __restrict__ out, float* __restrict__ out_tap, int64_t M, int64_t K, int64_t N) {
  using C = DnCfg<MT, SPLIT, NKW>;
  constexpr int D = C::D, RA = C::RA;
  __shared__ __align__(16) uint8_t ring[SPLIT][D * C::kSlot];
  __shared__ __align__(16) float sXs[SPLIT][NKW * RA];
  __shared__ float sWs[SPLIT][NKW];

  const int t = threadIdx.x, lane = t & 63;
  const int wave = wave_uniform(t >> 6);
  const int q = lane >> 4, lr = lane & 15;
  const int64_t KB = K / 128;
  const int64_t n0 = static_cast<int64_t>(blockIdx.x) * 16;
  const int64_t kb0 = wave * KB / SPLIT, kb1 = (wave + 1) * KB / SPLIT;
  const int nkb = static_cast<int>(kb1 - kb0);  // 0 when K has fewer groups than wavefronts
  uint8_t* my = ring[wave];

  // copy plan, h: instruction u fills slot rows 8u..8u+7; lane l fills row
  // 8u + l/8, physical chunk l%8, i.e. logical chunk (l%8) ^ (row & 7)
  const int crow = lane >> 3, pch = lane & 7;
  int64_t a_off[C::AI];
#pragma unroll
  for (int u = 0; u < C::AI; ++u) {
    const int row = 8 * u + crow;
    const int64_t gr = row < M ? row : M - 1;
    a_off[u] = gr * K + ((pch ^ (row & 7)) << 4);
  }
  // weights: half h of the tile, lane l fills row l/4, physical chunk l%4,
  // i.e. logical chunk (l%4) ^ ((l/16) mod 4)
  const int wr_ = lane >> 2, wc = (lane & 3) ^ ((lane >> 4) & 3);
  const uint8_t* wtile = wq + wtile_off(n0, 0, K) + wr_ * 64 + wc * 16;  // + kg * 2048 + h * 1024
  auto issue = [&](int b, int slot) {
    const int64_t kg = kb0 + (b < nkb ? b : nkb - 1);  // past the end: the last K-group again
    const uint32_t base = lds_u32(my + slot * C::kSlot);
#pragma unroll
    for (int u = 0; u < C::AI; ++u) dma16(aq + a_off[u] + kg * 128, wave_uniform(static_cast<int>(base) + u * 1024));
#pragma unroll
    for (int h = 0; h < 2; ++h)
      dma16(wtile + kg * 2048 + h * 1024, wave_uniform(static_cast<int>(base) + C::kA + h * 1024));
  };
  if (nkb > 0) {
#pragma unroll
    for (int b = 0; b < D - 1; ++b) issue(b, b);
  }

  // ---- this wavefront's scales, staged in LDS (loaded after the first copies)
  {
    constexpr int XPT = NKW * RA / 64;
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

  // the weight operand of lane (q, lr): row lr, logical chunks q (half 0) and q (half 1)
  const int wslot = lr * 64 + ((q ^ ((lr >> 2) & 3)) << 4);
  float acc[MT][4];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[i][r] = 0.0f;
  for (int b = 0; b < nkb; ++b) {
    wait_vm_lds<(D - 2) * C::PER>();  // K-group b has landed; slot (b-1) % D is read
    issue(b + D - 1, (b + D - 1) % D);
    const uint8_t* slot = my + (b % D) * C::kSlot;
    const v8i bf = cat_frag(*reinterpret_cast<const u4v*>(slot + C::kA + wslot),
                            *reinterpret_cast<const u4v*>(slot + C::kA + 1024 + wslot));
    const float w = sWs[wave][b];
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const uint8_t* row = slot + (16 * i + lr) * 128;
      const v8i af = cat_frag(*reinterpret_cast<const u4v*>(row + ((q ^ (lr & 7)) << 4)),
                              *reinterpret_cast<const u4v*>(row + (((4 + q) ^ (lr & 7)) << 4)));
      const float4 x4 = *reinterpret_cast<const float4*>(&sXs[wave][b * RA + 16 * i + 4 * q]);
      const v4f zero = {0.0f, 0.0f, 0.0f, 0.0f};
      const v4f p = mfma_fp8_16x16x128(af, bf, zero);
      acc[i][0] = __builtin_fmaf(p[0], x4.x * w, acc[i][0]);
      acc[i][1] = __builtin_fmaf(p[1], x4.y * w, acc[i][1]);
      acc[i][2] = __builtin_fmaf(p[2], x4.z * w, acc[i][2]);
      acc[i][3] = __builtin_fmaf(p[3], x4.w * w, acc[i][3]);
    }
  }
  wait_vm<0>();     // the trailing repeat copies
  __syncthreads();  // every ring is idle: reuse the space for the partials

  // ---- partials [wave][RA][16] -> sum in wavefront order -> bf16
  float* red = reinterpret_cast<float*>(&ring[0][0]);
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) red[(wave * RA + 16 * i + 4 * q + r) * 16 + lr] = acc[i][r];
  __syncthreads();
  for (int e = t; e < M * 16; e += SPLIT * 64) {
    const int row = e >> 4, col = e & 15;
    float sum = red[row * 16 + col];
#pragma unroll
    for (int w = 1; w < SPLIT; ++w) sum += red[(w * RA + row) * 16 + col];
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

// The same quantization after the two K halves of the gate/up sums are
// combined: g = part[0] + part[1] and u likewise (in that order), h =
// SiLU(g) u; parts [2][M][2I] fp32 (gate columns, then up). h_tap: the h
// that was quantized, or null.
__global__ __launch_bounds__(256) void skinny_hquant2_kernel(const float* __restrict__ part, uint8_t* __restrict__ hq,
                                                             float* __restrict__ hs, float* __restrict__ h_tap,
                                                             int64_t M, int64_t I) {
  const int64_t gi = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) >> 4;  // group index, row-major
  const int sub = threadIdx.x & 15;
  const int64_t G = I / 128;
  const bool ok = gi < M * G;
  const int64_t row = ok ? gi / G : 0, g = ok ? gi % G : 0;
  const int64_t c0 = g * 128 + sub * 8;
  const float* p0 = part + row * 2 * I;
  const float* p1 = p0 + M * 2 * I;
  float v[8];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const float4 ga = *reinterpret_cast<const float4*>(p0 + c0 + 4 * h);
    const float4 gb = *reinterpret_cast<const float4*>(p1 + c0 + 4 * h);
    const float4 ua = *reinterpret_cast<const float4*>(p0 + I + c0 + 4 * h);
    const float4 ub = *reinterpret_cast<const float4*>(p1 + I + c0 + 4 * h);
    v[4 * h + 0] = swiglu_fast(ga.x + gb.x, ua.x + ub.x);
    v[4 * h + 1] = swiglu_fast(ga.y + gb.y, ua.y + ub.y);
    v[4 * h + 2] = swiglu_fast(ga.z + gb.z, ua.z + ub.z);
    v[4 * h + 3] = swiglu_fast(ga.w + gb.w, ua.w + ub.w);
  }
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
  *reinterpret_cast<uint2*>(hq + row * I + c0) = make_uint2(lo, hi);
  if (sub == 0) hs[g * M + row] = s;
  if (h_tap != nullptr) {
    *reinterpret_cast<float4*>(h_tap + row * I + c0) = make_float4(v[0], v[1], v[2], v[3]);
    *reinterpret_cast<float4*>(h_tap + row * I + c0 + 4) = make_float4(v[4], v[5], v[6], v[7]);
  }
}

// Shapes the kernels cover: M <= 32 activation rows over all of K (NH = 1),
// or 33..64 rows over half of K (NH = 2), that fit the gate/up kernel's LDS
// and scale tables; down: K parts that fit its scale tables.
int gateup_halves(int64_t M) { return M <= 32 ? 1 : 2; }
bool gateup_v_ok(int64_t M, int64_t K) {
  const int64_t R = ((M + 15) / 16) * 16, KB = K / 128, nh = gateup_halves(M);
  const int64_t kbw = (KB + nh - 1) / nh;  // K-groups of the larger piece
  return M <= 64 && KB <= kVuMaxNkb && R * (kbw * 128 + 16) <= kVuXBytes && kbw * R <= kVuScales;
}
bool down_ok(int64_t M, int64_t K) { return M <= 64 && K / 128 <= kDnSplit * kDnMaxNkbW; }

}  // namespace

bool skinny_supported(int64_t M, int64_t H, int64_t I) {
  return M >= 1 && M <= kSkinnyMaxM && gateup_v_ok(M, H) && down_ok(M, I);
}

size_t skinny_gateup_ws_bytes(int64_t M, int64_t I) {
  // h [M x I] fp32, or for 33..64 rows the two K halves' gate and up sums [2][M][2I]
  const size_t n = static_cast<size_t>(M) * static_cast<size_t>(I) * (gateup_halves(M) == 1 ? 1 : 4);
  return ((n * sizeof(float) + 255) / 256) * 256;
}

// ws_buf: an fp32 buffer of skinny_gateup_ws_bytes() for h. The shape must
// pass skinny_supported().
hipError_t launch_gateup_skinny(hipStream_t st, const uint8_t* xq, const float* xs, const uint8_t* wq,
                                const float* ws, uint8_t* hq, float* hs, float* h_tap, int64_t M, int64_t H,
                                int64_t I, void* ws_buf) {
  float* hbuf = static_cast<float*>(ws_buf);
  const dim3 block(kVuWaves * 64);
  const int64_t groups = M * (I / 128);
  const dim3 qgrid(static_cast<unsigned>((groups + 15) / 16)), qblock(256);
  // up to 32 rows: 3 slab pairs x 4 K parts per workgroup (256 workgroups at
  // I = 12288); 33..64 rows, each workgroup on one K half: 6 pairs x 2 parts,
  // so the two halves still make one round of one workgroup per CU
  const unsigned gx1 = static_cast<unsigned>((I / 16 + 2) / 3), gx2 = static_cast<unsigned>((I / 16 + kNh2Pairs - 1) / kNh2Pairs);
  if (M <= 16)
    hipLaunchKernelGGL((skinny_gateup_kernel<1, kVuDR, 1, 3, 4>), dim3(gx1), block, 0, st, xq, xs, wq, ws, h_tap, hbuf, M, H,
                       I);
  else if (M <= 32)
    hipLaunchKernelGGL((skinny_gateup_kernel<2, kVuDR, 1, 3, 4>), dim3(gx1), block, 0, st, xq, xs, wq, ws, h_tap, hbuf, M, H,
                       I);
  else if (M <= 48)
    hipLaunchKernelGGL((skinny_gateup_kernel<3, kVuDR, 2, kNh2Pairs, kVuWaves / kNh2Pairs>), dim3(gx2, 2), block, 0, st, xq,
                       xs, wq, ws, h_tap, hbuf, M, H, I);
  else
    hipLaunchKernelGGL((skinny_gateup_kernel<4, kVuDR, 2, kNh2Pairs, kVuWaves / kNh2Pairs>), dim3(gx2, 2), block, 0, st, xq,
                       xs, wq, ws, h_tap, hbuf, M, H, I);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (M <= 32)
    hipLaunchKernelGGL(skinny_hquant_kernel, qgrid, qblock, 0, st, hbuf, hq, hs, M, I);
  else
    hipLaunchKernelGGL(skinny_hquant2_kernel, qgrid, qblock, 0, st, hbuf, hq, hs, h_tap, M, I);
  return hipGetLastError();
}

hipError_t launch_quant_groups_f32(hipStream_t st, const float* v, uint8_t* codes, float* scales, int64_t M, int64_t K) {
  const int64_t groups = M * (K / 128);
  hipLaunchKernelGGL(skinny_hquant_kernel, dim3(static_cast<unsigned>((groups + 15) / 16)), dim3(256), 0, st, v, codes,
                     scales, M, K);
  return hipGetLastError();
}

// The shape must pass skinny_supported().
hipError_t launch_down_skinny(hipStream_t st, const uint8_t* hq, const float* hs, const uint8_t* wq, const float* ws,
                              uint16_t* out, float* out_tap, int64_t M, int64_t H, int64_t I) {
  const dim3 grid(static_cast<unsigned>(H / 16)), block(kDnSplit * 64);
  // up to 32 rows and I <= 12288: 8 wavefronts of at most 12 K-groups each
  const bool wide = M <= 32 && I / 128 <= 8 * 12;
  const dim3 block8(8 * 64);
  if (M <= 16) {
    if (wide)
      hipLaunchKernelGGL((skinny_down_kernel<1, 8, 12>), grid, block8, 0, st, hq, hs, wq, ws, out, out_tap, M, I, H);
    else
      hipLaunchKernelGGL((skinny_down_kernel<1, kDnSplit, kDnMaxNkbW>), grid, block, 0, st, hq, hs, wq, ws, out, out_tap,
                         M, I, H);
  } else if (M <= 32) {
    if (wide)
      hipLaunchKernelGGL((skinny_down_kernel<2, 8, 12>), grid, block8, 0, st, hq, hs, wq, ws, out, out_tap, M, I, H);
    else
      hipLaunchKernelGGL((skinny_down_kernel<2, kDnSplit, kDnMaxNkbW>), grid, block, 0, st, hq, hs, wq, ws, out, out_tap,
                         M, I, H);
  } else if (M <= 48) {
    hipLaunchKernelGGL((skinny_down_kernel<3, kDnSplit, kDnMaxNkbW>), grid, block, 0, st, hq, hs, wq, ws, out, out_tap, M,
                       I, H);
  } else {
    hipLaunchKernelGGL((skinny_down_kernel<4, kDnSplit, kDnMaxNkbW>), grid, block, 0, st, hq, hs, wq, ws, out, out_tap, M,
                       I, H);
  }
  return hipGetLastError();
}

}  // namespace lacache
