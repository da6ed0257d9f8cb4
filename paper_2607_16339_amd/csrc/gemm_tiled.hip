// Tiled FP8 MFMA GEMMs with per-group dequantization (Sec. 3.4):
//   gate/up: x[M x H] . Wgu[2I x H]^T, fused SwiGLU and 1x128 re-quantization
//   down:    h[M x I] . Wd[H x I]^T -> bf16
//
// A workgroup of BM/32 wavefronts computes a BM-row x 256-weight-row tile.
// Each wavefront owns 64 rows x 128 weight rows (4 x 8 sub-tiles of 16x16).
// K is walked one 128-wide group at a time:
//   * the group's fp8 tiles (A: BM x 128 B, B: 256 x 128 B) and the BM
//     activation scales go global -> LDS with direct-to-LDS loads into one of
//     two LDS stages, issued one group ahead, so no registers hold staging
//     data and the copy of group kb+1 overlaps the MFMAs of group kb;
//   * every 16x16 sub-tile gets one 16x16x128 FP8 MFMA (exactly one K-group)
//     and its fp32 result is added to the accumulator times
//     RN32(x_scale[row] * w_scale[block]): four VALU FMAs per MFMA, which the
//     VALU issues while the matrix core works.
// One workgroup barrier per K-group.
//
// For gate/up the tile's 256 weight rows are the 128 gate rows and the 128
// matching up rows of one h-group, so each lane holds gate and up values of
// the same (row, column) and a row's whole 128-wide h-group lives in one
// workgroup: SwiGLU, the row amax and the e4m3 encoding happen in registers
// and LDS before anything is written; h never reaches memory.
#include "device.h"
#include "launch.h"

namespace lacache {
namespace {

constexpr int BNR = 256;           // weight rows per workgroup
constexpr int kMaxKGroups = 512;   // K <= 65536
#ifndef LACACHE_L2_PREFETCH
#define LACACHE_L2_PREFETCH 0
#endif
constexpr bool kL2Prefetch = LACACHE_L2_PREFETCH != 0;

// LDS tiles are [rows][128 bytes]; the eight 16-byte chunks of a row are
// permuted by an xor with (row / 2) mod 8, which spreads the 16 rows of an
// MFMA operand read over the banks (the best of the permutations measured).
__device__ __forceinline__ int swz(int row) { return (row >> 1) & 7; }
__device__ __forceinline__ int lds_off(int row, int chunk) { return row * 128 + ((chunk ^ swz(row)) << 4); }

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

// One LDS stage: A tile, B tile, activation scales.
template <int BM>
struct Stage {
  uint8_t a[BM * 128];
  uint8_t b[BNR * 128];
  alignas(16) float xs[BM + 64];  // BM scales + a spare slot for redundant copies
};

// s_waitcnt with only vmcnt constrained (gfx9 encoding: vmcnt in bits 3:0,
// expcnt 6:4 and lgkmcnt 11:8 left at their maxima). The builtin, unlike
// inline asm, is visible to the compiler's own wait-count tracking.
__device__ __forceinline__ void wait_vm0() { __builtin_amdgcn_s_waitcnt(0x0F70); }
// Workgroup barrier between pipeline steps. Each wave has already waited for
// its own copies into the next stage, and every LDS read of the current stage
// has been consumed, so no memory fence is needed (a fence would also wait
// for the L2 prefetches); the empty asm statements keep the compiler from
// moving LDS accesses across it.
__device__ __forceinline__ void stage_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}
template <int N>
__device__ __forceinline__ void wait_vm_prefetch() {
  static_assert(N >= 0 && N < 16, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | N);
}

// Scheduling hint: one MFMA followed by four VALU instructions.
__device__ __forceinline__ void sched_mfma_then_4valu() {
  __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
  __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
}

}  // namespace

template <bool kGateUp, int BM>
__global__ __launch_bounds__(BM / 32 * 64) void gemm_tiled_kernel(
    const uint8_t* __restrict__ aq, const float* __restrict__ as,  // [M x K] codes, [K/128 x M] scales
    const uint8_t* __restrict__ bq, const float* __restrict__ bs,  // [N x K] codes, [N/128 x K/128] scales
    uint8_t* __restrict__ hq, float* __restrict__ hs, float* __restrict__ h_tap,
    uint16_t* __restrict__ out, float* __restrict__ out_tap, int64_t M, int64_t K, int64_t N, int64_t I) {
  constexpr int NW = BM / 32;  // wavefronts: BM/64 along rows x 2 along weight rows
  static_assert(NW == 4 || NW == 8, "BM must be 128 or 256");
  __shared__ Stage<BM> st0, st1;
  __shared__ float sRed[2][BM];
  __shared__ float sW[2][kMaxKGroups];  // the two weight-block scale rows used by this workgroup

  const int t = threadIdx.x, lane = t & 63;
  // wavefront index made visibly uniform: scale loads and LDS bases go scalar
  const int wave = wave_uniform(t >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int q = lane >> 4, lr = lane & 15;
  int64_t tile_r, tile_c;
  xcd_grouped_tile(blockIdx.x, (M + BM - 1) / BM, gridDim.x / ((M + BM - 1) / BM), tile_r, tile_c);
  const int64_t m0 = tile_r * BM;
  const int64_t by = tile_c;  // gate/up: h-group; down: 256-column tile
  const int64_t KB = K / 128;
  const int64_t n0 = kGateUp ? 0 : by * BNR;

  // ---- direct-to-LDS copy plan. A wave's load instruction fills 64
  // consecutive 16-byte LDS slots (8 tile rows); lane l fills slot l, i.e.
  // row 8g + l/8, physical chunk l%8, so it fetches logical chunk
  // (l%8) ^ swz(row) of that row. Rows past M (or N) fetch a clamped row;
  // their results are never stored. Per-lane offsets are 32-bit, relative to
  // workgroup-uniform bases.
  constexpr int kAInst = BM / 8 / NW;  // per wave
  constexpr int kBInst = BNR / 8 / NW;
  const uint8_t* a_base = aq + m0 * K;
  uint32_t a_off[kAInst], b_off[kBInst];
#pragma unroll
  for (int u = 0; u < kAInst; ++u) {
    const int row = (wave * kAInst + u) * 8 + (lane >> 3);
    const int64_t r = m0 + row < M ? row : M - 1 - m0;
    a_off[u] = static_cast<uint32_t>(r * K + ((lane & 7) ^ swz(row)) * 16);
  }
  // gate/up: rows 0..127 of the tile come from the gate block, 128..255 from
  // the up block (base b_base_hi); down: one contiguous 256-row block
  const uint8_t* b_base = kGateUp ? bq + by * 128 * K : bq + n0 * K;
  const uint8_t* b_base_hi = kGateUp ? bq + (I + by * 128 - 128) * K : b_base;
#pragma unroll
  for (int u = 0; u < kBInst; ++u) {
    const int row = (wave * kBInst + u) * 8 + (lane >> 3);
    const int64_t r = (kGateUp || n0 + row < N) ? row : N - 1 - n0;
    b_off[u] = static_cast<uint32_t>(r * K + ((lane & 7) ^ swz(row)) * 16);
  }
  // activation scales: waves 0..BM/64-1 copy rows 64w..64w+63 (one float per
  // lane); the other waves copy the same rows into a spare slot
  const int xw = wave % (BM / 64);
  const uint32_t xs_off = static_cast<uint32_t>(m0 + xw * 64 + lane < M ? xw * 64 + lane : M - 1 - m0);
  const int xs_dst = wave < BM / 64 ? wave * 64 : BM;
  const float* xs_base = as + m0;

  // ---- L2 prefetch two K-groups ahead. A row's K-group is one 128-byte
  // cache line; a 1-byte load per lane pulls 64 lines into L2 while moving
  // only 64 bytes. Wave w covers tile rows 64 (w + NW u) .. +63 of the
  // BM + 256 rows (A rows first, then B rows).
  constexpr int kPRows = BM + BNR;
  constexpr int kPInst = kL2Prefetch ? (kPRows / 64 + NW - 1) / NW : 0;
  const uint8_t* p_base[kPInst > 0 ? kPInst : 1];
  uint32_t p_off[kPInst > 0 ? kPInst : 1];
#pragma unroll
  for (int u = 0; u < kPInst; ++u) {
    int row = 64 * (wave + NW * u) + lane;
    if (row >= kPRows) row = kPRows - 1;
    if (row < BM) {
      p_base[u] = a_base;
      p_off[u] = static_cast<uint32_t>((m0 + row < M ? row : M - 1 - m0) * K);
    } else {
      const int br = row - BM;
      p_base[u] = (kGateUp && br >= 128) ? b_base_hi : b_base;
      p_off[u] = static_cast<uint32_t>(((kGateUp || n0 + br < N) ? br : N - 1 - n0) * K);
    }
  }

  // (down: the wave's 128 columns may lie past N in the last column tile)
  const bool nb_ok = kGateUp || n0 + 128 * wn < N;
  // The workgroup's weight-block scales for all K-groups, staged in LDS once:
  // gate/up rows {gate block, up block}; down rows {block of wn = 0, wn = 1}.
  {
    const int64_t r0 = kGateUp ? by : n0 / 128;
    const int64_t r1 = kGateUp ? I / 128 + by : (n0 + 128 < N ? n0 / 128 + 1 : r0);
    for (int64_t i = t; i < 2 * KB; i += NW * 64) {
      const int64_t row = i < KB ? r0 : r1;
      sW[i < KB ? 0 : 1][i < KB ? i : i - KB] = bs[row * KB + (i < KB ? i : i - KB)];
    }
  }
  const int wsel0 = kGateUp ? 0 : wn, wsel1 = kGateUp ? 1 : wn;

  float acc[4][8][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[i][j][r] = 0.0f;

  // Copies K-group kn into stage `nxt` (asynchronously) and multiplies K-group
  // kb from stage `cur`. The two stages never alias; the restrict qualifiers
  // let the compiler see that, so reading `cur` does not wait for the copy.
  uint32_t sink = 0u;  // destination of the prefetch loads, live until the final vmcnt(0)
  auto prefetch = [&](int64_t kp) {
#pragma unroll
    for (int u = 0; u < kPInst; ++u) prefetch_l2(p_base[u] + kp * 128 + p_off[u], sink);
  };
  auto step = [&](const Stage<BM>* __restrict__ cur, Stage<BM>* __restrict__ nxt, int64_t kb, int64_t kn,
                  int64_t kp) {
    const int64_t ko = kn * 128;
#pragma unroll
    for (int u = 0; u < kAInst; ++u)
      lds_dma16(a_base + ko + a_off[u], nxt->a + (wave * kAInst + u) * 1024);
#pragma unroll
    for (int u = 0; u < kBInst; ++u) {
      const uint8_t* base = (kGateUp && (wave * kBInst + u) * 8 >= 128) ? b_base_hi : b_base;
      lds_dma16(base + ko + b_off[u], nxt->b + (wave * kBInst + u) * 1024);
    }
    lds_dma4(xs_base + kn * M + xs_off, nxt->xs + xs_dst);
    prefetch(kp);

    const float w0 = nb_ok ? sW[wsel0][kb] : 0.0f;
    const float w1 = nb_ok ? sW[wsel1][kb] : 0.0f;
    v8i af[4];
    float sc[2][4][4];  // RN32(x_scale * w_scale) for the two weight blocks
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      af[i] = load_frag(cur->a, 64 * wm + 16 * i + lr, q);
      const float4 xv = *reinterpret_cast<const float4*>(cur->xs + 64 * wm + 16 * i + 4 * q);
      const float xa[4] = {xv.x, xv.y, xv.z, xv.w};
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        sc[0][i][r] = xa[r] * w0;
        sc[1][i][r] = xa[r] * w1;
      }
    }
    // Software pipeline over the 32 sub-tiles: MFMA s is issued before the
    // four scale FMAs of MFMA s-1, so the VALU works on a finished result
    // while the matrix core runs; the B operand of slab j+1 is read from
    // LDS while slab j multiplies.
    auto brow = [&](int j) {
      return kGateUp ? (j < 4 ? 64 * wn + 16 * j : 128 + 64 * wn + 16 * (j - 4)) : 128 * wn + 16 * j;
    };
    v8i bcur = load_frag(cur->b, brow(0) + lr, q);
    v4f pprev = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const v8i bnext = j < 7 ? load_frag(cur->b, brow(j + 1) + lr, q) : bcur;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const v4f zero = {0.0f, 0.0f, 0.0f, 0.0f};
        const v4f p = mfma_fp8_16x16x128(af[i], bcur, zero);
        const int s = j * 4 + i;
        if (s > 0) {
          const int pi = (s - 1) & 3, pj = (s - 1) >> 2;
          const int blk = (kGateUp && pj >= 4) ? 1 : 0;
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[pi][pj][r] = __builtin_fmaf(pprev[r], sc[blk][pi][r], acc[pi][pj][r]);
        }
        pprev = p;
        sched_mfma_then_4valu();
      }
      bcur = bnext;
    }
    {
      const int blk = kGateUp ? 1 : 0;
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[3][7][r] = __builtin_fmaf(pprev[r], sc[blk][3][r], acc[3][7][r]);
    }
    // loads retire in issue order: this waits for the stage copy while the
    // kPInst prefetches issued after it stay in flight across the barrier
    wait_vm_prefetch<kPInst>();
    stage_barrier();
  };

  // ---- main loop: two LDS stages, the copy of the next group in flight. The
  // last step re-fetches its own group into the idle stage (never read).
  {
    const int64_t ko = 0;
#pragma unroll
    for (int u = 0; u < kAInst; ++u)
      lds_dma16(a_base + ko + a_off[u], st0.a + (wave * kAInst + u) * 1024);
#pragma unroll
    for (int u = 0; u < kBInst; ++u) {
      const uint8_t* base = (kGateUp && (wave * kBInst + u) * 8 >= 128) ? b_base_hi : b_base;
      lds_dma16(base + ko + b_off[u], st0.b + (wave * kBInst + u) * 1024);
    }
    lds_dma4(xs_base + xs_off, st0.xs + xs_dst);
    prefetch(KB > 1 ? 1 : 0);
    wait_vm_prefetch<kPInst>();
    __syncthreads();
  }
  auto clampk = [&](int64_t k) { return k < KB ? k : KB - 1; };
  for (int64_t kb = 0; kb < KB; kb += 2) {
    step(&st0, &st1, kb, clampk(kb + 1), clampk(kb + 2));
    if (kb + 1 >= KB) break;
    step(&st1, &st0, kb + 1, clampk(kb + 2), clampk(kb + 3));
  }
  wait_vm0();

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
          const float v = swiglu_fast(acc[i][j][r], acc[i][j + 4][r]);
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
    // ---- 1x128 quantization of each row's h-group; codes staged in LDS for coalesced stores
    uint8_t* codes = st0.a;  // BM x 128 bytes, free after the main loop
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 64 * wm + 16 * i + 4 * q + r;
        const float s = __builtin_fmaxf(sRed[0][row], sRed[1][row]) / kE4M3Max;
        const bool fast = scale_is_fast(s);
        const float rs = fast_rcp(s);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int col = 64 * wn + 16 * j + lr;
          const float v = h[i][j][r];
          uint32_t c = 0u;
          if (s != 0.0f) c = fast ? enc1_div_fast(v, s, rs) : enc1_e4m3(qdiv(v, s));
          codes[row * 128 + col] = static_cast<uint8_t>(c);
          if (h_tap != nullptr && m0 + row < M) h_tap[(m0 + row) * I + by * 128 + col] = h[i][j][r];
        }
      }
    __syncthreads();
    for (int c = t; c < BM * 8; c += NW * 64) {
      const int row = c >> 3, ch = c & 7;
      if (m0 + row < M)
        *reinterpret_cast<uint4*>(hq + (m0 + row) * I + by * 128 + ch * 16) =
            *reinterpret_cast<const uint4*>(codes + row * 128 + ch * 16);
    }
    for (int row = t; row < BM; row += NW * 64)
      if (m0 + row < M) hs[by * M + m0 + row] = __builtin_fmaxf(sRed[0][row], sRed[1][row]) / kE4M3Max;
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

template __global__ void gemm_tiled_kernel<true, 256>(const uint8_t*, const float*, const uint8_t*, const float*,
                                                     uint8_t*, float*, float*, uint16_t*, float*, int64_t, int64_t,
                                                     int64_t, int64_t);
template __global__ void gemm_tiled_kernel<true, 128>(const uint8_t*, const float*, const uint8_t*, const float*,
                                                     uint8_t*, float*, float*, uint16_t*, float*, int64_t, int64_t,
                                                     int64_t, int64_t);
template __global__ void gemm_tiled_kernel<false, 256>(const uint8_t*, const float*, const uint8_t*, const float*,
                                                      uint8_t*, float*, float*, uint16_t*, float*, int64_t, int64_t,
                                                      int64_t, int64_t);
template __global__ void gemm_tiled_kernel<false, 128>(const uint8_t*, const float*, const uint8_t*, const float*,
                                                      uint8_t*, float*, float*, uint16_t*, float*, int64_t, int64_t,
                                                      int64_t, int64_t);

namespace {

template <bool kGateUp, int BM>
hipError_t launch_tiled(hipStream_t st, const uint8_t* aq, const float* as, const uint8_t* bq, const float* bs,
                        uint8_t* hq, float* hs, float* h_tap, uint16_t* out, float* out_tap, int64_t M, int64_t K,
                        int64_t N, int64_t I) {
  const int64_t ny = kGateUp ? I / 128 : (N + BNR - 1) / BNR;
  const dim3 grid(static_cast<unsigned>(((M + BM - 1) / BM) * ny));
  hipLaunchKernelGGL((gemm_tiled_kernel<kGateUp, BM>), grid, dim3(BM / 32 * 64), 0, st, aq, as, bq, bs, hq, hs,
                     h_tap, out, out_tap, M, K, N, I);
  return hipGetLastError();
}

// Row-tile height: 256 when there are enough row tiles to fill the chip with
// one workgroup per CU, else 128.
bool use_bm256(int64_t M, int64_t col_tiles) { return ((M + 255) / 256) * col_tiles >= 512; }

}  // namespace

hipError_t launch_gateup_tiled(hipStream_t st, const uint8_t* xq, const float* xs, const uint8_t* wq,
                               const float* ws, uint8_t* hq, float* hs, float* h_tap, int64_t M, int64_t H,
                               int64_t I) {
  if (use_bm256(M, I / 128))
    return launch_tiled<true, 256>(st, xq, xs, wq, ws, hq, hs, h_tap, nullptr, nullptr, M, H, 2 * I, I);
  return launch_tiled<true, 128>(st, xq, xs, wq, ws, hq, hs, h_tap, nullptr, nullptr, M, H, 2 * I, I);
}

hipError_t launch_down_tiled(hipStream_t st, const uint8_t* hq, const float* hs, const uint8_t* wq, const float* ws,
                             uint16_t* out, float* out_tap, int64_t M, int64_t H, int64_t I) {
  if (use_bm256(M, (H + BNR - 1) / BNR))
    return launch_tiled<false, 256>(st, hq, hs, wq, ws, nullptr, nullptr, nullptr, out, out_tap, M, I, H, I);
  return launch_tiled<false, 128>(st, hq, hs, wq, ws, nullptr, nullptr, nullptr, out, out_tap, M, I, H, I);
}

}  // namespace lacache
