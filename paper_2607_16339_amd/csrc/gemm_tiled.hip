// Tiled FP8 MFMA GEMMs with per-group dequantization (Sec. 3.4):
//   gate/up: x[M x H] . Wgu[2I x H]^T, fused SwiGLU and 1x128 re-quantization
//   down:    h[M x I] . Wd[H x I]^T -> bf16
//
// A workgroup of BM/32 wavefronts computes a BM-row x 256-weight-row tile.
// Wavefront (wm, wn) owns rows 64 wm.. x weight rows 128 wn.. (4 x 8
// sub-tiles of 16x16), i.e. one 128-row weight block. K is walked one
// 128-wide group at a time:
//   * the group's fp8 tiles (A: BM x 128 B, B: 256 x 128 B) and the BM
//     activation scales go global -> LDS with direct-to-LDS copies into one
//     of two LDS stages, issued one group ahead, so no registers hold staging
//     data and the copy of group kb+1 overlaps the MFMAs of group kb;
//   * every 16x16 sub-tile gets one 16x16x128 FP8 MFMA (exactly one K-group)
//     and its fp32 result is added to the accumulator times
//     RN32(x_scale[row] * w_scale[block]): four VALU FMAs per MFMA, issued two
//     MFMAs later so that they find the result finished, while the matrix
//     core works on the next ones; the B operand of the next 16-row slab is
//     read from LDS while the current one multiplies.
// One workgroup barrier per K-group.
//
// For gate/up the tile's 256 weight rows are the 128 gate rows (wn = 0) and
// the 128 matching up rows (wn = 1) of one h-group: after the K loop the up
// wavefronts hand their values to the gate wavefronts through LDS, so a row's
// whole 128-wide h-group lives in one wavefront: SwiGLU, the row amax and the
// e4m3 encoding happen in registers before anything is written; h never
// reaches memory.
#include "device.h"
#include "launch.h"

namespace lacache {
namespace {

constexpr int BNR = 256;           // weight rows per workgroup
constexpr int kMaxKGroups = 512;   // K <= 65536

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

}  // namespace

// Wave layout: 8 wavefronts; a wavefront owns 64 rows x WC weight rows
// (WC = 128 for BM = 256, 64 for BM = 128), NJ = WC / 16 column slabs. For
// gate/up a wavefront's slabs are WC/2 gate rows and the WC/2 matching up
// rows, so SwiGLU pairs values held by the same lane.
constexpr int kTileWaves = 8;

template <bool kGateUp, int BM>
__global__ __launch_bounds__(kTileWaves * 64) void gemm_tiled_kernel(
    const uint8_t* __restrict__ aq, const float* __restrict__ as,  // [M x K] codes, [K/128 x M] scales
    const uint8_t* __restrict__ bq, const float* __restrict__ bs,  // [N x K] codes, [N/128 x K/128] scales
    uint8_t* __restrict__ hq, float* __restrict__ hs, float* __restrict__ h_tap,
    uint16_t* __restrict__ out, float* __restrict__ out_tap, float* __restrict__ part, int64_t M, int64_t K,
    int64_t N, int64_t I, int KS) {
  static_assert(BM == 128 || BM == 256, "BM must be 128 or 256");
  constexpr int NW = kTileWaves;
  constexpr int WC = BM == 256 ? 128 : 64;  // weight rows (output columns) per wavefront
  constexpr int NCW = BNR / WC;             // wavefronts along the weight rows
  constexpr int NJ = WC / 16;               // 16-wide column slabs per wavefront
  // LDS ring of kStages stages: 3 for BM = 128 (3 x 49.9 KB), 2 for BM = 256
  constexpr int kStages = BM == 128 ? 3 : 2;
  __shared__ Stage<BM> stg[kStages];
  __shared__ float sRed[NCW][BM];
  __shared__ float sW[2][kMaxKGroups];  // the two weight-block scale rows used by this workgroup

  const int t = threadIdx.x, lane = t & 63;
  // wavefront index made visibly uniform: scale loads and LDS bases go scalar
  const int wave = wave_uniform(t >> 6);
  const int wm = wave / NCW, wn = wave % NCW;
  const int q = lane >> 4, lr = lane & 15;
  // down with KS > 1: the KS workgroups of a tile split its K range and
  // store fp32 partials; a second kernel adds them in split order
  const int split = static_cast<int>(blockIdx.x % KS);
  int64_t tile_r, tile_c;
  const int64_t row_tiles = (M + BM - 1) / BM;
  xcd_grouped_tile(blockIdx.x / KS, row_tiles, (gridDim.x / KS) / row_tiles, tile_r, tile_c);
  const int64_t m0 = tile_r * BM;
  const int64_t by = tile_c;  // gate/up: h-group; down: 256-column tile
  const int64_t KB = K / 128;
  const int64_t kb0 = split * KB / KS, kb1 = (split + 1) * KB / KS;
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

  // (down: the wave's columns may lie past N in the last column tile)
  const bool nb_ok = kGateUp || n0 + WC * wn < N;
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

  float acc[4][NJ][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[i][j][r] = 0.0f;

  // Copies of K-group kn into stage dst (asynchronous).
  auto issue = [&](int64_t kn, Stage<BM>* dst) {
    const int64_t ko = kn * 128;
    const int la = static_cast<int>(lds_u32(dst->a)), lb = static_cast<int>(lds_u32(dst->b));
#pragma unroll
    for (int u = 0; u < kAInst; ++u) dma16(a_base + ko + a_off[u], wave_uniform(la + (wave * kAInst + u) * 1024));
#pragma unroll
    for (int u = 0; u < kBInst; ++u) {
      const uint8_t* base = (kGateUp && (wave * kBInst + u) * 8 >= 128) ? b_base_hi : b_base;
      dma16(base + ko + b_off[u], wave_uniform(lb + (wave * kBInst + u) * 1024));
    }
    dma4(xs_base + kn * M + xs_off, wave_uniform(static_cast<int>(lds_u32(dst->xs)) + xs_dst * 4));
  };

  // Multiplies K-group kb from stage cur.
  auto compute = [&](const Stage<BM>* cur, int64_t kb) {
    // gate/up: slabs 0..NJ/2-1 are gate rows, the rest the matching up rows
    // (two weight blocks); down: the wave's columns lie in one block
    const int dblk = (WC * wn) / 128;
    const float w0 = nb_ok ? sW[kGateUp ? 0 : dblk][kb] : 0.0f;
    const float w1 = nb_ok ? sW[kGateUp ? 1 : dblk][kb] : 0.0f;
    v8i af[4];
    float sc[kGateUp ? 2 : 1][4][4];  // RN32(x_scale * w_scale)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      af[i] = load_frag(cur->a, 64 * wm + 16 * i + lr, q);
      const float4 xv = *reinterpret_cast<const float4*>(cur->xs + 64 * wm + 16 * i + 4 * q);
      sc[0][i][0] = xv.x * w0;
      sc[0][i][1] = xv.y * w0;
      sc[0][i][2] = xv.z * w0;
      sc[0][i][3] = xv.w * w0;
      if (kGateUp) {
        sc[kGateUp ? 1 : 0][i][0] = xv.x * w1;
        sc[kGateUp ? 1 : 0][i][1] = xv.y * w1;
        sc[kGateUp ? 1 : 0][i][2] = xv.z * w1;
        sc[kGateUp ? 1 : 0][i][3] = xv.w * w1;
      }
    }
    auto brow = [&](int j) {
      return kGateUp ? (j < NJ / 2 ? (WC / 2) * wn + 16 * j : 128 + (WC / 2) * wn + 16 * (j - NJ / 2)) : WC * wn + 16 * j;
    };
    // Software pipeline over the 4 NJ sub-tiles s = 4 j + i: MFMA s, then the
    // scale FMAs of MFMA s - 2; the B operand of slab j + 1 is read while
    // slab j multiplies.
    v8i bb[2];
    bb[0] = load_frag(cur->b, brow(0) + lr, q);
    v4f pr[3];
#pragma unroll
    for (int s = 0; s < 4 * NJ; ++s) {
      const int j = s >> 2, i = s & 3;
      if (i == 0 && j < NJ - 1) bb[(j + 1) & 1] = load_frag(cur->b, brow(j + 1) + lr, q);
      const v4f zero = {0.0f, 0.0f, 0.0f, 0.0f};
      pr[s % 3] = mfma_fp8_16x16x128(af[i], bb[j & 1], zero);
      if (s >= 2) {
        const int ps = s - 2;
        const int blk = (kGateUp && (ps >> 2) >= NJ / 2) ? 1 : 0;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          acc[ps & 3][ps >> 2][r] = __builtin_fmaf(pr[ps % 3][r], sc[blk][ps & 3][r], acc[ps & 3][ps >> 2][r]);
      }
      // keep this order: the FMAs above read a result two MFMAs old, so they
      // neither wait for the matrix core nor delay the next MFMA
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int ps = 4 * NJ - 2; ps < 4 * NJ; ++ps)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        acc[ps & 3][ps >> 2][r] = __builtin_fmaf(pr[ps % 3][r], sc[kGateUp ? 1 : 0][ps & 3][r], acc[ps & 3][ps >> 2][r]);
  };

  // ---- main loop over a ring of kStages stages, the copies of the next
  // kStages - 1 groups in flight. Steps past the end re-fetch the last group
  // into an idle stage (never read), so every step waits for the same count.
  constexpr int kPer = kAInst + kBInst + 1;  // copies per wave per group
  auto clampk = [&](int64_t k) { return k < kb1 ? k : kb1 - 1; };
#pragma unroll
  for (int s = 0; s < kStages - 1; ++s) issue(clampk(kb0 + s), &stg[s]);
  __syncthreads();  // the weight scales are visible to every wave
  int cur = 0;      // stage of group kb
  for (int64_t kb = kb0; kb < kb1; ++kb) {
    wait_vm_lds<(kStages - 2) * kPer>();  // group kb has landed (later ones may still fly)
    bar();  // ... for every wave; and the stage of group kb - 1 is read by no one
    const int nxt = cur == 0 ? kStages - 1 : cur - 1;  // == (kb + kStages - 1) % kStages
    issue(clampk(kb + kStages - 1), &stg[nxt]);
    compute(&stg[cur], kb);
    cur = cur + 1 == kStages ? 0 : cur + 1;
  }
  wait_vm<0>();
  __syncthreads();  // every wave is done with the ring

  if (kGateUp) {
    // ---- SwiGLU: h = SiLU(g) * u, lanes hold matching gate (j) and up (j + NJ/2) values
    float h[4][NJ / 2][4];
    float am[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float a = 0.0f;
#pragma unroll
        for (int j = 0; j < NJ / 2; ++j) {
          const float v = swiglu_fast(acc[i][j][r], acc[i][j + NJ / 2][r]);
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
    // ---- 1x128 quantization of each row's h-group. A lane's codes for one
    // column slab are gathered four lanes at a time into a 32-bit word (lanes
    // 4m..4m+3 hold four consecutive columns) and stored from lane 4m.
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 64 * wm + 16 * i + 4 * q + r;
        float amax = sRed[0][row];
#pragma unroll
        for (int c = 1; c < NCW; ++c) amax = __builtin_fmaxf(amax, sRed[c][row]);
        const float s = amax / kE4M3Max;
        const float rs = fast_rcp(s);
        // codes of q0 * (1 -+ 2^-20), q0 = h * rs: where every pair agrees they
        // are E(RN32(h / s)) (see enc1_div_fast); else the division decides
        uint32_t cw[NJ / 2];
        bool agree = true;
#pragma unroll
        for (int j = 0; j < NJ / 2; ++j) {
          const float q0 = h[i][j][r] * rs;
          const float d = __builtin_fabsf(q0) * 0x1p-20f;
          const uint32_t w = static_cast<uint32_t>(__builtin_amdgcn_cvt_pk_fp8_f32(clip448(q0 - d), clip448(q0 + d), 0, false));
          cw[j] = w & 0xFFu;
          agree = agree && (w & 0xFFu) == ((w >> 8) & 0xFFu);
        }
        if (s == 0.0f) {
#pragma unroll
          for (int j = 0; j < NJ / 2; ++j) cw[j] = 0u;
        } else if (!(agree && scale_is_fast(s))) {
#pragma unroll
          for (int j = 0; j < NJ / 2; ++j) cw[j] = enc1_e4m3(qdiv(h[i][j][r], s));
        }
#pragma unroll
        for (int j = 0; j < NJ / 2; ++j) {
          const int col = (WC / 2) * wn + 16 * j + lr;
          uint32_t c = cw[j];
          c |= static_cast<uint32_t>(__shfl_down(static_cast<int>(c), 1, 64)) << 8;
          c |= static_cast<uint32_t>(__shfl_down(static_cast<int>(c), 2, 64)) << 16;
          if ((lr & 3) == 0 && m0 + row < M) *reinterpret_cast<uint32_t*>(hq + (m0 + row) * I + by * 128 + col) = c;
          if (h_tap != nullptr && m0 + row < M) h_tap[(m0 + row) * I + by * 128 + col] = h[i][j][r];
        }
      }
    for (int row = t; row < BM; row += NW * 64) {
      float amax = sRed[0][row];
#pragma unroll
      for (int c = 1; c < NCW; ++c) amax = __builtin_fmaxf(amax, sRed[c][row]);
      if (m0 + row < M) hs[by * M + m0 + row] = amax / kE4M3Max;
    }
  } else {
    // ---- bf16 output, nearest-even from the fp32 accumulator
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = m0 + 64 * wm + 16 * i + 4 * q + r;
        if (row >= M) continue;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const int64_t col = n0 + WC * wn + 16 * j + lr;
          if (col < N) {
            if (KS > 1) {
              part[(split * M + row) * N + col] = acc[i][j][r];
            } else {
              out[row * N + col] = static_cast<uint16_t>(f32_to_bf16(acc[i][j][r]));
              if (out_tap != nullptr) out_tap[row * N + col] = acc[i][j][r];
            }
          }
        }
      }
  }
}

template __global__ void gemm_tiled_kernel<true, 256>(const uint8_t*, const float*, const uint8_t*, const float*,
                                                     uint8_t*, float*, float*, uint16_t*, float*, float*, int64_t,
                                                     int64_t, int64_t, int64_t, int);
template __global__ void gemm_tiled_kernel<true, 128>(const uint8_t*, const float*, const uint8_t*, const float*,
                                                     uint8_t*, float*, float*, uint16_t*, float*, float*, int64_t,
                                                     int64_t, int64_t, int64_t, int);
template __global__ void gemm_tiled_kernel<false, 256>(const uint8_t*, const float*, const uint8_t*, const float*,
                                                      uint8_t*, float*, float*, uint16_t*, float*, float*, int64_t,
                                                      int64_t, int64_t, int64_t, int);
template __global__ void gemm_tiled_kernel<false, 128>(const uint8_t*, const float*, const uint8_t*, const float*,
                                                      uint8_t*, float*, float*, uint16_t*, float*, float*, int64_t,
                                                      int64_t, int64_t, int64_t, int);

namespace {

// out = RNE_bf16(sum of the KS partials, in split order); 4 columns per thread.
__global__ __launch_bounds__(256) void split_reduce_kernel(const float* __restrict__ part, uint16_t* __restrict__ out,
                                                           float* __restrict__ out_tap, int64_t MN, int KS) {
  const int64_t e = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 4;
  if (e >= MN) return;
  float4 acc = *reinterpret_cast<const float4*>(part + e);
  for (int sp = 1; sp < KS; ++sp) {
    const float4 p = *reinterpret_cast<const float4*>(part + sp * MN + e);
    acc.x += p.x; acc.y += p.y; acc.z += p.z; acc.w += p.w;
  }
  *reinterpret_cast<uint2*>(out + e) = make_uint2(pack_bf16x2(acc.x, acc.y), pack_bf16x2(acc.z, acc.w));
  if (out_tap != nullptr) *reinterpret_cast<float4*>(out_tap + e) = acc;
}

template <bool kGateUp, int BM>
hipError_t launch_tiled(hipStream_t st, const uint8_t* aq, const float* as, const uint8_t* bq, const float* bs,
                        uint8_t* hq, float* hs, float* h_tap, uint16_t* out, float* out_tap, float* part, int64_t M,
                        int64_t K, int64_t N, int64_t I, int KS) {
  const int64_t ny = kGateUp ? I / 128 : (N + BNR - 1) / BNR;
  const dim3 grid(static_cast<unsigned>(((M + BM - 1) / BM) * ny * KS));
  hipLaunchKernelGGL((gemm_tiled_kernel<kGateUp, BM>), grid, dim3(kTileWaves * 64), 0, st, aq, as, bq, bs, hq, hs,
                     h_tap, out, out_tap, part, M, K, N, I, KS);
  return hipGetLastError();
}

// Row-tile height: 256 when there are enough row tiles to fill the chip with
// one workgroup per CU, else 128.
bool use_bm256(int64_t M, int64_t col_tiles) { return ((M + 255) / 256) * col_tiles >= 512; }

// K splits of the down GEMM: enough workgroups for about one per CU, each
// split at least 16 K-groups long.
int down_splits(int64_t M, int64_t H, int64_t I) {
  const int64_t tiles = ((M + 127) / 128) * ((H + BNR - 1) / BNR);
  if (use_bm256(M, (H + BNR - 1) / BNR) || tiles >= 256) return 1;
  int64_t ks = (256 + tiles - 1) / tiles;
  const int64_t max_ks = (I / 128) / 16;
  if (ks > max_ks) ks = max_ks;
  return ks < 1 ? 1 : static_cast<int>(ks);
}

}  // namespace

size_t tiled_down_ws_bytes(int64_t M, int64_t H, int64_t I) {
  const int ks = down_splits(M, H, I);
  return ks > 1 ? static_cast<size_t>(ks) * static_cast<size_t>(M) * static_cast<size_t>(H) * 4 : 0;
}

// gate/up row-tile height by the number of rounds of one workgroup per CU:
// a 256-row tile does twice the work of a 128-row one in about 1.8 times
// the time.
bool gateup_bm256(int64_t M, int64_t I) {
  const int64_t cols = I / 128;
  const int64_t r256 = (((M + 255) / 256) * cols + 255) / 256, r128 = (((M + 127) / 128) * cols + 255) / 256;
  return 18 * r256 <= 10 * r128;
}

hipError_t launch_gateup_tiled(hipStream_t st, const uint8_t* xq, const float* xs, const uint8_t* wq,
                               const float* ws, uint8_t* hq, float* hs, float* h_tap, int64_t M, int64_t H,
                               int64_t I) {
  if (gateup_bm256(M, I))
    return launch_tiled<true, 256>(st, xq, xs, wq, ws, hq, hs, h_tap, nullptr, nullptr, nullptr, M, H, 2 * I, I, 1);
  return launch_tiled<true, 128>(st, xq, xs, wq, ws, hq, hs, h_tap, nullptr, nullptr, nullptr, M, H, 2 * I, I, 1);
}

hipError_t launch_down_tiled(hipStream_t st, const uint8_t* hq, const float* hs, const uint8_t* wq, const float* ws,
                             uint16_t* out, float* out_tap, int64_t M, int64_t H, int64_t I, void* ws_buf) {
  if (use_bm256(M, (H + BNR - 1) / BNR))
    return launch_tiled<false, 256>(st, hq, hs, wq, ws, nullptr, nullptr, nullptr, out, out_tap, nullptr, M, I, H, I,
                                    1);
  const int ks = down_splits(M, H, I);
  float* part = static_cast<float*>(ws_buf);
  hipError_t e = launch_tiled<false, 128>(st, hq, hs, wq, ws, nullptr, nullptr, nullptr, out, out_tap, part, M, I, H,
                                          I, ks);
  if (e != hipSuccess || ks == 1) return e;
  const int64_t mn = M * H;
  hipLaunchKernelGGL(split_reduce_kernel, dim3(static_cast<unsigned>((mn / 4 + 255) / 256)), dim3(256), 0, st, part,
                     out, out_tap, mn, ks);
  return hipGetLastError();
}

}  // namespace lacache
