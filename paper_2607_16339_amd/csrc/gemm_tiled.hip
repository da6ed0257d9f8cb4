// Tiled FP8 MFMA GEMMs with per-group dequantization (Sec. 3.4):
//   gate/up: x[M x H] . Wgu[2I x H]^T, fused SwiGLU and 1x128 re-quantization
//   down:    h[M x I] . Wd[H x I]^T -> bf16
//
// Work items are BM-row x 256-weight-row output tiles (times the K splits of
// the down GEMM). The grid is persistent: one workgroup per CU walks the items
// b, b + G, b + 2G, ... (G workgroups), and its copy ring runs straight across
// item boundaries, so the first K-groups of the next tile are already in LDS
// when a tile's epilogue ends and no workgroup launch or pipeline refill
// separates two tiles.
//
// A workgroup has 8 wavefronts; wavefront (wm, wn) owns 64 activation rows x
// WC weight rows (4 x NJ sub-tiles of 16 x 16). K is walked one 128-wide group
// at a time:
//   * the group's fp8 tiles (A: BM x 128 B, B: 256 x 128 B), the BM
//     activation scales and the tile's two weight-block scales go global ->
//     LDS with direct-to-LDS copies into a ring of stages, issued S - 1 groups
//     ahead, so no registers hold staging data;
//   * every 16x16 sub-tile gets one 16x16x128 FP8 MFMA (exactly one K-group)
//     whose fp32 result is added to the accumulator times
//     RN32(x_scale[row] * w_scale[block]): four VALU FMAs per MFMA, issued two
//     MFMAs later so that they find the result finished while the matrix core
//     works on the next ones.
// The MFMA takes the weight rows as its first operand, so a lane's four
// results are four consecutive output columns of one activation row: the
// epilogues pack e4m3 codes and bf16 values within a lane, and a row's max
// over the columns needs only two cross-lane steps.
//
// For gate/up the tile's 256 weight rows are the 128 gate rows and the 128
// matching up rows of one h-group; a wavefront's slabs are WC/2 gate rows and
// the WC/2 matching up rows, so SwiGLU pairs values held by one lane, and the
// row amax over the 128-wide h-group meets in LDS across the wavefronts of a
// row band. h never reaches memory.
#include <atomic>
#include <type_traits>

#include "device.h"
#include "launch.h"

namespace lacache {
namespace {

constexpr int BNR = 256;  // weight rows per tile

// LDS tiles are [rows][128 bytes]; the eight 16-byte chunks of a row are
// permuted by an xor with (row / 2) mod 8, which spreads the 16 rows of an
// MFMA operand read over the banks.
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

// One LDS stage: A tile, B tile, BM activation scales, the two weight-block
// scales of the K-group (slots BM and BM + 1 of a 64-slot region written by
// one copy instruction), and 64 spare slots for duplicate scale copies.
template <int BM>
struct Stage {
  uint8_t a[BM * 128];
  uint8_t b[BNR * 128];
  alignas(16) float xs[BM + 128];
};

// A work item: output tile (row tile, column tile) and its K range.
struct Item {
  int m0;   // first activation row
  int col;  // gate/up: h-group; down: 256-column tile
  int kb0, kb1;
  int split;
};

// Item w of R x C tiles x KS splits (R C KS < 2^31). The splits count as
// extra row tiles (split-major), so the XCD-grouped order of xcd_grouped_tile
// (here in 32-bit arithmetic) keeps items that share an operand (the same K
// range of the same rows or columns) on one XCD.
__device__ __forceinline__ Item item_at(int w, int R, int C, int KS, int KB, int BM) {
  const int RV = R * KS, T = RV * C;
  const int x = w % static_cast<int>(kXcds), slot = w / static_cast<int>(kXcds);
  const int per = T / static_cast<int>(kXcds), rem = T % static_cast<int>(kXcds);
  const int tt = (x < rem ? x * (per + 1) : rem * (per + 1) + (x - rem) * per) + slot;
  const int gsz = static_cast<int>(kTileGroupRows) * C;
  const int g = tt / gsz;
  const int first = g * static_cast<int>(kTileGroupRows);
  const int rows = RV - first < static_cast<int>(kTileGroupRows) ? RV - first : static_cast<int>(kTileGroupRows);
  const int wi = tt - g * gsz;
  const int vr = first + wi % rows;
  Item it;
  it.col = wi / rows;
  it.split = vr / R;
  it.m0 = (vr - it.split * R) * BM;
  it.kb0 = it.split * KB / KS;
  it.kb1 = (it.split + 1) * KB / KS;
  return it;
}

}  // namespace

constexpr int kTileWaves = 8;

template <bool kGateUp, int BM>
__global__ __launch_bounds__(kTileWaves * 64) void gemm_tiled_kernel(
    const uint8_t* __restrict__ aq, const float* __restrict__ as,  // [M x K] codes, [K/128 x M] scales
    const uint8_t* __restrict__ bq, const float* __restrict__ bs,  // [N x K] codes, [N/128 x K/128] scales
    uint8_t* __restrict__ hq, float* __restrict__ hs, float* __restrict__ h_tap,
    uint16_t* __restrict__ out, float* __restrict__ out_tap, float* __restrict__ part,
    const float* __restrict__ col_s, int64_t M, int64_t K, int64_t N, int64_t I, int KS, int W) {
  static_assert(BM == 128 || BM == 256, "BM must be 128 or 256");
  constexpr int NW = kTileWaves;
  constexpr int WC = BM == 256 ? 128 : 64;  // weight rows (output columns) per wavefront
  constexpr int NCW = BNR / WC;             // wavefronts along the weight rows
  constexpr int NJ = WC / 16;               // 16-wide column slabs per wavefront
  // LDS ring: 3 stages for BM = 128 (3 x 49.9 KB), 2 for BM = 256 (2 x 66.8 KB)
  constexpr int S = BM == 128 ? 3 : 2;
  __shared__ Stage<BM> stg[S];
  __shared__ float sRed[NCW][BM];

  const int t = threadIdx.x, lane = t & 63;
  // wavefront index made visibly uniform: LDS bases and item fields go scalar
  const int wave = wave_uniform(t >> 6);
  const int wm = wave / NCW, wn = wave % NCW;
  const int q = lane >> 4, lr = lane & 15;
  const int KB = static_cast<int>(K / 128);
  const int R = static_cast<int>((M + BM - 1) / BM);
  const int C = static_cast<int>(kGateUp ? I / 128 : (N + BNR - 1) / BNR);
  const int G = static_cast<int>(gridDim.x);

  constexpr int kCopyWaves = 4;

  // The copy wavefronts and the others run the same stream as two instances
  // of one loop: only the copy wavefronts' instance holds the copy cursor
  // (item, K-group, per-lane offsets) and issues the copies, so the other
  // wavefronts spend neither instructions nor registers on it.
  auto run = [&](auto copy_tag) {
    constexpr bool kCopy = decltype(copy_tag)::value;
    // ---- direct-to-LDS copy plan. Only the first kCopyWaves wavefronts (one
    // per SIMD) copy: a wavefront stalls while the memory pipeline takes its
    // copy instructions, and the other wavefront of its SIMD keeps the matrix
    // core busy meanwhile (all eight copying at once left it idle). A copy
    // instruction fills 64 consecutive 16-byte LDS slots (8 tile rows); lane l
    // fills slot l, i.e. row 8g + l/8, physical chunk l%8, so it fetches logical
    // chunk (l%8) ^ swz(row) of that row. Rows past M (or N) fetch a clamped
    // row; their results are never stored. Scales: each copy wavefront copies
    // the activation scales of rows 64 (w mod BM/64) .. + 63 (one float per
    // lane; copies beyond the first go to the spare slots) and the two
    // weight-block scales (lane 0 the first block, the others the second).
    constexpr int kAInst = BM / 8 / kCopyWaves;  // per copy wavefront
    constexpr int kBInst = BNR / 8 / kCopyWaves;
    constexpr int kPer = kAInst + kBInst + 2;  // copies per copy wavefront per K-group
    const int xband = wave % (BM / 64);
    const int xs_dst = wave < BM / 64 ? wave * 64 : BM + 64;

    // issue cursor: the item whose K-groups are being copied
    int iw = blockIdx.x, ikb = 0, ikb1 = 0;
    const uint8_t* a_base = aq;
    const uint8_t* b_base = bq;
    const uint8_t* b_base_hi = bq;
    const float* x_base = as;  // activation scales of the tile's rows (wave-uniform)
    uint32_t x_off = 0;        // ... this lane's byte offset (stride M floats per K-group)
    uint32_t w_off = 0;        // this lane's weight-block scale row, as a byte offset into bs
    uint32_t a_off[kCopy ? kAInst : 1], b_off[kCopy ? kBInst : 1];
    auto enter = [&](int w) {
      const Item it = item_at(w, R, C, KS, KB, BM);
      ikb = it.kb0;
      ikb1 = it.kb1;
      a_base = aq + static_cast<int64_t>(it.m0) * K;
      const int alim = static_cast<int>(M) - 1 - it.m0;  // last valid row of the tile
#pragma unroll
      for (int u = 0; u < (kCopy ? kAInst : 0); ++u) {
        const int row = (wave * kAInst + u) * 8 + (lane >> 3);
        const int r = row < alim ? row : alim;
        a_off[u] = static_cast<uint32_t>(r) * static_cast<uint32_t>(K) + ((lane & 7) ^ swz(row)) * 16;
      }
      // gate/up: tile rows 0..127 come from the gate block, 128..255 from the up
      // block (base b_base_hi); down: one contiguous 256-row block
      const int n0 = kGateUp ? 0 : it.col * BNR;
      const int blim = kGateUp ? BNR : static_cast<int>(N) - 1 - n0;
      b_base = kGateUp ? bq + static_cast<int64_t>(it.col) * 128 * K : bq + static_cast<int64_t>(n0) * K;
      b_base_hi = kGateUp ? bq + (I + static_cast<int64_t>(it.col) * 128 - 128) * K : b_base;
      // (weights in the tile layout of wtile_off: the slab bases above are the
      // same as row-major, the offsets within and the K-group step are not)
#pragma unroll
      for (int u = 0; u < (kCopy ? kBInst : 0); ++u) {
        const int row = (wave * kBInst + u) * 8 + (lane >> 3);
        const int r = row < blim ? row : blim;
        b_off[u] = static_cast<uint32_t>(wtile_off(r, ((lane & 7) ^ swz(row)) * 16, K));
      }
      {
        const int row = xband * 64 + lane;
        x_base = as + it.m0;
        x_off = static_cast<uint32_t>(row < alim ? row : alim) * 4u;
        // gate/up: {gate block, up block}; down: {block of columns n0.., the next
        // one (or the same past N)}
        const int r0 = kGateUp ? it.col : n0 / 128;
        const int r1 = kGateUp ? static_cast<int>(I / 128) + it.col : (n0 + 128 < N ? n0 / 128 + 1 : r0);
        w_off = static_cast<uint32_t>((lane == 0 ? r0 : r1) * KB) * 4u;
      }
    };
    // Copies of K-group kb of the cursor's item into stage dst (asynchronous).
    auto issue_group = [&](int kb, Stage<BM>* dst) {
      const int64_t ko = static_cast<int64_t>(kb) * 128;
      const int la = static_cast<int>(lds_u32(dst->a)), lb = static_cast<int>(lds_u32(dst->b));
#pragma unroll
      for (int u = 0; u < (kCopy ? kAInst : 0); ++u) dma16s(a_base + ko, a_off[u], wave_uniform(la + (wave * kAInst + u) * 1024));
#pragma unroll
      for (int u = 0; u < (kCopy ? kBInst : 0); ++u) {
        const uint8_t* base = (kGateUp && (wave * kBInst + u) * 8 >= 128) ? b_base_hi : b_base;
        dma16s(base + ko * 16, b_off[u], wave_uniform(lb + (wave * kBInst + u) * 1024));
      }
      const int lx = static_cast<int>(lds_u32(dst->xs));
      dma4s(x_base + static_cast<int64_t>(kb) * M, x_off, wave_uniform(lx + xs_dst * 4));
      dma4s(bs + kb, w_off, wave_uniform(lx + BM * 4));
    };
    // The next K-group in the workgroup's sequence. Past the last one the last
    // group is copied again into the idle stage (never read), so every step
    // waits for the same count.
    auto issue_next = [&](Stage<BM>* dst) {
      issue_group(ikb < ikb1 ? ikb : ikb1 - 1, dst);
      if (ikb < ikb1 && ++ikb == ikb1 && iw + G < W) {
        iw += G;
        enter(iw);
      }
    };

    float acc[4][NJ][4];

    // Multiplies the K-group in stage cur into acc.
    auto compute = [&](const Stage<BM>* cur) {
      auto brow = [&](int j) {
        return kGateUp ? (j < NJ / 2 ? (WC / 2) * wn + 16 * j : 128 + (WC / 2) * wn + 16 * (j - NJ / 2)) : WC * wn + 16 * j;
      };
      // Every LDS read the first MFMAs and FMAs need is issued up front, in the
      // order they are needed (LDS reads complete in order): the first B slab,
      // the scales, then the four A slabs. MFMA i waits only for its own
      // operands, and the scale products are formed after MFMA 1, when the
      // first FMAs need them, instead of holding MFMA 0 back by a round trip.
      v8i bb[2];
      bb[0] = load_frag(cur->b, brow(0) + lr, q);
      __builtin_amdgcn_sched_barrier(0);
      float xv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) xv[i] = cur->xs[64 * wm + 16 * i + lr];
      // gate/up: slabs 0..NJ/2-1 are gate rows (block scale in slot BM), the
      // rest the matching up rows (slot BM + 1); down: the wave's columns lie in
      // one block, slot BM + (WC wn) / 128
      const float w0 = cur->xs[BM + (kGateUp ? 0 : (WC * wn) / 128)];
      const float w1 = cur->xs[BM + 1];
      __builtin_amdgcn_sched_barrier(0);
      v8i af[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = load_frag(cur->a, 64 * wm + 16 * i + lr, q);
      __builtin_amdgcn_sched_barrier(0);
      float sc[kGateUp ? 2 : 1][4];  // RN32(x_scale * w_scale) of this lane's row
      // Software pipeline over the 4 NJ sub-tiles s = 4 j + i: MFMA s, then the
      // scale FMAs of MFMA s - 2; the B operand of slab j + 1 is read while slab
      // j multiplies.
      v4f pr[3];
#pragma unroll
      for (int s = 0; s < 4 * NJ; ++s) {
        const int j = s >> 2, i = s & 3;
        if (i == 0 && j < NJ - 1) bb[(j + 1) & 1] = load_frag(cur->b, brow(j + 1) + lr, q);
        const v4f zero = {0.0f, 0.0f, 0.0f, 0.0f};
        pr[s % 3] = mfma_fp8_16x16x128(bb[j & 1], af[i], zero);
        // keep MFMA s ahead of the FMAs below: they read a result two MFMAs
        // old, so they neither wait for the matrix core nor delay the next MFMA
        __builtin_amdgcn_sched_barrier(0);
        if (s == 1) {
#pragma unroll
          for (int i2 = 0; i2 < 4; ++i2) {
            sc[0][i2] = xv[i2] * w0;
            if (kGateUp) sc[kGateUp ? 1 : 0][i2] = xv[i2] * w1;
          }
        }
        if (s >= 2) {
          const int ps = s - 2;
          const int blk = (kGateUp && (ps >> 2) >= NJ / 2) ? 1 : 0;
#pragma unroll
          for (int r = 0; r < 4; ++r)
            acc[ps & 3][ps >> 2][r] = __builtin_fmaf(pr[ps % 3][r], sc[blk][ps & 3], acc[ps & 3][ps >> 2][r]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int ps = 4 * NJ - 2; ps < 4 * NJ; ++ps)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          acc[ps & 3][ps >> 2][r] = __builtin_fmaf(pr[ps % 3][r], sc[kGateUp ? 1 : 0][ps & 3], acc[ps & 3][ps >> 2][r]);
    };

    // ---- the stream: S - 1 K-groups ahead of the multiply, across items
    if (kCopy) {
      enter(iw);
#pragma unroll
      for (int s = 0; s < S - 1; ++s) issue_next(&stg[s]);
    }
    int cur = 0;  // stage of the K-group being multiplied

    for (int w = blockIdx.x; w < W; w += G) {
      const Item it = item_at(w, R, C, KS, KB, BM);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[i][j][r] = 0.0f;

      for (int kb = it.kb0; kb < it.kb1; ++kb) {
        // a copy wave's copies of the group have landed (later ones may still
        // fly; loads retire in issue order, so epilogue stores in between only
        // make the wait longer) ...
        if (kCopy)
          wait_vm_lds<(S - 2) * kPer>();
        else
          wait_lds();
        bar();  // ... and every wave's; and the stage of the previous group is read by no one
        if (kCopy) issue_next(&stg[cur == 0 ? S - 1 : cur - 1]);  // into the stage freed by the previous group
        compute(&stg[cur]);
        cur = cur + 1 == S ? 0 : cur + 1;
      }

      if (col_s != nullptr) {
        // per-channel weight scales: output column n times col_s[n]
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const int64_t n = kGateUp ? (j < NJ / 2 ? 0 : I) + static_cast<int64_t>(it.col) * 128 + (WC / 2) * wn +
                                          16 * (j < NJ / 2 ? j : j - NJ / 2) + 4 * q
                                    : static_cast<int64_t>(it.col) * BNR + WC * wn + 16 * j + 4 * q;
          const float4 cs = (kGateUp || n < N) ? *reinterpret_cast<const float4*>(col_s + n) : make_float4(0, 0, 0, 0);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            acc[i][j][0] *= cs.x;
            acc[i][j][1] *= cs.y;
            acc[i][j][2] *= cs.z;
            acc[i][j][3] *= cs.w;
          }
        }
      }
      if (kGateUp) {
        // ---- SwiGLU: h = SiLU(g) * u; lanes hold matching gate (j) and up
        // (j + NJ/2) values; h replaces g in acc
        float am[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float a = 0.0f;
#pragma unroll
          for (int j = 0; j < NJ / 2; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float v = swiglu_fast(acc[i][j][r], acc[i][j + NJ / 2][r]);
              acc[i][j][r] = v;
              a = __builtin_fmaxf(a, __builtin_fabsf(v));
            }
          // over the four lanes that hold the row's other columns
          a = __builtin_fmaxf(a, __shfl_xor(a, 16, 64));
          a = __builtin_fmaxf(a, __shfl_xor(a, 32, 64));
          am[i] = a;
        }
        if (q == 0) {
#pragma unroll
          for (int i = 0; i < 4; ++i) sRed[wn][64 * wm + 16 * i + lr] = am[i];
        }
        wait_lds();
        bar();  // the row amax of every wavefront of the band is in LDS
        // ---- 1x128 quantization of each row's h-group (without hq: h only)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (hq == nullptr) {
            const int64_t grow = static_cast<int64_t>(it.m0) + 64 * wm + 16 * i + lr;
            if (grow < M) {
#pragma unroll
              for (int j = 0; j < NJ / 2; ++j)
                *reinterpret_cast<float4*>(h_tap + grow * I + static_cast<int64_t>(it.col) * 128 + (WC / 2) * wn +
                                           16 * j + 4 * q) =
                    make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
            }
            continue;
          }
          const int row = 64 * wm + 16 * i + lr;
          const int64_t grow = static_cast<int64_t>(it.m0) + row;
          float amax = sRed[0][row];
#pragma unroll
          for (int c = 1; c < NCW; ++c) amax = __builtin_fmaxf(amax, sRed[c][row]);
          const float s = amax / kE4M3Max;
          const FastQuant fq = fast_quant(s);
          const bool fast = scale_is_fast(s);
          const bool ok = grow < M;
#pragma unroll
          for (int j = 0; j < NJ / 2; ++j) {
            // E(RN32(h / s)) by the bracket where it decides, else by the division
            uint32_t code;
            const bool agree = enc4_bracket(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3], fq, code);
            if (s == 0.0f)
              code = 0u;
            else if (!(fast && agree))
              code = enc4_e4m3(qdiv(acc[i][j][0], s), qdiv(acc[i][j][1], s), qdiv(acc[i][j][2], s),
                               qdiv(acc[i][j][3], s));
            const int64_t col = static_cast<int64_t>(it.col) * 128 + (WC / 2) * wn + 16 * j + 4 * q;
            if (ok) {
              *reinterpret_cast<uint32_t*>(hq + grow * I + col) = code;
              if (h_tap != nullptr)
                *reinterpret_cast<float4*>(h_tap + grow * I + col) =
                    make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
            }
          }
          if (wn == 0 && q == 0 && ok) hs[it.col * M + grow] = s;
        }
      } else {
        // ---- bf16 output (nearest-even from the fp32 accumulator), or the fp32
        // partial sum of this K split
        const int64_t n0 = static_cast<int64_t>(it.col) * BNR;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int64_t row = static_cast<int64_t>(it.m0) + 64 * wm + 16 * i + lr;
          if (row >= M) continue;
#pragma unroll
          for (int j = 0; j < NJ; ++j) {
            const int64_t col = n0 + WC * wn + 16 * j + 4 * q;
            if (col >= N) continue;
            if (KS > 1) {
              *reinterpret_cast<float4*>(part + (it.split * M + row) * N + col) =
                  make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
            } else {
              *reinterpret_cast<uint2*>(out + row * N + col) =
                  make_uint2(pack_bf16x2(acc[i][j][0], acc[i][j][1]), pack_bf16x2(acc[i][j][2], acc[i][j][3]));
              if (out_tap != nullptr)
                *reinterpret_cast<float4*>(out_tap + row * N + col) =
                    make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
            }
          }
        }
      }
    }
    if (kCopy) wait_vm<0>();  // the trailing repeat copies
  };
  if (wave < kCopyWaves)
    run(std::true_type{});
  else
    run(std::false_type{});
}

// Compute units of the current device (the persistent grid's size), cached
// per device; 256 when the runtime cannot tell.
int device_cu_count() {
  static std::atomic<int> cached[64];  // 0: not looked up yet (zero-initialized)
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

template __global__ void gemm_tiled_kernel<true, 256>(const uint8_t*, const float*, const uint8_t*, const float*,
                                                     uint8_t*, float*, float*, uint16_t*, float*, float*, const float*, int64_t,
                                                     int64_t, int64_t, int64_t, int, int);
template __global__ void gemm_tiled_kernel<true, 128>(const uint8_t*, const float*, const uint8_t*, const float*,
                                                     uint8_t*, float*, float*, uint16_t*, float*, float*, const float*, int64_t,
                                                     int64_t, int64_t, int64_t, int, int);
template __global__ void gemm_tiled_kernel<false, 256>(const uint8_t*, const float*, const uint8_t*, const float*,
                                                      uint8_t*, float*, float*, uint16_t*, float*, float*, const float*, int64_t,
                                                      int64_t, int64_t, int64_t, int, int);
template __global__ void gemm_tiled_kernel<false, 128>(const uint8_t*, const float*, const uint8_t*, const float*,
                                                      uint8_t*, float*, float*, uint16_t*, float*, float*, const float*, int64_t,
                                                      int64_t, int64_t, int64_t, int, int);

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
                        int64_t K, int64_t N, int64_t I, int KS, const float* col_s) {
  const int64_t ny = kGateUp ? I / 128 : (N + BNR - 1) / BNR;
  const int W = static_cast<int>(((M + BM - 1) / BM) * ny * KS);  // work items (< 2^31 by the size limits)
  // one workgroup per CU (the LDS ring allows no more)
  const int G = W < device_cu_count() ? W : device_cu_count();
  hipLaunchKernelGGL((gemm_tiled_kernel<kGateUp, BM>), dim3(static_cast<unsigned>(G)), dim3(kTileWaves * 64), 0, st,
                     aq, as, bq, bs, hq, hs, h_tap, out, out_tap, part, col_s, M, K, N, I, KS, W);
  return hipGetLastError();
}

// Row-tile height, by rounds of one workgroup per CU: 256-row tiles unless
// 128-row tiles fill no more rounds. A round of 256-row tiles (twice the
// work) takes about 1.4-1.6 times a round of 128-row tiles over the same K,
// so fewer rounds of the larger tile win whenever the smaller one needs more;
// with equal rounds the smaller tile leaves fewer CUs idle (and the down GEMM
// then splits K when it has fewer tiles than CUs).
bool use_bm256(int64_t M, int64_t col_tiles) {
  const int64_t cus = device_cu_count();
  const int64_t r256 = (((M + 255) / 256) * col_tiles + cus - 1) / cus;
  const int64_t r128 = (((M + 127) / 128) * col_tiles + cus - 1) / cus;
  return r128 > r256;
}

// K splits of the down GEMM: as many as fit in one round of one workgroup
// per CU, each split at least 16 K-groups long. Rounding up instead spills a
// few items into a second round: at H = 4096, I = 12288, M = 700 (96 tiles)
// 3 splits took 75.5 us against 56.8 us for 2.
int down_splits(int64_t M, int64_t H, int64_t I) {
  const int64_t tiles = ((M + 127) / 128) * ((H + BNR - 1) / BNR), cus = device_cu_count();
  if (use_bm256(M, (H + BNR - 1) / BNR) || tiles >= cus) return 1;
  int64_t ks = cus / tiles;
  const int64_t max_ks = (I / 128) / 16;
  if (ks > max_ks) ks = max_ks;
  return ks < 1 ? 1 : static_cast<int>(ks);
}

}  // namespace

size_t tiled_down_ws_bytes(int64_t M, int64_t H, int64_t I) {
  const int ks = down_splits(M, H, I);
  return ks > 1 ? static_cast<size_t>(ks) * static_cast<size_t>(M) * static_cast<size_t>(H) * 4 : 0;
}

hipError_t launch_gateup_tiled(hipStream_t st, const uint8_t* xq, const float* xs, const uint8_t* wq,
                               const float* ws, uint8_t* hq, float* hs, float* h_tap, int64_t M, int64_t H,
                               int64_t I, const float* col_s) {
  if (use_bm256(M, I / 128))
    return launch_tiled<true, 256>(st, xq, xs, wq, ws, hq, hs, h_tap, nullptr, nullptr, nullptr, M, H, 2 * I, I, 1,
                                   col_s);
  return launch_tiled<true, 128>(st, xq, xs, wq, ws, hq, hs, h_tap, nullptr, nullptr, nullptr, M, H, 2 * I, I, 1,
                                 col_s);
}

hipError_t launch_down_tiled(hipStream_t st, const uint8_t* hq, const float* hs, const uint8_t* wq, const float* ws,
                             uint16_t* out, float* out_tap, int64_t M, int64_t H, int64_t I, void* ws_buf,
                             const float* col_s) {
  if (use_bm256(M, (H + BNR - 1) / BNR))
    return launch_tiled<false, 256>(st, hq, hs, wq, ws, nullptr, nullptr, nullptr, out, out_tap, nullptr, M, I, H, I,
                                    1, col_s);
  const int ks = down_splits(M, H, I);
  float* part = static_cast<float*>(ws_buf);
  hipError_t e = launch_tiled<false, 128>(st, hq, hs, wq, ws, nullptr, nullptr, nullptr, out, out_tap, part, M, I, H,
                                          I, ks, col_s);
  if (e != hipSuccess || ks == 1) return e;
  const int64_t mn = M * H;
  hipLaunchKernelGGL(split_reduce_kernel, dim3(static_cast<unsigned>((mn / 4 + 255) / 256)), dim3(256), 0, st, part,
                     out, out_tap, mn, ks);
  return hipGetLastError();
}

}  // namespace lacache
