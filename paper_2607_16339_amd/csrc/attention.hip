// First-layer FlashAttention with FACache (Sec. 3.3, FACache; Eqs. 2-6).
//
// Work decomposition. A workgroup of W wavefronts owns 32 query rows per
// wavefront (32 W rows) of one head and streams 64-key tiles of K and V
// through an S-stage LDS ring filled by direct global->LDS copies, so the
// copies of the next S - 1 tiles overlap the MFMAs of the current one.
// Per tile every wavefront
//   * computes S^T = K Q^T with bf16 MFMAs 32x32x16 (Q^T stays in registers;
//     lane (g, r) holds keys 8a + 4g + i of query r, a, i = 0..3);
//   * updates the online-softmax state (m, l) in the log2 domain (Eqs. 2-5,
//     the 1/sqrt(d) scale folded into the exponent); each of the two lanes
//     that share a query row keeps its own partial l, and the two are added
//     whenever the whole state is needed;
//   * accumulates O~^T += V^T P^T (Eq. 6) with P rounded to bf16. The V^T
//     operand is read from the row-major V tile with the transposing LDS
//     read (ds_read_b64_tr_b16): each lane gets 4 consecutive keys of one
//     dimension, matching the key order P^T inherits from the S^T layout.
//
// Key order and FACache. Every query row streams the key blocks inside U
// (ascending), then those overlapping the current block C (ascending). After
// the U blocks the two partial sums l are merged, and in populate mode the
// wavefronts whose 64-row block lies inside U store (m, l, O~) in the cache.
// In resume mode those wavefronts load that state and compute only the C
// blocks (a workgroup with no row in a block overlapping C streams only
// those); the others recompute everything. All three modes therefore run the
// same arithmetic in the same order, and a resume on inputs that changed only
// inside C reproduces plain attention of the new inputs bit for bit.
//
// Scheduling. Work item w = (head, query block) in head-major order, heavy
// query blocks (those overlapping C) first within a head; consecutive work
// items go to the same XCD (workgroups are dealt to the 8 XCDs round-robin),
// so the query blocks of a head share that XCD's L2 copy of its K and V. In
// resume mode, when the grid takes more than one round, each XCD takes its
// heavy items before its light ones.
#include "device.h"
#include "launch.h"

namespace lacache {
namespace {

typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef short s4 __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) s4 lds_s4;

constexpr int kD = 128;                   // head dimension
constexpr int kKB = 64;                   // keys per tile = rows per FACache block
constexpr int kQR = 32;                   // query rows per wavefront
constexpr int kTileBytes = kKB * kD * 2;  // one K or V tile (16 KiB)
constexpr int kStageBytes = 2 * kTileBytes;

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  float* cm;
  float* cl;
  float* co;
  float* lse;
  int64_t N;
  int nqb;      // query blocks (of 32 W rows) per head
  int nkb;      // key blocks (of 64 rows) per head
  int cb0, nc;  // key blocks overlapping C: [cb0, cb0 + nc)
  int qbh0;     // first query block overlapping those key blocks
  int nheavy;   // query blocks overlapping them
  int total;    // workgroups
  int heavy_first;  // resume: each XCD's heavy items before its light ones
  float scale_log2;
};

__device__ __forceinline__ v16f mfma32(bf8 a, bf8 b, v16f c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// two transposing 8-byte LDS reads -> one 8-element operand
__device__ __forceinline__ bf8 read_tr2(const uint8_t* p0, const uint8_t* p1) {
  const s4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)(p0));
  const s4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)(p1));
  return __builtin_bit_cast(bf8, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
}

// two fp32 -> bf16 (round to nearest even) in one v_cvt_pk_bf16_f32
typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16_rne(float lo, float hi) {
  const bf2 v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
  return __builtin_bit_cast(uint32_t, v);
}

// Slot s of an XCD's chunk [lo, lo + n) of the head-major item list, with the
// chunk's heavy items (query blocks j < nh of a head, which stream every key
// block) first and its light ones after. Resume uses this order: a light item
// streams only the C blocks, a heavy one all of them, and heavy items dealt
// out late would leave their long chains to the end of the call. A bijection
// of [lo, lo + n) for 0 < nh < nqb (else the identity).
__device__ __forceinline__ int heavy_first(int lo, int s, int n, int nqb, int nh) {
  if (nh <= 0 || nh >= nqb) return lo + s;
  auto heavy_below = [&](int x) { return (x / nqb) * nh + (x % nqb < nh ? x % nqb : nh); };
  const int h0 = heavy_below(lo), nhc = heavy_below(lo + n) - h0;
  if (s < nhc) {
    const int gh = h0 + s;  // global index among heavy items
    return (gh / nh) * nqb + gh % nh;
  }
  const int nl = nqb - nh;
  const int gl = (lo - h0) + (s - nhc);  // global index among light items
  return (gl / nl) * nqb + nh + gl % nl;
}

// kMode 0: populate, 1: resume, 2: plain attention; W wavefronts, S stages
template <int kMode, int W, int S>
__global__ __launch_bounds__(64 * W, 2) void facache_attention_kernel(AttnArgs a) {
  __shared__ __align__(16) uint8_t smem[S * kStageBytes];
  constexpr int QR = kQR, WR = W * QR;
  constexpr int kPer = 2 * 1024 / (64 * W);  // copies per thread per tile
  const int t = threadIdx.x, lane = t & 63, wave = wave_uniform(t >> 6);
  const int g = lane >> 5, r = lane & 31;

  // work item: consecutive items on one XCD (resume: the chunk's heavy items first)
  const int bid = blockIdx.x, xcd = bid & 7, slot = bid >> 3;
  const int per = a.total >> 3, rem = a.total & 7;
  const int lo = xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per;
  const int w = (kMode == 1 && a.heavy_first) ? heavy_first(lo, slot, xcd < rem ? per + 1 : per, a.nqb, a.nheavy)
                                              : lo + slot;
  const int64_t h = w / a.nqb;
  const int j = w - static_cast<int>(h) * a.nqb;
  const bool heavy = j < a.nheavy;
  const int qb = heavy ? a.qbh0 + j : (j - a.nheavy < a.qbh0 ? j - a.nheavy : j);
  const int64_t row0 = static_cast<int64_t>(qb) * WR + wave * QR;  // this wavefront's first query row
  const bool valid = row0 < a.N;
  const int64_t qblk = row0 / kKB;
  const bool in_u = !(qblk >= a.cb0 && qblk < a.cb0 + a.nc);
  const bool use_cache = kMode == 1 && in_u;  // this wavefront resumes from the cache
  const bool light = kMode == 1 && !heavy;     // ... and so does every wavefront of the workgroup
  const int nU = a.nkb - a.nc;
  const int nlist = light ? a.nc : a.nkb;
  const int64_t hN = h * a.N;
  const uint16_t* kh = a.k + hN * kD;
  const uint16_t* vh = a.v + hN * kD;

  // Q^T operands: query row0 + r, dims 16 kk + 8 g ..
  const int64_t sb = hN + (valid ? row0 + r : 0);  // this lane's query row (state index)
  bf8 qf[8];
#pragma unroll
  for (int kk = 0; kk < 8; ++kk) qf[kk] = *reinterpret_cast<const bf8*>(a.q + sb * kD + 16 * kk + 8 * g);

  float m = -__builtin_inff(), l = 0.0f;
  v16f ot[4];  // O~^T: element 4 b + i of tile dt = dim 32 dt + 8 b + 4 g + i of query r
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) ot[dt][e] = 0.0f;
  if (use_cache && valid) {
    m = a.cm[sb];
    l = g == 0 ? a.cl[sb] : 0.0f;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const float4 c4 = *reinterpret_cast<const float4*>(a.co + sb * kD + 32 * dt + 8 * b + 4 * g);
        ot[dt][4 * b + 0] = c4.x;
        ot[dt][4 * b + 1] = c4.y;
        ot[dt][4 * b + 2] = c4.z;
        ot[dt][4 * b + 3] = c4.w;
      }
  }

  // i-th key block of this workgroup's list
  auto key_block = [&](int i) -> int {
    if (light) return a.cb0 + i;
    return i < nU ? (i < a.cb0 ? i : i + a.nc) : a.cb0 + (i - nU);
  };
  // Copy K and V tiles of list entry i into stage s. LDS slot p (16 bytes)
  // holds key p / 16, 16-byte chunk (p % 16) ^ swizzle(key): K swizzles by
  // key % 16 (conflict-free 16-byte MFMA operand reads), V by 4 (key % 4)
  // (conflict-free transposing reads).
  const uint32_t smem_u32 = lds_u32(smem);
  auto issue = [&](int i, int st) {
    const int64_t kr0 = static_cast<int64_t>(key_block(i)) * kKB;
    const uint32_t kl = smem_u32 + st * kStageBytes, vl = kl + kTileBytes;
#pragma unroll
    for (int n = 0; n < kPer / 2; ++n) {
      const int p0 = n * 64 * W + wave * 64, p = p0 + lane;
      const int key = p >> 4, cp = p & 15;
      dma16(kh + (kr0 + key) * kD + 8 * (cp ^ (key & 15)), kl + 16 * p0);
      dma16(vh + (kr0 + key) * kD + 8 * (cp ^ (4 * (key & 3))), vl + 16 * p0);
    }
  };

  // per-lane LDS offsets
  const int G = lane >> 4, io = lane & 15;
  // V^T operand (transposing read): the lane addresses key 4 (G/2) + io/4 (+ 16 ks + 8 hh)
  // and dims 32 dt + 16 (G%2) + 4 (io%4); chunk swizzle 4 (key % 4) = 4 (io/4)
  const int e_sw = io >> 2;
  const int v_base = (4 * (G >> 1) + (io >> 2)) * 256 + (2 * (G & 1) + ((io & 3) >> 1)) * 16 + 8 * (io & 1);
  const float c = a.scale_log2;

  auto compute = [&](int st) {
    const uint8_t* Kt = smem + st * kStageBytes;
    const uint8_t* Vt = Kt + kTileBytes;
    // S^T = K Q^T
    v16f sa[2];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int e = 0; e < 16; ++e) sa[tt][e] = 0.0f;
    // the two key tiles alternate, so consecutive MFMAs are independent
#pragma unroll
    for (int kk = 0; kk < 8; ++kk)
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
        const int key = 32 * tt + r;
        const bf8 kf = *reinterpret_cast<const bf8*>(Kt + key * 256 + (((2 * kk + g) ^ (key & 15)) << 4));
        sa[tt] = mfma32(kf, qf[kk], sa[tt]);
      }
    // online softmax (Eqs. 2-5) and the P^T operands
    float mx = sa[0][0];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = __builtin_fmaxf(mx, sa[tt][e]);
    mx = __builtin_fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float mn = __builtin_fmaxf(m, mx * c);         // Eq. 2
    const float alpha = __builtin_amdgcn_exp2f(m - mn);  // Eq. 3
    m = mn;
    float ps = 0.0f;
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sa[tt][e], c, -mn));  // Eq. 4
        sa[tt][e] = p;
        ps += p;
      }
    l = alpha * l + ps;  // Eq. 5 (this lane's keys)
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int e = 0; e < 16; ++e) ot[dt][e] *= alpha;
    // step ks covers keys 16 ks .. 16 ks + 15: elements 8 (ks % 2) .. + 7 of S^T tile ks / 2
    bf8 pb[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int tt = ks >> 1, e0 = 8 * (ks & 1);
      const uint4 w4 = make_uint4(pack_bf16_rne(sa[tt][e0 + 0], sa[tt][e0 + 1]),
                                  pack_bf16_rne(sa[tt][e0 + 2], sa[tt][e0 + 3]),
                                  pack_bf16_rne(sa[tt][e0 + 4], sa[tt][e0 + 5]),
                                  pack_bf16_rne(sa[tt][e0 + 6], sa[tt][e0 + 7]));
      pb[ks] = __builtin_bit_cast(bf8, w4);
    }
    // O~^T += V^T P^T (Eq. 6)
    // the four dimension tiles alternate, so consecutive MFMAs are independent
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const uint8_t* vd = Vt + v_base + 64 * (dt ^ e_sw);
        const bf8 vf = read_tr2(vd + (16 * ks) * 256, vd + (16 * ks + 8) * 256);
        ot[dt] = mfma32(vf, pb[ks], ot[dt]);
      }
  };

  // merge the two partial sums of a row into the lane with g == 0
  auto merge_l = [&]() {
    const float tot = l + __shfl_xor(l, 32, 64);
    l = g == 0 ? tot : 0.0f;
  };

#pragma unroll
  for (int i = 0; i < S - 1; ++i)
    if (i < nlist) issue(i, i);
  for (int i = 0; i < nlist; ++i) {
    // this thread's copies of tile i have landed (those of the next S - 2 may be in flight) ...
    if (i + S - 2 < nlist)
      wait_vm<(S - 2) * kPer>();
    else
      wait_vm<0>();
    bar();  // ... and everyone's have; everyone is done reading the stage refilled next
    if (i + S - 1 < nlist) issue(i + S - 1, (i + S - 1) % S);
    if (valid && !(use_cache && !light && i < nU)) compute(i % S);  // a resuming wavefront skips the U blocks
    if (!light && i == nU - 1) {
      merge_l();
      if (kMode == 0 && in_u && valid) {
        if (g == 0) {
          a.cm[sb] = m;
          a.cl[sb] = l;
        }
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int b = 0; b < 4; ++b)
            *reinterpret_cast<float4*>(a.co + sb * kD + 32 * dt + 8 * b + 4 * g) =
                make_float4(ot[dt][4 * b], ot[dt][4 * b + 1], ot[dt][4 * b + 2], ot[dt][4 * b + 3]);
      }
    }
  }

  if (!valid) return;
  const float lt = l + __shfl_xor(l, 32, 64);
  const float inv = 1.0f / lt;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int b = 0; b < 4; ++b)
      *reinterpret_cast<uint2*>(a.o + sb * kD + 32 * dt + 8 * b + 4 * g) =
          make_uint2(pack_bf16_rne(ot[dt][4 * b] * inv, ot[dt][4 * b + 1] * inv),
                     pack_bf16_rne(ot[dt][4 * b + 2] * inv, ot[dt][4 * b + 3] * inv));
  if (a.lse != nullptr && g == 0) a.lse[sb] = (m + __log2f(lt)) * 0.69314718055994531f;
}

template <int W, int S>
hipError_t launch_ws(hipStream_t st, AttnArgs a, int64_t heads, int mode) {
  constexpr int WR = W * kQR;
  a.nqb = static_cast<int>((a.N + WR - 1) / WR);
  a.qbh0 = a.nc > 0 ? a.cb0 * kKB / WR : 0;
  a.nheavy = a.nc > 0 ? static_cast<int>(((a.cb0 + a.nc) * int64_t(kKB) - 1) / WR) - a.qbh0 + 1 : 0;
  a.total = static_cast<int>(heads * a.nqb);
  // heavy items first only when the grid takes more than one round (two
  // workgroups per CU): in a single round every item starts at once and the
  // order only decides which items share a CU
  a.heavy_first = a.total > 2 * device_cu_count() ? 1 : 0;
  const dim3 grid(static_cast<unsigned>(a.total)), block(64 * W);
  if (mode == 0)
    hipLaunchKernelGGL((facache_attention_kernel<0, W, S>), grid, block, 0, st, a);
  else if (mode == 1)
    hipLaunchKernelGGL((facache_attention_kernel<1, W, S>), grid, block, 0, st, a);
  else
    hipLaunchKernelGGL((facache_attention_kernel<2, W, S>), grid, block, 0, st, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_facache_attention(hipStream_t st, const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                    uint16_t* o, float* cm, float* cl, float* co, float* lse, int64_t heads, int64_t N,
                                    int64_t c0, int64_t c1, int mode) {
  AttnArgs a{};
  a.q = q;
  a.k = k;
  a.v = v;
  a.o = o;
  a.cm = cm;
  a.cl = cl;
  a.co = co;
  a.lse = lse;
  a.N = N;
  a.nkb = static_cast<int>(N / kKB);
  if (c0 < c1) {
    a.cb0 = static_cast<int>(c0 / kKB);
    a.nc = static_cast<int>((c1 + kKB - 1) / kKB) - a.cb0;
  }
  a.scale_log2 = 1.4426950408889634f / 11.313708498984761f;  // log2(e) / sqrt(128)
  return launch_ws<4, 2>(st, a, heads, mode);
}

}  // namespace lacache
