// C ABI of the FP8 FFN library (declared in include/lacache.h): host-side
// argument validation, the library-owned workspace and kernel-path dispatch.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <vector>

#include "lacache.h"
#include "launch.h"

// Workspace of lacache_ffn_fp8_noalloc: a fixed device array that the code
// object holds on every device the library runs on, until the process ends.
// In host code `scratch` names a host-side stand-in, not device memory: only
// the address that hipGetSymbolAddress returns on a device may reach a kernel
// or a copy.
constexpr size_t kNoAllocBytes = size_t(LACACHE_NOALLOC_SCRATCH_BYTES);
static __device__ __align__(256) uint8_t scratch[kNoAllocBytes];

namespace {

using namespace lacache;

constexpr int64_t kGroup = 128;  // the only supported group size (1x128 and 128x128)
constexpr int64_t kMaxH = 16384;
constexpr int64_t kMaxI = 65536;
constexpr int64_t kMaxM = int64_t(1) << 24;
constexpr int64_t kMaxN = 2 * kMaxI;
constexpr int64_t kAttnHeadDim = 128;
constexpr int64_t kAttnBlock = 64;
constexpr int64_t kAttnMaxHeads = 4096;
constexpr int64_t kAttnMaxN = int64_t(1) << 20;

std::atomic<int> g_policy{0};

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Range {
  uintptr_t lo, hi;  // [lo, hi)
};
Range rng(const void* p, size_t bytes) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(p);
  return {a, a + bytes};
}
bool overlap(Range a, Range b) { return a.lo < b.hi && b.lo < a.hi; }

// Outputs must not overlap inputs (or each other).
bool disjoint(std::initializer_list<Range> outs, std::initializer_list<Range> ins) {
  std::vector<Range> o(outs), i(ins);
  for (size_t a = 0; a < o.size(); ++a) {
    if (o[a].hi == o[a].lo) continue;
    for (const Range& b : i)
      if (b.hi != b.lo && overlap(o[a], b)) return false;
    for (size_t b = a + 1; b < o.size(); ++b)
      if (o[b].hi != o[b].lo && overlap(o[a], o[b])) return false;
  }
  return true;
}

int check_group(int group) { return group == kGroup ? LACACHE_OK : LACACHE_ERR_UNSUPPORTED; }

int check_dim(int64_t d, int64_t max) {
  if (d <= 0 || d % kGroup != 0) return LACACHE_ERR_INVALID_ARG;
  if (d > max) return LACACHE_ERR_UNSUPPORTED;
  return LACACHE_OK;
}

int check_m(int64_t M) {
  if (M < 0) return LACACHE_ERR_INVALID_ARG;
  if (M > kMaxM) return LACACHE_ERR_UNSUPPORTED;
  return LACACHE_OK;
}

#define RETURN_IF(x)                  \
  do {                                \
    const int s_ = (x);               \
    if (s_ != LACACHE_OK) return s_;  \
  } while (0)

bool ptrs_ok(std::initializer_list<const void*> ps) {
  for (const void* p : ps)
    if (p == nullptr || !aligned16(p)) return false;
  return true;
}
bool opt_ptr_ok(const void* p) { return p == nullptr || aligned16(p); }

int hip_status(hipError_t e) { return e == hipSuccess ? LACACHE_OK : LACACHE_ERR_HIP; }

// Kernel path for the GEMM stages.
enum class Path { kSkinny, kTiled };
int choose_path(int64_t M, int64_t H, int64_t I, Path* p) {
  const int pol = g_policy.load();
  const bool skinny_ok = skinny_supported(M, H, I) || M == 0;
  if (pol == 1) {
    if (!skinny_ok) return LACACHE_ERR_UNSUPPORTED;
    *p = Path::kSkinny;
  } else if (pol == 2) {
    *p = Path::kTiled;
  } else {
    *p = (M <= kSkinnyMaxM && skinny_ok) ? Path::kSkinny : Path::kTiled;
  }
  return LACACHE_OK;
}

// fp32 scratch of the GEMM stages: the skinny gate/up h (M <= kSkinnyMaxM),
// or the split-K partials of the tiled down GEMM, whichever path runs (both
// are possible at small M: by shape and by the path policy).
size_t scratch_bytes(int64_t M, int64_t H, int64_t I) {
  const size_t sk = M <= kSkinnyMaxM ? skinny_gateup_ws_bytes(M, I) : 0;
  const size_t tl = tiled_down_ws_bytes(M, H, I);
  return sk > tl ? sk : tl;
}

// ---------------------------------------------------------------------------
// Library-owned workspace: one grow-only device buffer per device. A buffer
// that a larger call supersedes is kept (not freed) until
// lacache_release_workspace: calls queued on any stream, and HIP graphs
// captured earlier, may still use it. Growth needs hipMalloc, which a stream
// under capture must not see, so a call that would grow the workspace while
// its stream is being captured returns LACACHE_ERR_CAPTURE instead.
// ---------------------------------------------------------------------------
struct DeviceWs {
  void* ptr = nullptr;
  size_t bytes = 0;
  std::vector<void*> retired;
};
std::mutex g_ws_mu;
std::vector<DeviceWs> g_ws;

// Returns a workspace of at least `bytes` on the current device.
int get_workspace(hipStream_t st, size_t bytes, void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return LACACHE_ERR_HIP;
  std::lock_guard<std::mutex> lk(g_ws_mu);
  if (static_cast<size_t>(dev) >= g_ws.size()) g_ws.resize(dev + 1);
  DeviceWs& w = g_ws[dev];
  if (w.bytes < bytes) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(st, &cs) != hipSuccess) return LACACHE_ERR_HIP;
    if (cs != hipStreamCaptureStatusNone) return LACACHE_ERR_CAPTURE;
    const char* force_fail = std::getenv("LACACHE_TEST_FAIL_ALLOC");
    if (force_fail != nullptr && force_fail[0] == '1') return LACACHE_ERR_ALLOC;
    // grow by at least half, so that a run of slowly growing calls keeps at
    // most about twice the largest size alive
    const size_t want = w.ptr == nullptr ? bytes : (bytes > w.bytes + w.bytes / 2 ? bytes : w.bytes + w.bytes / 2);
    void* p = nullptr;
    if (hipMalloc(&p, want) != hipSuccess) {
      (void)hipGetLastError();
      if (want == bytes || hipMalloc(&p, bytes) != hipSuccess) {
        (void)hipGetLastError();
        return LACACHE_ERR_ALLOC;
      }
      if (w.ptr != nullptr) w.retired.push_back(w.ptr);
      w.ptr = p;
      w.bytes = bytes;
    } else {
      if (w.ptr != nullptr) w.retired.push_back(w.ptr);
      w.ptr = p;
      w.bytes = want;
    }
  }
  *out = w.ptr;
  return LACACHE_OK;
}

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept.
constexpr int kMaxDevices = 64;
std::mutex g_na_mu;
void* g_na_ptr[kMaxDevices] = {};

int noalloc_scratch(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return LACACHE_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return LACACHE_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lk(g_na_mu);
  if (g_na_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) {
      (void)hipGetLastError();
      return LACACHE_ERR_HIP;
    }
    g_na_ptr[dev] = p;
  }
  *out = g_na_ptr[dev];
  return LACACHE_OK;
}

// Workspace layout (every region 256-byte aligned):
//   [scratch: the skinny gate/up h (M <= kSkinnyMaxM) or the split-K partials
//    of the tiled down GEMM, the larger of the two; may be empty]
//   [xq: M x H][xs: H/128 x M fp32][hq: M x I][hs: I/128 x M fp32]
struct FfnWs {
  void* scratch;
  uint8_t* xq;
  float* xs;
  uint8_t* hq;
  float* hs;
  size_t total;
};
FfnWs ffn_layout(void* base, int64_t M, int64_t H, int64_t I) {
  FfnWs w{};
  char* b = static_cast<char*>(base);
  size_t off = 0;
  w.scratch = b;
  off += align256(scratch_bytes(M, H, I));
  w.xq = reinterpret_cast<uint8_t*>(b + off);
  off += align256(static_cast<size_t>(M * H));
  w.xs = reinterpret_cast<float*>(b + off);
  off += align256(static_cast<size_t>(H / kGroup * M) * 4);
  w.hq = reinterpret_cast<uint8_t*>(b + off);
  off += align256(static_cast<size_t>(M * I));
  w.hs = reinterpret_cast<float*>(b + off);
  off += align256(static_cast<size_t>(I / kGroup * M) * 4);
  w.total = off;
  return w;
}

int run_gateup(hipStream_t st, Path path, const uint8_t* xq, const float* xs, const uint8_t* wq, const float* ws,
               uint8_t* hq, float* hs, float* tap, int64_t M, int64_t H, int64_t I, void* skinny_ws) {
  if (path == Path::kSkinny)
    return hip_status(launch_gateup_skinny(st, xq, xs, wq, ws, hq, hs, tap, M, H, I, skinny_ws));
  return hip_status(launch_gateup_tiled(st, xq, xs, wq, ws, hq, hs, tap, M, H, I));
}

int run_down(hipStream_t st, Path path, const uint8_t* hq, const float* hs, const uint8_t* wq, const float* ws,
             uint16_t* out, float* tap, int64_t M, int64_t H, int64_t I, void* scratch) {
  if (path == Path::kSkinny) return hip_status(launch_down_skinny(st, hq, hs, wq, ws, out, tap, M, H, I));
  return hip_status(launch_down_tiled(st, hq, hs, wq, ws, out, tap, M, H, I, scratch));
}

int validate_ffn(const uint16_t* x, const uint16_t* norm_w, const uint8_t* wgu_q, const float* wgu_s,
                 const uint8_t* wd_q, const float* wd_s, uint16_t* out, int64_t M, int64_t H, int64_t I, int group) {
  RETURN_IF(check_group(group));
  RETURN_IF(check_m(M));
  RETURN_IF(check_dim(H, kMaxH));
  RETURN_IF(check_dim(I, kMaxI));
  if (M == 0) return LACACHE_OK;  // nothing to read or write: pointers are not looked at
  if (!ptrs_ok({x, norm_w, wgu_q, wgu_s, wd_q, wd_s, out})) return LACACHE_ERR_INVALID_ARG;
  const size_t mh = static_cast<size_t>(M * H);
  if (!disjoint({rng(out, mh * 2)},
                {rng(x, mh * 2), rng(norm_w, H * 2), rng(wgu_q, 2 * I * H), rng(wgu_s, (2 * I / 128) * (H / 128) * 4),
                 rng(wd_q, H * I), rng(wd_s, (H / 128) * (I / 128) * 4)}))
    return LACACHE_ERR_INVALID_ARG;
  return LACACHE_OK;
}

// y non-null: x = RNE_bf16(x + y) in place first (x is then written).
int ffn_core(hipStream_t st, const uint16_t* x, const uint16_t* y, const uint16_t* norm_w, const uint8_t* wgu_q,
             const float* wgu_s, const uint8_t* wd_q, const float* wd_s, uint16_t* out, int64_t M, int64_t H,
             int64_t I, Path path, const FfnWs& w) {
  if (launch_rmsnorm_quant(st, const_cast<uint16_t*>(x), norm_w, w.xq, w.xs, M, H, y) != hipSuccess)
    return LACACHE_ERR_HIP;
  RETURN_IF(run_gateup(st, path, w.xq, w.xs, wgu_q, wgu_s, w.hq, w.hs, nullptr, M, H, I, w.scratch));
  return run_down(st, path, w.hq, w.hs, wd_q, wd_s, out, nullptr, M, H, I, w.scratch);
}

}  // namespace

extern "C" {

int lacache_quant_weights(void* stream, const uint16_t* w, uint8_t* w_q, float* w_s, int64_t N, int64_t K,
                          int group) {
  RETURN_IF(check_group(group));
  RETURN_IF(check_dim(N, kMaxN));
  RETURN_IF(check_dim(K, kMaxN));
  if (!ptrs_ok({w, w_q, w_s})) return LACACHE_ERR_INVALID_ARG;
  if (!disjoint({rng(w_q, N * K), rng(w_s, (N / 128) * (K / 128) * 4)}, {rng(w, N * K * 2)}))
    return LACACHE_ERR_INVALID_ARG;
  return hip_status(launch_quant_weights(static_cast<hipStream_t>(stream), w, w_q, w_s, N, K));
}

int lacache_pack_weights(void* stream, const uint8_t* w_q_rowmajor, uint8_t* w_q, int64_t N, int64_t K) {
  RETURN_IF(check_dim(N, kMaxN));
  RETURN_IF(check_dim(K, kMaxN));
  if (!ptrs_ok({w_q_rowmajor, w_q})) return LACACHE_ERR_INVALID_ARG;
  if (overlap(rng(w_q, N * K), rng(w_q_rowmajor, N * K))) return LACACHE_ERR_INVALID_ARG;
  return hip_status(launch_pack_weights(static_cast<hipStream_t>(stream), w_q_rowmajor, w_q, N, K));
}

int lacache_rmsnorm_quant(void* stream, const uint16_t* x, const uint16_t* norm_w, uint8_t* xq, float* xs,
                          int64_t M, int64_t H, int group) {
  RETURN_IF(check_group(group));
  RETURN_IF(check_m(M));
  RETURN_IF(check_dim(H, kMaxH));
  if (M == 0) return LACACHE_OK;
  if (!ptrs_ok({x, norm_w, xq, xs})) return LACACHE_ERR_INVALID_ARG;
  if (!disjoint({rng(xq, M * H), rng(xs, (H / 128) * M * 4)}, {rng(x, M * H * 2), rng(norm_w, H * 2)}))
    return LACACHE_ERR_INVALID_ARG;
  // (x is only read: no y)
  return hip_status(launch_rmsnorm_quant(static_cast<hipStream_t>(stream), const_cast<uint16_t*>(x), norm_w, xq, xs,
                                         M, H));
}

int lacache_add_rmsnorm_quant(void* stream, uint16_t* resid, const uint16_t* y, const uint16_t* norm_w, uint8_t* xq,
                              float* xs, int64_t M, int64_t H, int group) {
  RETURN_IF(check_group(group));
  RETURN_IF(check_m(M));
  RETURN_IF(check_dim(H, kMaxH));
  if (M == 0) return LACACHE_OK;
  if (!ptrs_ok({resid, y, norm_w, xq, xs})) return LACACHE_ERR_INVALID_ARG;
  const size_t mh = static_cast<size_t>(M * H);
  if (!disjoint({rng(resid, mh * 2), rng(xq, mh), rng(xs, (H / 128) * M * 4)},
                {rng(y, mh * 2), rng(norm_w, H * 2)}) ||
      !disjoint({rng(resid, mh * 2)}, {rng(xq, mh), rng(xs, (H / 128) * M * 4)}))
    return LACACHE_ERR_INVALID_ARG;
  return hip_status(launch_rmsnorm_quant(static_cast<hipStream_t>(stream), resid, norm_w, xq, xs, M, H, y));
}

int lacache_gateup_swiglu_quant(void* stream, const uint8_t* xq, const float* xs, const uint8_t* wgu_q,
                                const float* wgu_s, uint8_t* hq, float* hs, float* h_tap, int64_t M, int64_t H,
                                int64_t I, int group) {
  RETURN_IF(check_group(group));
  RETURN_IF(check_m(M));
  RETURN_IF(check_dim(H, kMaxH));
  RETURN_IF(check_dim(I, kMaxI));
  Path path;
  RETURN_IF(choose_path(M, H, I, &path));
  if (M == 0) return LACACHE_OK;
  if (!ptrs_ok({xq, xs, wgu_q, wgu_s, hq, hs}) || !opt_ptr_ok(h_tap)) return LACACHE_ERR_INVALID_ARG;
  if (!disjoint({rng(hq, M * I), rng(hs, (I / 128) * M * 4), rng(h_tap, h_tap ? M * I * 4 : 0)},
                {rng(xq, M * H), rng(xs, (H / 128) * M * 4), rng(wgu_q, 2 * I * H),
                 rng(wgu_s, (2 * I / 128) * (H / 128) * 4)}))
    return LACACHE_ERR_INVALID_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  void* skinny = nullptr;
  if (path == Path::kSkinny) RETURN_IF(get_workspace(st, skinny_gateup_ws_bytes(M, I), &skinny));
  return run_gateup(st, path, xq, xs, wgu_q, wgu_s, hq, hs, h_tap, M, H, I, skinny);
}

int lacache_down_proj(void* stream, const uint8_t* hq, const float* hs, const uint8_t* wd_q, const float* wd_s,
                      uint16_t* out, float* out_tap, int64_t M, int64_t H, int64_t I, int group) {
  RETURN_IF(check_group(group));
  RETURN_IF(check_m(M));
  RETURN_IF(check_dim(H, kMaxH));
  RETURN_IF(check_dim(I, kMaxI));
  Path path;
  RETURN_IF(choose_path(M, H, I, &path));
  if (M == 0) return LACACHE_OK;
  if (!ptrs_ok({hq, hs, wd_q, wd_s, out}) || !opt_ptr_ok(out_tap)) return LACACHE_ERR_INVALID_ARG;
  if (!disjoint({rng(out, M * H * 2), rng(out_tap, out_tap ? M * H * 4 : 0)},
                {rng(hq, M * I), rng(hs, (I / 128) * M * 4), rng(wd_q, H * I), rng(wd_s, (H / 128) * (I / 128) * 4)}))
    return LACACHE_ERR_INVALID_ARG;
  void* scratch = nullptr;
  if (path == Path::kTiled && tiled_down_ws_bytes(M, H, I) > 0)
    RETURN_IF(get_workspace(static_cast<hipStream_t>(stream), tiled_down_ws_bytes(M, H, I), &scratch));
  return run_down(static_cast<hipStream_t>(stream), path, hq, hs, wd_q, wd_s, out, out_tap, M, H, I, scratch);
}

size_t lacache_ffn_workspace_bytes(int64_t M, int64_t H, int64_t I, int group) {
  if (check_group(group) != LACACHE_OK || check_m(M) != LACACHE_OK || check_dim(H, kMaxH) != LACACHE_OK ||
      check_dim(I, kMaxI) != LACACHE_OK)
    return 0;
  return ffn_layout(nullptr, M, H, I).total;
}

int lacache_ffn_fp8(void* stream, const uint16_t* x, const uint16_t* norm_w, const uint8_t* wgu_q,
                    const float* wgu_s, const uint8_t* wd_q, const float* wd_s, uint16_t* out, int64_t M, int64_t H,
                    int64_t I, int group) {
  RETURN_IF(validate_ffn(x, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, M, H, I, group));
  Path path;
  RETURN_IF(choose_path(M, H, I, &path));
  if (M == 0) return LACACHE_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  void* base = nullptr;
  RETURN_IF(get_workspace(st, ffn_layout(nullptr, M, H, I).total, &base));
  return ffn_core(st, x, nullptr, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, M, H, I, path, ffn_layout(base, M, H, I));
}

int lacache_ffn_fp8_addnorm(void* stream, uint16_t* resid, const uint16_t* y, const uint16_t* norm_w,
                            const uint8_t* wgu_q, const float* wgu_s, const uint8_t* wd_q, const float* wd_s,
                            uint16_t* out, int64_t M, int64_t H, int64_t I, int group) {
  RETURN_IF(validate_ffn(resid, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, M, H, I, group));
  if (M == 0) return LACACHE_OK;
  const size_t mh = static_cast<size_t>(M * H);
  if (!ptrs_ok({y}) || !disjoint({rng(resid, mh * 2), rng(out, mh * 2)},
                                 {rng(y, mh * 2), rng(norm_w, H * 2), rng(wgu_q, 2 * I * H),
                                  rng(wgu_s, (2 * I / 128) * (H / 128) * 4), rng(wd_q, H * I),
                                  rng(wd_s, (H / 128) * (I / 128) * 4)}))
    return LACACHE_ERR_INVALID_ARG;
  Path path;
  RETURN_IF(choose_path(M, H, I, &path));
  hipStream_t st = static_cast<hipStream_t>(stream);
  void* base = nullptr;
  RETURN_IF(get_workspace(st, ffn_layout(nullptr, M, H, I).total, &base));
  return ffn_core(st, resid, y, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, M, H, I, path, ffn_layout(base, M, H, I));
}

int lacache_ffn_fp8_ws(void* stream, const uint16_t* x, const uint16_t* norm_w, const uint8_t* wgu_q,
                       const float* wgu_s, const uint8_t* wd_q, const float* wd_s, uint16_t* out, int64_t M,
                       int64_t H, int64_t I, int group, void* workspace, size_t ws_bytes) {
  RETURN_IF(validate_ffn(x, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, M, H, I, group));
  Path path;
  RETURN_IF(choose_path(M, H, I, &path));
  if (M == 0) return LACACHE_OK;
  const FfnWs lay = ffn_layout(workspace, M, H, I);
  if (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0 || ws_bytes < lay.total)
    return LACACHE_ERR_INVALID_ARG;
  const size_t mh = static_cast<size_t>(M * H);
  if (!disjoint({rng(workspace, lay.total)},
                {rng(x, mh * 2), rng(out, mh * 2), rng(norm_w, H * 2), rng(wgu_q, 2 * I * H),
                 rng(wgu_s, (2 * I / 128) * (H / 128) * 4), rng(wd_q, H * I), rng(wd_s, (H / 128) * (I / 128) * 4)}))
    return LACACHE_ERR_INVALID_ARG;
  return ffn_core(static_cast<hipStream_t>(stream), x, nullptr, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, M, H, I, path,
                  lay);
}

int lacache_ffn_fp8_noalloc(void* stream, const uint16_t* x, const uint16_t* norm_w, const uint8_t* wgu_q,
                            const float* wgu_s, const uint8_t* wd_q, const float* wd_s, uint16_t* out, int64_t M,
                            int64_t H, int64_t I, int group) {
  RETURN_IF(validate_ffn(x, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, M, H, I, group));
  Path path;
  RETURN_IF(choose_path(M, H, I, &path));
  if (M == 0) return LACACHE_OK;
  if (ffn_layout(nullptr, M, H, I).total > kNoAllocBytes) return LACACHE_ERR_UNSUPPORTED;
  void* base = nullptr;
  RETURN_IF(noalloc_scratch(&base));
  // every kernel writes each workspace element it reads first, so nothing in
  // the array needs clearing
  return ffn_core(static_cast<hipStream_t>(stream), x, nullptr, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, M, H, I, path,
                  ffn_layout(base, M, H, I));
}

// ---------------------------------------------------------------------------
// Coarse quantization granularities (per token, per tensor)
// ---------------------------------------------------------------------------

int lacache_quant_weights_g(void* stream, const uint16_t* w, uint8_t* w_q, float* w_s, float* w_row_s, int64_t N,
                            int64_t K, int granularity) {
  if (granularity == LACACHE_GRAN_GROUP) return lacache_quant_weights(stream, w, w_q, w_s, N, K, 128);
  if (granularity != LACACHE_GRAN_TOKEN && granularity != LACACHE_GRAN_TENSOR) return LACACHE_ERR_INVALID_ARG;
  RETURN_IF(check_dim(N, kMaxN));
  RETURN_IF(check_dim(K, kMaxN));
  if (!ptrs_ok({w, w_q, w_s, w_row_s})) return LACACHE_ERR_INVALID_ARG;
  if (!disjoint({rng(w_q, N * K), rng(w_s, (N / 128) * (K / 128) * 4), rng(w_row_s, N * 4)}, {rng(w, N * K * 2)}))
    return LACACHE_ERR_INVALID_ARG;
  return hip_status(launch_quant_weights_rows(static_cast<hipStream_t>(stream), w, w_q, w_s, w_row_s, N, K,
                                              granularity == LACACHE_GRAN_TENSOR));
}

int lacache_rmsnorm_f32(void* stream, const uint16_t* x, const uint16_t* norm_w, float* y, int64_t M, int64_t H) {
  RETURN_IF(check_m(M));
  RETURN_IF(check_dim(H, kMaxH));
  if (M == 0) return LACACHE_OK;
  if (!ptrs_ok({x, norm_w, y})) return LACACHE_ERR_INVALID_ARG;
  if (!disjoint({rng(y, M * H * 4)}, {rng(x, M * H * 2), rng(norm_w, H * 2)})) return LACACHE_ERR_INVALID_ARG;
  return hip_status(launch_rmsnorm_f32(static_cast<hipStream_t>(stream), x, norm_w, y, M, H));
}

int lacache_quant_rows_g(void* stream, const float* v, uint8_t* q, float* s_kgm, float* s_rows, int64_t M, int64_t K,
                         int granularity) {
  if (granularity < LACACHE_GRAN_GROUP || granularity > LACACHE_GRAN_TENSOR) return LACACHE_ERR_INVALID_ARG;
  RETURN_IF(check_m(M));
  RETURN_IF(check_dim(K, kMaxI));
  if (M == 0) return LACACHE_OK;
  const bool group = granularity == LACACHE_GRAN_GROUP;
  if (!ptrs_ok({v, q, s_kgm}) || (!group && !ptrs_ok({s_rows})) || !opt_ptr_ok(s_rows)) return LACACHE_ERR_INVALID_ARG;
  if (!disjoint({rng(q, M * K), rng(s_kgm, (K / 128) * M * 4), rng(s_rows, (!group && s_rows) ? M * 4 : 0)},
                {rng(v, M * K * 4)}))
    return LACACHE_ERR_INVALID_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (group) return hip_status(launch_quant_groups_f32(st, v, q, s_kgm, M, K));
  return hip_status(launch_quant_rows_f32(st, v, q, s_kgm, s_rows, M, K, granularity == LACACHE_GRAN_TENSOR));
}

int lacache_gateup_swiglu_f32(void* stream, const uint8_t* xq, const float* xs, const uint8_t* wgu_q,
                              const float* wgu_s, const float* wgu_row_s, float* h, int64_t M, int64_t H, int64_t I,
                              int group) {
  RETURN_IF(check_group(group));
  RETURN_IF(check_m(M));
  RETURN_IF(check_dim(H, kMaxH));
  RETURN_IF(check_dim(I, kMaxI));
  if (M == 0) return LACACHE_OK;
  if (!ptrs_ok({xq, xs, wgu_q, wgu_s, h}) || !opt_ptr_ok(wgu_row_s)) return LACACHE_ERR_INVALID_ARG;
  if (!disjoint({rng(h, M * I * 4)}, {rng(xq, M * H), rng(xs, (H / 128) * M * 4), rng(wgu_q, 2 * I * H),
                                      rng(wgu_s, (2 * I / 128) * (H / 128) * 4),
                                      rng(wgu_row_s, wgu_row_s ? 2 * I * 4 : 0)}))
    return LACACHE_ERR_INVALID_ARG;
  return hip_status(launch_gateup_tiled(static_cast<hipStream_t>(stream), xq, xs, wgu_q, wgu_s, nullptr, nullptr, h, M,
                                        H, I, wgu_row_s));
}

int lacache_down_proj_g(void* stream, const uint8_t* hq, const float* hs, const uint8_t* wd_q, const float* wd_s,
                        const float* wd_row_s, uint16_t* out, float* out_tap, int64_t M, int64_t H, int64_t I,
                        int group) {
  RETURN_IF(check_group(group));
  RETURN_IF(check_m(M));
  RETURN_IF(check_dim(H, kMaxH));
  RETURN_IF(check_dim(I, kMaxI));
  if (M == 0) return LACACHE_OK;
  if (!ptrs_ok({hq, hs, wd_q, wd_s, out}) || !opt_ptr_ok(out_tap) || !opt_ptr_ok(wd_row_s))
    return LACACHE_ERR_INVALID_ARG;
  if (!disjoint({rng(out, M * H * 2), rng(out_tap, out_tap ? M * H * 4 : 0)},
                {rng(hq, M * I), rng(hs, (I / 128) * M * 4), rng(wd_q, H * I), rng(wd_s, (H / 128) * (I / 128) * 4),
                 rng(wd_row_s, wd_row_s ? H * 4 : 0)}))
    return LACACHE_ERR_INVALID_ARG;
  void* scratch = nullptr;
  if (tiled_down_ws_bytes(M, H, I) > 0)
    RETURN_IF(get_workspace(static_cast<hipStream_t>(stream), tiled_down_ws_bytes(M, H, I), &scratch));
  return hip_status(launch_down_tiled(static_cast<hipStream_t>(stream), hq, hs, wd_q, wd_s, out, out_tap, M, H, I,
                                      scratch, wd_row_s));
}

size_t lacache_ffn_g_workspace_bytes(int64_t M, int64_t H, int64_t I) {
  if (check_m(M) != LACACHE_OK || check_dim(H, kMaxH) != LACACHE_OK || check_dim(I, kMaxI) != LACACHE_OK) return 0;
  const size_t m = static_cast<size_t>(M);
  return align256(m * static_cast<size_t>(H > I ? H : I) * 4) + align256(m * H) + align256((H / 128) * m * 4) +
         align256(m * I) + align256((I / 128) * m * 4) + align256(m * 4) + align256(tiled_down_ws_bytes(M, H, I));
}

int lacache_ffn_fp8_g(void* stream, const uint16_t* x, const uint16_t* norm_w, const uint8_t* wgu_q,
                      const float* wgu_s, const float* wgu_row_s, const uint8_t* wd_q, const float* wd_s,
                      const float* wd_row_s, uint16_t* out, int64_t M, int64_t H, int64_t I, int granularity) {
  if (granularity == LACACHE_GRAN_GROUP) return lacache_ffn_fp8(stream, x, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, M, H, I, 128);
  if (granularity != LACACHE_GRAN_TOKEN && granularity != LACACHE_GRAN_TENSOR) return LACACHE_ERR_INVALID_ARG;
  RETURN_IF(validate_ffn(x, norm_w, wgu_q, wgu_s, wd_q, wd_s, out, M, H, I, 128));
  if (M == 0) return LACACHE_OK;
  if (!ptrs_ok({wgu_row_s, wd_row_s}) ||
      !disjoint({rng(out, M * H * 2)}, {rng(wgu_row_s, 2 * I * 4), rng(wd_row_s, H * 4)}))
    return LACACHE_ERR_INVALID_ARG;
  void* base = nullptr;
  RETURN_IF(get_workspace(static_cast<hipStream_t>(stream), lacache_ffn_g_workspace_bytes(M, H, I), &base));
  // [fp32 y, then h][xq][xs][hq][hs][row scales][split-K partials]
  char* b = static_cast<char*>(base);
  const size_t m = static_cast<size_t>(M);
  float* f = reinterpret_cast<float*>(b);
  b += align256(m * static_cast<size_t>(H > I ? H : I) * 4);
  uint8_t* xq = reinterpret_cast<uint8_t*>(b);
  b += align256(m * H);
  float* xs = reinterpret_cast<float*>(b);
  b += align256((H / 128) * m * 4);
  uint8_t* hq = reinterpret_cast<uint8_t*>(b);
  b += align256(m * I);
  float* hs = reinterpret_cast<float*>(b);
  b += align256((I / 128) * m * 4);
  float* rows = reinterpret_cast<float*>(b);
  b += align256(m * 4);
  void* part = b;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const bool tensor = granularity == LACACHE_GRAN_TENSOR;
  RETURN_IF(hip_status(launch_rmsnorm_f32(st, x, norm_w, f, M, H)));
  RETURN_IF(hip_status(launch_quant_rows_f32(st, f, xq, xs, rows, M, H, tensor)));
  RETURN_IF(hip_status(launch_gateup_tiled(st, xq, xs, wgu_q, wgu_s, nullptr, nullptr, f, M, H, I, wgu_row_s)));
  RETURN_IF(hip_status(launch_quant_rows_f32(st, f, hq, hs, rows, M, I, tensor)));
  return hip_status(launch_down_tiled(st, hq, hs, wd_q, wd_s, out, nullptr, M, H, I, part, wd_row_s));
}

// ---------------------------------------------------------------------------
// Token-wise first layer (EmbedCache, RoPECache)
// ---------------------------------------------------------------------------

int lacache_embed_rmsnorm(void* stream, const int32_t* token_ids, const int32_t* rows, int64_t R,
                          const uint16_t* embed, int64_t vocab, const uint16_t* norm_w, uint16_t* embed_cache,
                          int64_t N, uint16_t* y, int64_t H) {
  if (R < 0 || vocab <= 0 || N <= 0) return LACACHE_ERR_INVALID_ARG;
  RETURN_IF(check_dim(H, kMaxH));
  if (R > kMaxM || N > kMaxM) return LACACHE_ERR_UNSUPPORTED;
  if (R == 0) return LACACHE_OK;
  if (!ptrs_ok({token_ids, rows, embed, norm_w, embed_cache, y})) return LACACHE_ERR_INVALID_ARG;
  const size_t hb = static_cast<size_t>(H) * 2;
  if (!disjoint({rng(embed_cache, N * hb), rng(y, R * hb)},
                {rng(token_ids, R * 4), rng(rows, R * 4), rng(embed, vocab * hb), rng(norm_w, hb)}))
    return LACACHE_ERR_INVALID_ARG;
  return hip_status(launch_embed_rmsnorm(static_cast<hipStream_t>(stream), token_ids, rows, R, embed, vocab, norm_w,
                                         embed_cache, N, y, H));
}

int lacache_linear_bf16(void* stream, const uint16_t* a, const uint16_t* w, uint16_t* out, float* out_tap, int64_t M,
                        int64_t N, int64_t K) {
  RETURN_IF(check_m(M));
  RETURN_IF(check_dim(N, kMaxN));
  RETURN_IF(check_dim(K, kMaxN));
  if (M == 0) return LACACHE_OK;
  if (!ptrs_ok({a, w, out}) || !opt_ptr_ok(out_tap)) return LACACHE_ERR_INVALID_ARG;
  if (!disjoint({rng(out, M * N * 2), rng(out_tap, out_tap ? M * N * 4 : 0)}, {rng(a, M * K * 2), rng(w, N * K * 2)}))
    return LACACHE_ERR_INVALID_ARG;
  return hip_status(launch_linear_bf16(static_cast<hipStream_t>(stream), a, w, out, out_tap, M, N, K));
}

int lacache_rope_scatter(void* stream, const uint16_t* qkv, const int32_t* rows, int64_t R, const float* rope_cos,
                         const float* rope_sin, uint16_t* q, uint16_t* k, uint16_t* v, int64_t heads, int64_t N) {
  if (R < 0 || heads <= 0 || N <= 0) return LACACHE_ERR_INVALID_ARG;
  if (heads > kAttnMaxHeads || N > kAttnMaxN || R > kMaxM) return LACACHE_ERR_UNSUPPORTED;
  if (R == 0) return LACACHE_OK;
  if (!ptrs_ok({qkv, rows, rope_cos, rope_sin, q, k, v})) return LACACHE_ERR_INVALID_ARG;
  const size_t cache = static_cast<size_t>(heads * N) * 128 * 2, tab = static_cast<size_t>(N) * 64 * 4;
  if (!disjoint({rng(q, cache), rng(k, cache), rng(v, cache)},
                {rng(qkv, R * 3 * heads * 128 * 2), rng(rows, R * 4), rng(rope_cos, tab), rng(rope_sin, tab)}))
    return LACACHE_ERR_INVALID_ARG;
  return hip_status(launch_rope_scatter(static_cast<hipStream_t>(stream), qkv, rows, R, rope_cos, rope_sin, q, k, v,
                                        heads, N));
}

size_t lacache_first_layer_workspace_bytes(int64_t R, int64_t heads, int64_t H) {
  if (R < 0 || heads <= 0 || check_dim(H, kMaxH) != LACACHE_OK) return 0;
  return align256(static_cast<size_t>(R * H) * 2) + align256(static_cast<size_t>(R * 3 * heads * 128) * 2);
}

int lacache_first_layer_tokens(void* stream, const int32_t* token_ids, const int32_t* rows, int64_t R,
                               const uint16_t* embed, int64_t vocab, const uint16_t* norm_w, const uint16_t* w_qkv,
                               const float* rope_cos, const float* rope_sin, uint16_t* embed_cache, uint16_t* q,
                               uint16_t* k, uint16_t* v, int64_t heads, int64_t N, int64_t H) {
  if (R < 0 || vocab <= 0 || N <= 0 || heads <= 0) return LACACHE_ERR_INVALID_ARG;
  RETURN_IF(check_dim(H, kMaxH));
  if (heads > kAttnMaxHeads || N > kAttnMaxN || R > kMaxM || 3 * heads * 128 > kMaxN) return LACACHE_ERR_UNSUPPORTED;
  if (R == 0) return LACACHE_OK;
  if (!ptrs_ok({token_ids, rows, embed, norm_w, w_qkv, rope_cos, rope_sin, embed_cache, q, k, v}))
    return LACACHE_ERR_INVALID_ARG;
  const size_t hb = static_cast<size_t>(H) * 2, cache = static_cast<size_t>(heads * N) * 128 * 2;
  const size_t tab = static_cast<size_t>(N) * 64 * 4, nq = static_cast<size_t>(3 * heads * 128);
  if (!disjoint({rng(embed_cache, N * hb), rng(q, cache), rng(k, cache), rng(v, cache)},
                {rng(token_ids, R * 4), rng(rows, R * 4), rng(embed, vocab * hb), rng(norm_w, hb),
                 rng(w_qkv, nq * hb), rng(rope_cos, tab), rng(rope_sin, tab)}))
    return LACACHE_ERR_INVALID_ARG;
  void* base = nullptr;
  RETURN_IF(get_workspace(static_cast<hipStream_t>(stream), lacache_first_layer_workspace_bytes(R, heads, H), &base));
  uint16_t* y = static_cast<uint16_t*>(base);
  uint16_t* qkv = reinterpret_cast<uint16_t*>(static_cast<char*>(base) + align256(static_cast<size_t>(R * H) * 2));
  hipStream_t st = static_cast<hipStream_t>(stream);
  RETURN_IF(hip_status(launch_embed_rmsnorm(st, token_ids, rows, R, embed, vocab, norm_w, embed_cache, N, y, H)));
  RETURN_IF(hip_status(launch_linear_bf16(st, y, w_qkv, qkv, nullptr, R, static_cast<int64_t>(nq), H)));
  return hip_status(launch_rope_scatter(st, qkv, rows, R, rope_cos, rope_sin, q, k, v, heads, N));
}

int lacache_add_bf16(void* stream, uint16_t* x_inout, const uint16_t* y, int64_t n) {
  if (n < 0) return LACACHE_ERR_INVALID_ARG;
  if (n == 0) return LACACHE_OK;
  if (!ptrs_ok({x_inout, y})) return LACACHE_ERR_INVALID_ARG;
  if (overlap(rng(x_inout, n * 2), rng(y, n * 2))) return LACACHE_ERR_INVALID_ARG;
  return hip_status(launch_add_bf16(static_cast<hipStream_t>(stream), x_inout, y, n));
}

int lacache_encode_e4m3(void* stream, const float* v, uint8_t* codes, int64_t n) {
  if (n < 0) return LACACHE_ERR_INVALID_ARG;
  if (n > (int64_t(1) << 32)) return LACACHE_ERR_UNSUPPORTED;
  if (n == 0) return LACACHE_OK;
  if (!ptrs_ok({v, codes})) return LACACHE_ERR_INVALID_ARG;
  if (overlap(rng(v, n * 4), rng(codes, n))) return LACACHE_ERR_INVALID_ARG;
  return hip_status(launch_encode_e4m3(static_cast<hipStream_t>(stream), v, codes, n));
}

int lacache_facache_attention(void* stream, const uint16_t* q, const uint16_t* k, const uint16_t* v, uint16_t* o,
                              float* lse, float* cache_m, float* cache_l, float* cache_o, int64_t heads, int64_t N,
                              int64_t d, int64_t c_begin, int64_t c_end, int mode) {
  if (heads < 0 || N < 0 || mode < 0 || mode > 2) return LACACHE_ERR_INVALID_ARG;
  if (c_begin < 0 || c_begin > c_end || c_end > N) return LACACHE_ERR_INVALID_ARG;
  if (d != kAttnHeadDim || N % kAttnBlock != 0 || heads > kAttnMaxHeads || N > kAttnMaxN)
    return LACACHE_ERR_UNSUPPORTED;
  if (heads == 0 || N == 0) return LACACHE_OK;
  if (!ptrs_ok({q, k, v, o}) || !opt_ptr_ok(lse)) return LACACHE_ERR_INVALID_ARG;
  const size_t act = static_cast<size_t>(heads * N * d) * 2, st = static_cast<size_t>(heads * N) * 4;
  const Range ro = rng(o, act), rq = rng(q, act), rk = rng(k, act), rv = rng(v, act);
  const Range rs = lse != nullptr ? rng(lse, st) : Range{0, 0};
  if (mode == 2) {
    if (!disjoint({ro, rs}, {rq, rk, rv})) return LACACHE_ERR_INVALID_ARG;
  } else {
    if (!ptrs_ok({cache_m, cache_l, cache_o})) return LACACHE_ERR_INVALID_ARG;
    const Range rm = rng(cache_m, st), rl = rng(cache_l, st), rc = rng(cache_o, st * d);
    const bool ok =
        mode == 0 ? disjoint({ro, rs, rm, rl, rc}, {rq, rk, rv}) : disjoint({ro, rs}, {rq, rk, rv, rm, rl, rc});
    if (!ok) return LACACHE_ERR_INVALID_ARG;
  }
  return hip_status(launch_facache_attention(static_cast<hipStream_t>(stream), q, k, v, o, cache_m, cache_l, cache_o,
                                             lse, heads, N, c_begin, c_end, mode));
}

int lacache_set_path_policy(int policy) {
  if (policy < 0 || policy > 2) return LACACHE_ERR_INVALID_ARG;
  return g_policy.exchange(policy);
}

const char* lacache_status_string(int status) {
  switch (status) {
    case LACACHE_OK: return "LACACHE_OK";
    case LACACHE_ERR_INVALID_ARG: return "LACACHE_ERR_INVALID_ARG";
    case LACACHE_ERR_UNSUPPORTED: return "LACACHE_ERR_UNSUPPORTED";
    case LACACHE_ERR_HIP: return "LACACHE_ERR_HIP";
    case LACACHE_ERR_ALLOC: return "LACACHE_ERR_ALLOC";
    case LACACHE_ERR_CAPTURE: return "LACACHE_ERR_CAPTURE";
    default: return "LACACHE_UNKNOWN_STATUS";
  }
}

void lacache_release_workspace(void) {
  std::lock_guard<std::mutex> lk(g_ws_mu);
  int cur = 0;
  const bool have_cur = hipGetDevice(&cur) == hipSuccess;
  for (size_t d = 0; d < g_ws.size(); ++d) {
    if (g_ws[d].ptr == nullptr && g_ws[d].retired.empty()) continue;
    if (hipSetDevice(static_cast<int>(d)) == hipSuccess) {
      (void)hipDeviceSynchronize();
      if (g_ws[d].ptr != nullptr) (void)hipFree(g_ws[d].ptr);
      for (void* p : g_ws[d].retired) (void)hipFree(p);
    }
    g_ws[d] = DeviceWs{};
  }
  if (have_cur) (void)hipSetDevice(cur);
}

}  // extern "C"
