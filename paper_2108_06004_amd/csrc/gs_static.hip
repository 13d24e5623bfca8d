// gs_static.hip -- gs_unsketch_topk_static: the estimate and top-k selection of
// gs_unsketch_topk (Alg. 2: median of the r signed cells, the k largest |estimate|) for
// callers that cannot allocate device memory. No context: the hash family comes from the
// caller's gs_config on every call, and the selection's scratch (candidate keys, the staged
// digit-1 bucket, histograms, the output bitmap, the control block) lives in one fixed
// device array of this file, `scratch`. It runs the same kernels as gs_unsketch_topk's full
// path (every coordinate estimated), on pointers into that array.
#include <cstdio>
#include <mutex>

#include "../../include/gs.h"
#include "gs_internal.hpp"

namespace {

constexpr int64_t kMaxD = GS_STATIC_MAX_D;
constexpr int64_t kAlignWords = 64;  // 256-byte alignment of every region
constexpr int64_t up(int64_t n) { return (n + kAlignWords - 1) / kAlignWords * kAlignWords; }
constexpr int64_t kCtlWords = up((int64_t)((sizeof(gs::SelectCtl) + 3) / 4));
constexpr int64_t kFlagWords = 64;  // look-back words of the emit, 2 per emit block: 32 at kMaxD (checked per call)

// Layout of the array in 32-bit words.
constexpr int64_t kCandKey = 0;                            // [kMaxD] key of coordinate t
constexpr int64_t kStageKey = kCandKey + up(kMaxD);        // [kMaxD] staged keys
constexpr int64_t kStageIdx = kStageKey + up(kMaxD);       // [kMaxD] their coordinates
constexpr int64_t kBitmap = kStageIdx + up(kMaxD);         // [kMaxD / 32] output bitmap
constexpr int64_t kFlags = kBitmap + up((kMaxD + 31) / 32);
// Cleared at the start of every call (the selection needs them zero and leaves them zero,
// but a call that was never completed, or one overlapping on another stream, may not have).
constexpr int64_t kZero = kFlags + kFlagWords;
constexpr int64_t kHist = kZero;                           // [kDigit1Bins]
constexpr int64_t kHist2 = kHist + gs::kDigit1Bins;        // [kDigitBins]
constexpr int64_t kHistC = kHist2 + gs::kDigitBins;        // [kDigit1Bins] (not read: dense candidates)
constexpr int64_t kCtl = kHistC + gs::kDigit1Bins;         // SelectCtl
constexpr int64_t kZeroWords = kCtl + kCtlWords - kZero;
constexpr int64_t kWords = kZero + kZeroWords;
static_assert(kCtl % kAlignWords == 0, "control block alignment");

}  // namespace

// The scratch of gs_unsketch_topk_static: 12.1 bytes per coordinate of GS_STATIC_MAX_D
// (48.6 MiB). Each GPU the library runs on holds its own copy for the life of the process.
// Host code never passes this name to a kernel: on the host it is only a stand-in for the
// device symbol; the device address comes from hipGetSymbolAddress (per device, below).
static __device__ __align__(256) uint32_t scratch[kWords];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_setup_mu;
uint32_t* g_scratch_ptr[kMaxDevices];  // device address of `scratch` on each device, once set up
int g_num_cus[kMaxDevices];

// Once per device, with that device current: look up its copy of `scratch`.
hipError_t scratch_of_current_device(uint32_t** ptr, int* num_cus) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_setup_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    int n = 0;
    e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    g_num_cus[dev] = n > 0 ? n : 256;
    g_scratch_ptr[dev] = static_cast<uint32_t*>(p);
  }
  *ptr = g_scratch_ptr[dev];
  *num_cus = g_num_cus[dev];
  return hipSuccess;
}

gs_status invalid(const char* msg) {
  gs::set_free_error(msg);
  return GS_ERR_INVALID_ARG;
}

gs_status device_error(const char* where, hipError_t e) {
  char buf[256];
  std::snprintf(buf, sizeof buf, "gs_unsketch_topk_static: %s: %s", where, hipGetErrorString(e));
  gs::set_free_error(buf);
  return GS_ERR_DEVICE;
}

}  // namespace

extern "C" gs_status gs_unsketch_topk_static(const gs_config* cfg, void* stream, const float* merged, int64_t k,
                                             float* est, int32_t* idx) {
  constexpr int64_t p = GS_MERSENNE_P;
  gs::set_free_error("");
  if (!cfg) return invalid("gs_unsketch_topk_static: cfg is NULL");
  if (!merged || !idx) return invalid("gs_unsketch_topk_static: NULL array");
  if (cfg->d < 1 || cfg->d > kMaxD)
    return invalid("gs_unsketch_topk_static: d must satisfy 1 <= d <= GS_STATIC_MAX_D (4,194,304)");
  if (cfg->r < 1 || cfg->r > GS_MAX_ROWS) return invalid("gs_unsketch_topk_static: r must satisfy 1 <= r <= 16");
  if (cfg->c < 1 || cfg->c > p - 1) return invalid("gs_unsketch_topk_static: c must satisfy 1 <= c <= 2^31 - 2");
  if (k < 1 || k > cfg->d) return invalid("gs_unsketch_topk_static: k must satisfy 1 <= k <= d");
  if (!cfg->hash_a || !cfg->hash_b || !cfg->sign_a || !cfg->sign_b)
    return invalid("gs_unsketch_topk_static: hash parameter array is NULL");
  gs::HashSet hs{};
  hs.r = cfg->r;
  for (int j = 0; j < cfg->r; ++j) {
    const uint32_t a = cfg->hash_a[j], b = cfg->hash_b[j], a2 = cfg->sign_a[j], b2 = cfg->sign_b[j];
    if (a < 1 || a >= p || b >= p || a2 < 1 || a2 >= p || b2 >= p)
      return invalid("gs_unsketch_topk_static: hash parameters must satisfy 1 <= a < p and 0 <= b < p");
    hs.row[j] = gs::RowHash{a, b, a2, b2};
  }
  gs::set_divisor(hs, (uint32_t)cfg->c);

  uint32_t* base = nullptr;
  int num_cus = 0;
  hipError_t e = scratch_of_current_device(&base, &num_cus);
  if (e != hipSuccess) return device_error("scratch set-up", e);
  const int64_t d = cfg->d;
  if (2 * gs::emit_blocks_for(d) > kFlagWords) return device_error("scratch layout", hipErrorInvalidValue);
  const gs::SelectBufs bufs{base + kCandKey,
                            reinterpret_cast<int32_t*>(base + kStageIdx),  // candidates are dense: never read
                            d,
                            base + kStageKey,
                            reinterpret_cast<int32_t*>(base + kStageIdx),
                            base + kHist,
                            base + kHist2,
                            base + kHistC,
                            reinterpret_cast<gs::SelectCtl*>(base + kCtl),
                            base + kBitmap,
                            reinterpret_cast<unsigned long long*>(base + kFlags),
                            gs::emit_blocks_for(d),
                            gs::kEmitSpinDefault};
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  e = gs::launch_fill_zero(s, reinterpret_cast<float*>(base + kZero), kZeroWords);  // a kernel, not a memset
  if (e == hipSuccess) e = gs::launch_unsketch_topk_dense(hs, d, num_cus, bufs, s, merged, k, est, idx);
  if (e != hipSuccess) return device_error("launch", e);
  return GS_OK;
}
