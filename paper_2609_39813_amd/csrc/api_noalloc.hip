// The generic trial reducer with its scratch in a file-scope device array: an entry point for
// callers that cannot allocate (code under graph capture, tight serving loops). The kernels are
// those of bs_policy_bias_estimate; only the home of the per-block partials differs.
#include <mutex>

#include "bsp_kernels.h"

using namespace bsp;

namespace {

constexpr int64_t kNoAllocMaxM = (int64_t)1 << 26;         // outputs per call
constexpr int64_t kScratchDoubles = 3 * (kNoAllocMaxM / 256);  // 3 fp64 partials per 256-output block: 6 MiB
constexpr int kMaxDevices = 64;

// Every GPU the library runs on holds its own copy until the process ends. In host code the name
// is a host-side stand-in, never a device address: kernels get the per-device pointer below.
static __device__ __align__(256) double scratch[kScratchDoubles];

std::mutex g_mu;
double* g_ptr[kMaxDevices] = {};

// The device's address of `scratch`, resolved once per device with that device current.
bs_status scratch_ptr(double** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return BS_EHIP;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return BS_EHIP;
    g_ptr[dev] = (double*)p;
  }
  *out = g_ptr[dev];
  return BS_OK;
}

}  // namespace

extern "C" {

int64_t bs_policy_bias_noalloc_max(void) { return kNoAllocMaxM; }

bs_status bs_policy_bias_estimate_noalloc(const float* delta, int K, int64_t m, const float* g_ref, float* mean_err,
                                          float* se, double* summary, void* stream) {
  if (K < 1 || m < 0 || (m > 0 && (!delta || !mean_err))) return BS_EINVAL;
  if (m > kNoAllocMaxM) return BS_ESHAPE;
  double* ws = nullptr;
  const bs_status s = scratch_ptr(&ws);
  if (s != BS_OK) return s;
  // every partial the summary reads is written by this call's first kernel: nothing to clear
  return launch_policy_bias(delta, K, m, g_ref, mean_err, se, summary, ws, (hipStream_t)stream);
}

}  // extern "C"
