// C-ABI entry point reducing any call's estimate arrays to the summary statistics of App. D.4.
#include "bsp_kernels.h"
#include "k_layer.h"

using namespace bsp;

namespace {

// sums [3] = (sum b^2, sum ref^2, sum se^2) -> (||b||, ||ref||, R = sum b^2 / sum se^2)
__global__ void estimate_summary_kernel(const double* __restrict__ sums, double* __restrict__ summary) {
  if (threadIdx.x != 0) return;
  summary[0] = sqrt(sums[0]);
  summary[1] = sqrt(sums[1]);
  summary[2] = sums[2] > 0.0 ? sums[0] / sums[2] : __builtin_nan("");
}

size_t summary_ws_doubles() { return sumsq_part_size() + 3; }

}  // namespace

extern "C" {

size_t bs_estimate_summary_workspace_size(void) {
  Carver c;
  c.take<double>(summary_ws_doubles());
  return c.used();
}

bs_status bs_estimate_summary(const float* bias, const float* se, const float* ref, int64_t n, double* summary,
                              void* ws, size_t ws_bytes, void* stream) {
  if (n < 0 || !summary || (n > 0 && !bias)) return BS_EINVAL;
  if (!ws || ((uintptr_t)ws & 255) || ws_bytes < bs_estimate_summary_workspace_size()) return BS_EWORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  double* part = (double*)ws;
  double* sums = part + sumsq_part_size();
  SumsqBatch b{};
  // a missing array sums to 0 (job with no data and n == 1)
  b.job[b.count++] = SumsqJob{n > 0 ? bias : nullptr, n > 0 ? n : 1, sums + 0};
  b.job[b.count++] = SumsqJob{(n > 0 && ref) ? ref : nullptr, (n > 0 && ref) ? n : 1, sums + 1};
  b.job[b.count++] = SumsqJob{(n > 0 && se) ? se : nullptr, (n > 0 && se) ? n : 1, sums + 2};
  const bs_status s = launch_sumsq_batch(b, part, st);
  if (s != BS_OK) return s;
  estimate_summary_kernel<<<1, 64, 0, st>>>(sums, summary);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

}  // extern "C"
