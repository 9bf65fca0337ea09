// Entry points whose kernels are not in this build yet: they validate nothing and
// report BS_EUNSUPPORTED, so the library still exports every declared symbol.
#include "bsp_kernels.h"

extern "C" {

size_t bs_linear_bwd_workspace_size(int64_t M, int64_t k, int64_t n, int n_pol, int K) {
  (void)M; (void)k; (void)n; (void)n_pol; (void)K;
  return 0;
}
bs_status bs_linear_bwd_policy(const void*, const void*, const void*, bs_dtype, int64_t, int64_t, int64_t, bs_fp8,
                               const int*, int, int, uint64_t, uint32_t, float*, float*, bs_est, bs_est, const float*,
                               const float*, double*, float*, bs_diag*, void*, size_t, void*) {
  return BS_EUNSUPPORTED;
}

}  // extern "C"
