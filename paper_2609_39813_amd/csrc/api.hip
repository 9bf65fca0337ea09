// C-ABI entry points: argument checking, workspace layout and the launch sequence of
// each call. Every step of the computation runs in the kernels of this library.
#include "bsp_kernels.h"
#include "k_norm.h"
#include "norm_run.h"

using namespace bsp;

#define BS_TRY(x)                  \
  do {                             \
    const bs_status _s = (x);      \
    if (_s != BS_OK) return _s;    \
  } while (0)

extern "C" {

const char* bs_status_string(bs_status s) {
  switch (s) {
    case BS_OK: return "ok";
    case BS_EINVAL: return "invalid argument";
    case BS_ESHAPE: return "unsupported shape";
    case BS_EDTYPE: return "unsupported dtype";
    case BS_EUNSUPPORTED: return "not implemented by the library";
    case BS_EWORKSPACE: return "workspace missing, misaligned or too small";
    case BS_EHIP: return "HIP runtime error";
  }
  return "unknown status";
}

int bs_version(void) { return 100; }

bs_status bs_qround(const void* x, bs_dtype xt, int64_t n, bs_fp8 fmt, bs_round mode, uint64_t seed, uint32_t trial,
                    uint32_t use, const float* scale_in, uint8_t* codes, float* scale_out, bs_diag* diag,
                    void* stream) {
  if (n < 0 || !diag || !scale_out || (n > 0 && (!x || !codes))) return BS_EINVAL;
  if (xt != BS_F32 && xt != BS_BF16) return BS_EDTYPE;
  if ((fmt != BS_E4M3 && fmt != BS_E5M2) || (mode != BS_RNE && mode != BS_SR)) return BS_EINVAL;
  return launch_store(x, xt, n, fmt, mode, seed, trial, use, scale_in, codes, scale_out, diag, (hipStream_t)stream,
                      false);
}

bs_status bs_gemm_bf16_nt(const void* A, int64_t lda, const void* B, int64_t ldb, float* C, int64_t ldc, int64_t M,
                          int64_t N, int64_t K, float alpha, int accumulate, void* stream) {
  if (M < 0 || N < 0 || K < 0 || !C || (K > 0 && (!A || !B)) || ldc < N) return BS_EINVAL;
  if (M > 0x7FFFFFFF || N > 0x7FFFFFFF || K > 0x7FFFFFFF || lda < K || ldb < K) return BS_ESHAPE;
  GemmArgs g{};
  g.A[0] = (const u16*)A;
  g.B[0] = (const u16*)B;
  g.nseg = 1;
  g.M = (int)M;
  g.N = (int)N;
  g.K = (int)K;
  g.lda = lda;
  g.ldb = ldb;
  g.ldc = ldc;
  g.alpha = alpha;
  g.accumulate = accumulate;
  g.C = C;
  return launch_gemm(g, (hipStream_t)stream);
}

size_t bs_policy_bias_workspace_size(int K, int64_t m) {
  (void)K;
  Carver c;
  c.take<double>((size_t)(3 * ((m + 255) / 256) + 3));
  return c.used();
}

bs_status bs_policy_bias_estimate(const float* delta, int K, int64_t m, const float* g_ref, float* mean_err, float* se,
                                  double* summary, void* ws, size_t ws_bytes, void* stream) {
  if (K < 1 || m < 0 || (m > 0 && (!delta || !mean_err))) return BS_EINVAL;
  if (!ws || ((uintptr_t)ws & 255) || ws_bytes < bs_policy_bias_workspace_size(K, m)) return BS_EWORKSPACE;
  return launch_policy_bias(delta, K, m, g_ref, mean_err, se, summary, (double*)ws, (hipStream_t)stream);
}

// ------------------------------------------------------------------------------------
// RMSNorm -> FP8 store -> Linear (the runner is in norm_run.hip)
// ------------------------------------------------------------------------------------
size_t bs_rmsnorm_linear_workspace_size(int64_t T, int64_t d, int64_t n, int n_pol, int K) {
  (void)n_pol;
  return norm_ws_size(T, d, n, K);
}

bs_status bs_rmsnorm_linear_fwd_bwd(const void* X, const float* gain, const void* W, const void* dY, bs_dtype dt,
                                    int64_t T, int64_t d, int64_t n, float eps, bs_fp8 fmt, bs_round fwd_mode,
                                    const bs_norm_policy* pol, int n_pol, int K, uint64_t seed, uint32_t store_id,
                                    float* Y, uint8_t* u_codes, float* u_scale, float* dgain_ref, float* dW_ref,
                                    float* dX_ref, bs_est dgain, bs_est dW, bs_est dX, bs_diag* diag, void* ws,
                                    size_t ws_bytes, void* stream) {
  NormIO io{X, dt, gain, W, dt, dY, dt, T, d, n, eps, fmt, fwd_mode, pol, n_pol, K, seed, store_id,
            Y, u_codes, u_scale, dgain_ref, dW_ref, dX_ref, dgain, dW, dX, diag};
  return norm_run(io, ws, ws_bytes, (hipStream_t)stream);
}

}  // extern "C"
