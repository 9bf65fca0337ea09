// Argument blocks and launchers of the normalization-store kernels.
#pragma once
#include "bsp_kernels.h"

namespace bsp {

enum { NP_VAL = 0, NP_RESU = 1, NP_RESN = 2 };

struct NormPlaneArgs {
  const float* u;          // [T, d] quantizer input
  const uint8_t* codes;    // [T, d] forward codes
  const float* scale;      // device scalar s
  const u16* counts;       // [T, d] new-rounding up counts (NP_RESN)
  int K;
  F8 f;
  int64_t T, d;
  u16* out[3];             // planes [d][ldo]
  int nterms;
  int64_t ldo;
};

template <typename XT>
struct GainArgs {
  const XT* X;
  const float* rstd;
  const float* gain;
  const float* u;
  const float* du;
  const uint8_t* codes;
  const u16* counts;       // nullable: N term
  const float* scale;
  int K;
  int want_r;
  F8 f;
  int64_t T, d;
  double* part;            // [3][nrt][d]
};

template <typename XT>
struct DxArgs {
  const XT* X;
  const float* rstd;
  const float* gain;
  const float* du;
  const uint8_t* codes;
  const float* scale;
  F8 f;
  int64_t T, d;
  float* dx_ref;
  float* dx_r;             // nullable: the R reading at the norm-input use
};

bs_status launch_rmsnorm_fwd(const void* X, bs_dtype dt, const float* gain, int64_t T, int64_t d, float eps, float* u,
                             float* rstd, bs_diag* diag, hipStream_t st);
bs_status launch_norm_planes(int mode, const NormPlaneArgs& a, hipStream_t st);
bs_status launch_val_rows(const uint8_t* codes, int64_t n, int fmt, u16* out, hipStream_t st);
template <typename T>
bs_status launch_gain_t(const GainArgs<T>& a, float* ref, float* bias_r, float* bias_n, hipStream_t st);
bs_status launch_gain_se(const float* part, int K, int64_t T, int64_t d, const float* scale, const float* gain,
                         double* S, float* se, hipStream_t st);
template <typename T>
bs_status launch_dx_t(const DxArgs<T>& a, hipStream_t st);

bs_status launch_combine_alt(const float* ref, const float* alt, int64_t n, float* mean_out, float* bias_out,
                             float* se_out, hipStream_t st);

}  // namespace bsp
