// Argument blocks and launchers of the normalization-store kernels.
#pragma once
#include "bsp_kernels.h"
#include "k_combine.h"

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
  int f16 = 0;             // fp16 planes: NP_VAL the values (exact for FP8 codes); NP_RESU the
                           // two-term split of the residual 2^e (e = f16_scale_exp of max(*amax_u,
                           // s FMAX), less one: |u - s val| <= |u| + s FMAX), 2^-e to *inv_out;
                           // NP_RESN one exact term of the residual times resn_scale (K <= 256)
  const float* amax_u = nullptr;  // device max |u| (nullable)
  float* inv_out = nullptr;
  float resn_scale = 1.0f;        // a power of two that keeps K max-step within fp16
};

// rows per block of the gain use's column partial sums (the partial array holds one row of
// partials per tile of GAIN_RT rows)
constexpr int GAIN_RT = 16;

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

// Per-trial weight-use residual planes: for trials k0 .. k0 + nb - 1 (new roundings of u at
// the store's scale, use id `use`), plane b [d][ldo] of out holds sign * (up_k - [C_u rounded
// up]) * step (one exact bf16 term; zero for t >= T), and of outW the new rounding's value
// val(C_u) + that step (the forward's value when they agree). Either output nullable. ldo a
// multiple of 64, d of 4, the outputs and u 16-byte and codes 4-byte aligned (BS_EINVAL
// otherwise).
struct TrialPlaneArgs {
  const float* u;
  const uint8_t* codes;
  const float* scale;
  F8 f;
  int64_t T, d, ldo;
  uint64_t seed;
  uint32_t use;
  int k0, nb;
  u16* out;  // [nb][d][ldo]
  int f16 = 0;  // fp16 values (exact: FP8 values and steps) instead of bf16
  u16* outW = nullptr;  // [nb][d][ldo]
};
bs_status launch_trial_planes(const TrialPlaneArgs& a, hipStream_t st);
// Shifted fp64 sums over trials of delta [nb][m] (trials k0 ..): trial 1 is stored as the shift
// d1; S1 += delta - d1, S2 += (delta - d1)^2 for the others, in trial order.
bs_status launch_trial_accum(const float* delta, int nb, int k0, int64_t m, float* d1, double* S1, double* S2,
                             hipStream_t st);
// se = sqrt(max(S2 - S1^2 / K, 0) / (K - 1) / K) (0 for K = 1)
bs_status launch_trial_se(const double* S1, const double* S2, int K, int64_t m, float* se, hipStream_t st);

// column sums of [3][nrt][d] fp64 partials (row tiles in order within 16 segments, the segments by
// a fixed tree) into ref, bias_r and bias_n [d] (bias_r / bias_n nullable)
bs_status launch_gain_final(const double* part, int64_t nrt, int64_t d, float* ref, float* bias_r, float* bias_n,
                            hipStream_t st);

bs_status launch_combine_alt(const float* ref, const float* alt, int64_t n, float* mean_out, float* bias_out,
                             float* se_out, hipStream_t st);

}  // namespace bsp
