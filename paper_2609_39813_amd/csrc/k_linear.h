// Argument blocks and launchers of the E5M2-gradient Linear backward kernels.
#pragma once
#include "bsp_kernels.h"

namespace bsp {

struct ResidArgs {
  const u16* dY;          // [M][n] bf16 incoming gradient
  const u16* counts;      // [M][n] up counts of the use's new roundings
  const float* scale;     // device s
  int K;
  F8 f;
  int64_t M, n;
  u16* rows[3];           // nullable: E split into 3 terms, row-major [M][n]
  u16* cols[3];           // nullable: E split into 3 terms, transposed [n][ldo]
  int64_t ldo;
};

bs_status launch_resid_planes(const ResidArgs& a, hipStream_t st);
// A0 = sum (s sign lo - dY) AW and B0 = sum (s sign lo - dY) XB (fp64), into out[0..1]
bs_status launch_kappa_fixed(const u16* dY, const float* scale, int fmt, int64_t M, int64_t n, const float* AW,
                             const float* XB, double* part, double* out, hipStream_t st);
// kappa = (1/K) sum_k (A0 + s Sa_k)(B0 + s Sb_k), Sa_k / Sb_k = sums of block partials
bs_status launch_kappa_final(const double* fixed, const double* pa, int ia, const double* pb, int ib, int64_t nblk,
                             int K, const float* scale, double* kappa, hipStream_t st);

}  // namespace bsp
