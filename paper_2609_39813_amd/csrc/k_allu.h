// Kernels of the decoder layer's "every use at once" check: with one letter (U, R or N) read at
// every use of every store, the backward's gradients move away from the reference through the
// normalization-input, D and weight uses. These kernels form those moves (deltas against the
// reference) from residual operands, in fp64 where they are sums.
#pragma once
#include "bsp_kernels.h"

namespace bsp {

enum { LETTER_U = 0, LETTER_R = 1, LETTER_N = 2 };

// A store as the uses read it: its fp32 input x (token-major [T][d], or head-major rows of 64 for
// the attention output), the forward's codes and scale, and the key of a new rounding.
struct StoreRead {
  const float* x;
  const uint8_t* codes;
  const float* scale;
  F8 f;
  int letter;
  uint64_t seed;
  uint32_t trial, use;
};

// Gain use of a normalization store (Eq. norm-uses): column partial sums over 16-row tiles of
// z_g (du + ddu) - z du = (z_g - z)(du + ddu) + z ddu, z = fl32(X r) the original, z_g what the
// letter reads (z; s val(C) / gain; s val(new rounding) / gain). ddu nullable (the incoming
// gradient's own move).
template <typename XT>
struct AlluGainArgs {
  const XT* X;
  const float* rstd;
  const float* gain;
  StoreRead rd;     // rd.x = u (the store input, for the new rounding)
  const float* du;  // [T][d] the reference incoming gradient at the use
  const float* ddu; // nullable [T][d]
  int64_t T, d;
  double* part;     // [ceil(T / 16)][d]
};
template <typename XT>
bs_status launch_allu_gain(const AlluGainArgs<XT>& a, hipStream_t st);

// Normalization-input use: per row t, the move of r (dz - z_x (dz . z_x) / d) with dz = gain (du +
// ddu) and z_x what the letter reads, against the reference (z, gain du):
// r (gain ddu - (z_x (dz_L . z_x) - z (dz_ref . z)) / d), plus add (nullable) elementwise.
template <typename XT>
struct AlluDxArgs {
  const XT* X;
  const float* rstd;
  const float* gain;
  StoreRead rd;
  const float* du;
  const float* ddu;  // nullable
  const float* add;  // nullable [T][d]
  int64_t T, d;
  float* out;        // [T][d]
  uint32_t* amax = nullptr;  // nullable: slots (AMAX_SLOTS) raised to max |out|
};
template <typename XT>
bs_status launch_allu_dx(const AlluDxArgs<XT>& a, hipStream_t st);

// The gain and normalization-input uses of one store together: one read of X, u, du and ddu
// serves both. The gain use's partial sums per 16-row tile have allu_gain's layout. Within a
// tile, each group of 4 rows is summed in row order, then the 4 groups in order. d > 1024
// falls back to the two separate kernels.
template <typename XT>
struct AlluGainDxArgs {
  AlluDxArgs<XT> dx;  // the normalization-input use (dx.rd its read of the store)
  StoreRead rd_g;     // the gain use's read of the same store (rd_g.x == dx.rd.x)
  double* part;       // [ceil(T / 16)][d]
};
template <typename XT>
bs_status launch_allu_gain_dx(const AlluGainDxArgs<XT>& a, hipStream_t st);

// D use (Eq. dterm): per head-major row, rowsum(ddO * O_D) + rowsum(dO * (O_D - O)), O_D what the
// letter reads of the attention output (rd.x = O head-major), ddO nullable.
struct AlluDArgs {
  StoreRead rd;
  const float* dO;   // [rows][64] the reference incoming gradient at the D use
  const float* ddO;  // nullable [rows][64], or with ddo_heads > 0 token-major [B][S][ddo_heads 64]
  int64_t rows;
  float* out;        // [rows]
  uint32_t* amax = nullptr;  // nullable: slots (AMAX_SLOTS) raised to max |out|
  int ddo_heads = 0, ddo_S = 0;  // ddO token-major: heads and sequence length (row = (b H + h) S + s)
};
bs_status launch_allu_d(const AlluDArgs& a, hipStream_t st);

// mean of K trials from shifted sums: out = d1 + S1 / K
bs_status launch_trial_mean(const float* d1, const double* S1, int K, int64_t m, float* out, hipStream_t st);
// out[i] = v for n floats (any v, NaN included)
bs_status launch_fill(float* out, int64_t n, float v, hipStream_t st);

}  // namespace bsp
