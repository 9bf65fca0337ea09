// The fused multi-policy combine of a gradient's estimates (launch in k_norm.hip).
#pragma once
#include "bsp_kernels.h"

namespace bsp {

// Every policy's estimate of one gradient in one pass over its reference: policy p writes
// mean_p = ref + bias_p (or alt_p, with bias_p = alt_p - ref, when alt_p is set), bias_p and se_p
// at offset p n of the nullable output bases (inputs bias_p / se_p nullable = 0).
constexpr int COMBINE_MAX_POL = 16;
struct CombineMulti {
  const float* ref;
  int n_pol, vec;
  const float* bias[COMBINE_MAX_POL];
  const float* se[COMBINE_MAX_POL];
  const float* alt[COMBINE_MAX_POL];
  float *mean, *bias_out, *se_out;  // bases of [n_pol][n] outputs (nullable)
};
bs_status launch_combine_multi(CombineMulti c, int64_t n, hipStream_t st);

}  // namespace bsp
