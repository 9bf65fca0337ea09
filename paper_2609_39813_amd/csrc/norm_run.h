// The normalization-store runner shared by the C-ABI entry and the decoder layer.
#pragma once
#include "bsp_kernels.h"

namespace bsp {

struct NormIO {
  const void* X;       // [T][d], dtype xt
  bs_dtype xt;
  const float* gain;   // [d]
  const void* W;       // [d][n], dtype wt
  bs_dtype wt;
  const void* dY;      // [T][n], dtype gt; nullptr: forward only (u_codes, u_scale, Y)
  bs_dtype gt;
  int64_t T, d, n;
  float eps;
  int fmt, fwd_mode;
  const bs_norm_policy* pol;
  int n_pol, K;
  uint64_t seed;
  uint32_t store_id;
  float* Y;
  uint8_t* u_codes;
  float* u_scale;
  float *dgain_ref, *dW_ref, *dX_ref;
  bs_est dgain, dW, dX;
  bs_diag* diag;
  float* u_out = nullptr;     // optional: the fp32 quantizer input u [T][d]
  float* rstd_out = nullptr;  // optional: the inverse rms per row [T]
  float* du_out = nullptr;    // optional: the incoming gradient at u, du = dY W^T [T][d]
};

size_t norm_ws_size(int64_t T, int64_t d, int64_t n, int K);
bs_status norm_run(const NormIO& io, void* ws, size_t ws_bytes, hipStream_t st);

}  // namespace bsp
