// The decoder layer's "every use at once" check: each letter U, R, N read at every use of every
// store in one backward, K trials for N (the forward held fixed), against the straight-through
// reference; the layer entry point runs it after the per-use check.
#pragma once
#include "bsp_kernels.h"

namespace bsp {

// The layer's realized forward, reference backward and per-use results the check starts from.
struct AlluIO {
  int B, S, d, H, F, K;
  float eps;
  int fmt;
  uint64_t seed;
  const u16* x;            // [T][d] bf16
  const float *gain1, *gain2;
  const u16 *Wqkv, *Wo, *Wgu;  // [d][3d], [d][d], [d][2F] bf16
  const u16 *Q, *Kk, *V;   // [B][H][S][64] bf16
  const float *O, *Otok, *h, *a;  // O head-major, O token-major, h [T][d], a [T][F]
  const uint8_t *c_u1, *c_O, *c_Otok, *c_u2, *c_a;
  const float* scales;     // [4] u1, O, u2, a
  // the per-use check's normalization operands: u1, u2 [T][d], their inverse rms [T], and du at
  // u1 and u2 (dQKV Wqkv^T, [dg | dhh] Wgu^T) [T][d]
  const float *u1, *u2, *r1, *r2, *du1, *du2;
  const float *dgh, *dh, *dOh, *dqkv;  // reference incoming gradients: [T][2F], [T][d], head-major [T][d], [T][3d]
  // the reference gradients and the per-use biases of the uses whose incoming gradient is the
  // reference's whatever the letter (their means over the same draws are the per-use ones)
  const float *ref[8];     // dx, dgain1, dWqkv, dWo, dgain2, dWg|dWu ([d][2F]), -, dWd
  const float* wd_bias;    // [3][F*d]
  const float* wgu_bias;   // [3][d*2F]
  const float* g2_bias;    // [3][d]
  const float* g2_se;      // [3][d]
  // outputs (each nullable): per letter, bias and se of dx, dgain1, dWqkv, dWo, dgain2, dWg, dWu, dWd
  float* bias[3][8];
  float* se[3][8];
  double* table;           // [8][3][3] (nullable)
};

size_t allu_ws_size(int B, int S, int d, int H, int F, int K);
bs_status allu_run(const AlluIO& io, void* ws, size_t ws_bytes, hipStream_t st);

}  // namespace bsp
