// The attention runner shared by the C-ABI entry and the decoder layer.
#pragma once
#include "bsp_kernels.h"

namespace bsp {

struct AttnIO {
  const void *Q, *Kt, *V;   // [B,H,S,64] bf16
  const void* dO;           // bf16 [B,H,S,64]; or
  const float* dO32;        // fp32 [B,H,S,64]; both null: forward and store only
  int B, H, S, dh, causal;
  float scale;
  const float* O;           // nullable: the original output to store
  int fmt, fwd_mode;
  const bs_read* pol;
  int n_pol, K;
  uint64_t seed;
  uint32_t store_id;
  float* O_out;
  uint8_t* O_codes;
  float* O_scale;
  float *dQ_ref, *dK_ref, *dV, *D_ref;
  bs_est dQ, dK;
  bs_diag* diag;
  // level-2 averaging (the forward's rounding resampled per trial, incoming gradient
  // dO + beta r_k; dO bf16 only): the D use's split per policy [n_pol][4][B*H*S] (nullable),
  // the paired statistic [2][B*H*S] (nullable), the mean incoming gradient (nullable)
  int level2 = 0;
  float beta = 0.0f;
  float* d_use = nullptr;
  float* T = nullptr;
  float* dO_mean = nullptr;
};

// K and dk_se size the per-trial path of dK's se (K trials of the key-major pass under N)
size_t attn_ws_size(int B, int H, int S, int dh, int K = 1, bool dk_se = false);
bs_status attn_run(const AttnIO& io, void* ws, size_t ws_bytes, hipStream_t st);

}  // namespace bsp
