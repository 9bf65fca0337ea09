// Argument blocks and launchers of the attention kernels (dh = 64).
#pragma once
#include "bsp_kernels.h"

namespace bsp {

constexpr int ATTN_MAX_POL = 8;

struct AttnArgs {
  const u16 *Q, *K, *V;  // [B*H][S][64] bf16
  int S, causal;
  float scale;
  float* m;      // [B*H][S] row max of c log2(e) S
  float* l;      // [B*H][S] row sum of 2^(c log2(e) S - m)
  float* O_out;  // nullable [B*H][S][64] fp32
  const u16* Vt; // V^T [B*H][64][Sp] (zero past S), from launch_attn_transpose
  int Sp;
  const float* scale_mul;  // nullable device [1]: the scores' scale is scale * scale_mul[0]
};

struct AttnDArgs {
  const float* O;         // original output, fp32
  const u16* dO;          // bf16 (used when dO32 is null)
  const float* dO32;      // nullable: fp32 incoming gradient
  const uint8_t* codes;   // forward's store of O
  const float* scale;     // device s
  int64_t rows;           // B*H*S
  F8 f;
  uint64_t seed;
  uint32_t use;           // new roundings' use id
  int K, want_n;
  float *D_ref, *dD_R, *dD_N, *sd_N;  // [rows]
  float* dD_trials = nullptr;         // nullable [K][rows]: each trial's dD_k (want_n)
};

// Level-2 averaging at the D use: trial k rounds O anew (trial k, use_fwd) and its incoming
// gradient is g_k = dO + beta r_k, r_k the forward's rounding error; a new rounding r'_k uses
// (trial k, use_n). Per row: the means over trials of D_ref and of the R and N errors, their
// mean-error parts, couplings and se, and the paired statistic T; per element the mean g.
struct AttnL2Args {
  const float* O;         // original output, fp32 [rows][64]
  const u16* dO;          // bf16 [rows][64]
  const float* scale;     // device s of the store
  int64_t rows;
  F8 f;
  int fwd_mode;
  uint64_t seed;
  uint32_t use_fwd, use_n;
  int K;
  float beta;
  float* dO_mean;         // [rows][64] mean incoming gradient
  float *D_ref, *dD_R, *dD_N;  // [rows] means over trials
  float *stat_R, *stat_N; // nullable [4][rows]: mean error, its mean-error part, coupling, se
  float* T;               // nullable [2][rows]: mean and se of the paired statistic
};

struct AttnBwdArgs {
  const u16 *Q, *K, *V, *dO;
  const float* dO32;  // nullable: fp32 incoming gradient (enters as three exact bf16 terms)
  // operand copies written by launch_attn_prep: Q^T, K^T [B*H][64][Sp] and the incoming
  // gradient's planes (row-major [B*H][S][64], only for an fp32 gradient) and their transposes
  const u16 *Qt, *Kt;
  const u16* dOp[3];
  const u16* dOt[3];
  int Sp;
  const float *m, *l, *D_ref, *dD_R, *dD_N, *sd_N;  // dD_R / dD_N / sd_N nullable
  int S, causal, ntrial;  // ntrial: K, the number of new roundings
  float scale;
  float *dQ_ref, *dK_ref, *dV;
  int n_pol;
  int pol[ATTN_MAX_POL];
  float* mean[ATTN_MAX_POL];   // dQ estimates, already offset per policy
  float* bias[ATTN_MAX_POL];
  float* se[ATTN_MAX_POL];
  float* kmean[ATTN_MAX_POL];  // dK estimates
  float* kbias[ATTN_MAX_POL];
  int k_only = 0;              // 1: the key-major pass only (dK, dV and their estimates)
  // fp16 operands (no policies, no dD): with V16 non-null, dOp[0..1] and dOt[0..1] hold the
  // two-term fp16 split of dO 2^e (launch_attn_split_f16), V16 = fp16(V 2^f) [B*H][S][64], Qt16
  // and Kt16 the transposed copies of fp16(Q 2^q) and fp16(K 2^k); dS enters as its two-term
  // split at the scale 2^s of launch_attn_f16_scales. f16_inv (device) = {2^-e, 2^-f, 2^-q, 2^-k,
  // 2^s, 2^-s-q, 2^-s-k}.
  const u16* V16 = nullptr;
  const u16 *Qt16 = nullptr, *Kt16 = nullptr;
  const float* f16_inv = nullptr;
  uint32_t* amax = nullptr;  // nullable: slots (AMAX_SLOTS) raised to max |.| of dQ_ref, dK_ref, dV
};

bs_status launch_attn_fwd(const AttnArgs& a, int B, int H, hipStream_t st);
bs_status launch_attn_d(const AttnDArgs& a, hipStream_t st);
bs_status launch_attn_l2(const AttnL2Args& a, hipStream_t st);
// X_i^T [BH][64][Sp] (zero past S) of n <= 4 bf16 X_i [BH][S][64] (16-byte aligned)
bs_status launch_attn_transpose(const u16* const* X, u16* const* Xt, int n, int BH, int S, int Sp, hipStream_t st);
// the three bf16 planes of an fp32 incoming gradient [BH][S][64] and their transposes
bs_status launch_attn_split(const float* dO32, int BH, int S, int Sp, u16* const* dOp, u16* const* dOt,
                            hipStream_t st);
// the two fp16 planes (split2_f16) of dO32 2^e, e from the max in slots (an AMAX_SLOTS array,
// f16_scale_exp), and their transposes (head-major [BH][S][64] planes); 2^-e to inv_out. dO32 is
// head-major, or with htok > 0 token-major [BH / htok][S][htok 64] (htok heads)
bs_status launch_attn_split_f16(const float* dO32, int BH, int S, int Sp, int htok, const uint32_t* slots,
                                float* inv_out, u16* const* dOp, u16* const* dOt, hipStream_t st);
// dS's scale of the fp16 backward (f16_inv above, entries 4..6 from entries 2, 3): 2^s from the
// bound 64 max|dO| max|V| + max|D| of |dS| = P |dP - D| (P <= 1, 64 terms per dP), the maxima
// held in the slot arrays (AMAX_SLOTS) sdO, sV, sD
bs_status launch_attn_f16_scales(const uint32_t* sdO, const uint32_t* sV, const uint32_t* sD, float* f16_inv,
                                 hipStream_t st);
bs_status launch_attn_bwd(const AttnBwdArgs& a, int B, int H, hipStream_t st);

}  // namespace bsp
