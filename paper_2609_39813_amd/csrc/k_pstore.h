// Argument block and launchers of the FP8 store of attention probabilities and its two uses
// (dh = 64): the gradient of V and the softmax's backward, each reading the original, the
// forward's rounding or new roundings (App. B.2-B.4).
#pragma once
#include "bsp_kernels.h"

namespace bsp {

// Bias fields, each a [q][k] tile set (tile-major, see PstoreArgs::fld):
//   softmax's backward ds - J(p) dp for the reads R J(p_q), N J(a), K K(a), J2 J2(a, b),
//   Q2 J2(p_q, a); F_REF holds the reference ds = J(p) dp itself; at the gradient of V,
//   V_U holds p - p_q and V_N the mean over trials of a minus p_q.
enum { PF_REF = 0, PF_R, PF_N, PF_K, PF_J2, PF_Q2, PF_VU, PF_VN, PF_COUNT };
constexpr int PF_SOFTMAX = 6;   // PF_REF .. PF_Q2 enter dQ and dK
constexpr int PSTORE_KMAX = 32; // trials per call (their per-row sums live in registers)
constexpr int PSTORE_T = 64;     // head dimension, and the side of a score tile
constexpr int PSTORE_RC = 16;    // trials per walk of the row-sum pass (16 bits of up-decisions)

// 64 x 64 tiles per head of a bias field: the tiles (qb, kb) on or below the diagonal when
// causal (kb <= qb, row-major within the triangle), else all nqb^2
inline __host__ __device__ int64_t pstore_tiles(int nqb, int causal) {
  return causal ? (int64_t)nqb * (nqb + 1) / 2 : (int64_t)nqb * nqb;
}

constexpr int PSTORE_MAXPOL = 8;

// one gradient's per-policy outputs [BH][S][64] each (nullable)
struct PstoreOut {
  float* mean[PSTORE_MAXPOL];
  float* bias[PSTORE_MAXPOL];
};

struct PstoreArgs {
  const u16 *Q, *K, *V, *dO;        // [BH][S][64] bf16
  const u16 *Qt, *Kt, *Vt, *dOt;    // transposed copies [BH][64][Sp] (zero past S)
  int S, Sp, causal, BH;
  float scale;                      // softmax scale c
  const float* scale_mul;           // null (the scores' scale is c)
  const float *m, *l;               // row max of c log2(e) S and row sum, [BH][S]
  F8 f;
  int fmt, fwd_mode;
  uint64_t seed;
  uint32_t use_fwd, use_a, use_b;   // the forward's rounding (trial 0); new roundings a, b (trials 1..K)
  int ntrial;                       // K, the number of new roundings per use
  bs_diag* diag;                    // scale, amax, saturations of the store
  float* P_scale;                   // nullable: [1] copy of the store's scale
  uint8_t* codes;                   // [BH][S][S], zero above the causal diagonal
  float* P_out;                     // nullable: the realized fp32 probabilities [BH][S][S]
  float* O;                         // [BH][S][64] forward output p_q V
  float *D, *DR, *E, *Ee, *Ps1;     // per row (query) sums, [BH][S] (see launch_pstore_rows)
  float *Ga, *Ha, *Gb;              // per trial and row, [ntrial][BH][S]
  uint32_t* ubits;                  // up-decisions, per chunk c of jn <= 16 trials a plane of one word
                                    // per element (trial 16c + j: a at bit 2 (jn - 1 - j) + 1, b at
                                    // bit 2 (jn - 1 - j)), tiles as the fields, each tile's words
                                    // thread-major (16 per thread)
  int draw_a, draw_b;               // a policy reads new rounding a / b (else their draws are skipped)
  float* fld[PF_COUNT];             // [BH][pstore_tiles][64 k][64 q] fp32, tile by (query block, key block)
  float *dQ_ref, *dK_ref, *dV_ref;  // [BH][S][64]
  // the policies' estimates, written by the passes' epilogues: mean = reference + bias
  int n_pol;
  int sm_field[PSTORE_MAXPOL];      // bias field of the softmax read: PF_R .. PF_Q2, or PF_REF = none
  int v_field[PSTORE_MAXPOL];       // dV read: 0 none (R), 1 p - p_q (U), 2 mean a - p_q (N)
  PstoreOut dQ, dK, dV;
};

// amax = max over rows of 1 / l (the largest probability of each row), s = fl32(amax / FMAX)
bs_status launch_pstore_scale(const PstoreArgs& a, hipStream_t st);
// codes of P (and P_out) and O = p_q V
bs_status launch_pstore_fwd(const PstoreArgs& a, hipStream_t st);
// per-row sums over keys, with r = p_q - p, e = lo - p and h the grid step at p (real units):
// D = sum p dp, DR = sum r dp, E = sum e dp, Ee = sum e, Ps1 = sum p - 1; per trial k (u_k the
// up-decision of new rounding a, v_k of b): Ga = sum u_k h dp, Ha = sum u_k h, Gb = sum v_k h dp
bs_status launch_pstore_rows(const PstoreArgs& a, hipStream_t st);
// bias fields (stored for the key-major passes), dQ_ref and the policies' dQ estimates
bs_status launch_pstore_dq(const PstoreArgs& a, hipStream_t st);
// dK_ref and the policies' dK estimates, then dV_ref and their dV estimates, from the stored
// fields and codes
bs_status launch_pstore_dkv(const PstoreArgs& a, hipStream_t st);

}  // namespace bsp
