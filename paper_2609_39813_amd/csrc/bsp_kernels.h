// Internal launchers of the gfx950 kernels (host-callable, enqueue on a stream).
#pragma once
#include "bsp_common.h"

namespace bsp {

constexpr int GEMM_MAX_SEG = 8;
struct GemmArgs {
  const u16* A[GEMM_MAX_SEG];
  const u16* B[GEMM_MAX_SEG];
  int nseg;
  int M, N, K;
  int64_t lda, ldb, ldc;
  float alpha;
  const float* alpha_dev;  // nullable: alpha is multiplied by *alpha_dev
  int accumulate;
  float* C;
  float* part = nullptr;    // nullable: split-K partials, part_cap floats (device workspace)
  int64_t part_cap = 0;
  int nprod = 0;            // distinct products among the segments (split terms of one product
                            // count once); 0: every segment is a product of its own
  int f16 = 0;              // 1: every operand holds fp16 values (the 2-term fp16 split), else bf16
  const float* alpha_dev2 = nullptr;  // nullable: a second device multiplier of alpha
  uint32_t* amax = nullptr;  // nullable: slots (AMAX_SLOTS) raised to max |C| of the values written
                             // (C's new values, accumulate = 0 only; the pipelined kernel only)
  // batch > 1: that many independent contractions, z = 0 .. batch - 1, each with every segment's
  // A and B offset by z sA, z sB elements, C by z sC and alpha_dev2 by z s_alpha2 (no split-K;
  // the pipelined kernel only)
  int batch = 1;
  int64_t sA = 0, sB = 0, sC = 0, s_alpha2 = 0;
};

// alpha of a launch (batch member z) with its device multipliers
__device__ __forceinline__ float gemm_alpha(const GemmArgs& g, int z = 0) {
  float a = g.alpha;
  if (g.alpha_dev) a *= *g.alpha_dev;
  if (g.alpha_dev2) a *= g.alpha_dev2[(int64_t)z * g.s_alpha2];
  return a;
}

// algorithmic flop of a contraction launch: 2 M N K per distinct product
inline double gemm_flops(const GemmArgs& g) {
  return 2.0 * g.M * g.N * (double)g.K * (g.nprod > 0 ? g.nprod : g.nseg) * g.batch;
}
// flop the matrix cores execute: 2 M N K per segment (every bf16 term of a split operand)
inline double gemm_exec_flops(const GemmArgs& g) { return 2.0 * g.M * g.N * (double)g.K * g.nseg * g.batch; }

// Append the products A_i B_j (i + j <= maxsum) of nA and nB bf16 terms to g's segments: with
// three-term splits the products of order 2^-24 and above (maxsum 2); with two-term fp16 splits
// (one exact term against two, or two against two with maxsum 1) those of order 2^-22 and above.
inline bool gemm_add_products(GemmArgs& g, const u16* const* A, int nA, const u16* const* B, int nB,
                              int maxsum = 2) {
  if (g.nprod == 0 && g.nseg > 0) g.nprod = g.nseg;  // segments set before: one product each
  ++g.nprod;
  for (int s = 0; s <= maxsum; ++s)
    for (int i = 0; i < nA; ++i) {
      const int j = s - i;
      if (j < 0 || j >= nB) continue;
      if (g.nseg >= GEMM_MAX_SEG) return false;
      g.A[g.nseg] = A[i];
      g.B[g.nseg] = B[j];
      ++g.nseg;
    }
  return true;
}

bs_status launch_gemm(const GemmArgs& g, hipStream_t st);

// Records HIP events around a kernel launch while profiling is enabled (bs_profile_enable).
// `work` is the launch's algorithmic work (flop for a contraction) and `exec` the work its units
// execute (flop of every split term), summed by bs_profile_work.
class ProfScope {
 public:
  ProfScope(const char* name, hipStream_t st, double work = 0.0, double exec = 0.0);
  ~ProfScope();

 private:
  const char* name_;
  hipStream_t st_;
  double work_, exec_;
  hipEvent_t a_, b_;
};

bs_status launch_store(const void* x, bs_dtype xt, int64_t n, int fmt, int mode, uint64_t seed, uint32_t trial,
                       uint32_t use, const float* scale_in, uint8_t* codes, float* scale_out, bs_diag* diag,
                       hipStream_t st, bool amax_done);
enum { FC_COUNT = 0, FC_COLSUM = 1, FC_BLOCKSUM = 2 };
template <typename X>
struct FreshArgs {
  const X* x;          // [T][d] values to round (fp32 or bf16), scaled by 1/s
  int64_t T, d;
  F8 f;
  const float* scale;  // device s
  uint64_t seed;
  uint32_t use;
  int K;
  u16* counts;         // [T][d] up counts (nullable)
  const float* w1;     // [T][d] weights (FC_COLSUM, FC_BLOCKSUM)
  const float* w2;     // [T][d] second weight (FC_BLOCKSUM, nullable)
  double* partial;     // FC_BLOCKSUM: [K][2][nblocks]
  float* colsum = nullptr;  // FC_COLSUM: [K][ceil(T/32)][d]
  int trial0 = 1;      // the K trials are trial0 .. trial0 + K - 1
};
template <typename X>
bs_status launch_fresh_count_t(const FreshArgs<X>& a, int mode, hipStream_t st);
inline int64_t fresh_count_blocks(int64_t T, int64_t d) { return ((d + 255) / 256) * ((T + 31) / 32); }

bs_status launch_fresh_count(const float* u, int64_t T, int64_t d, int fmt, const float* scale, uint64_t seed,
                             uint32_t use, int K, u16* counts, const float* w, float* colsum, hipStream_t st);

bs_status launch_combine(const float* ref, const float* bias, const float* se, int64_t n, float* mean_out,
                         float* bias_out, float* se_out, hipStream_t st);

bs_status launch_fill2d(float* p, int64_t rows, int64_t cols, int64_t ld, float v, hipStream_t st);
bs_status launch_fill_f64(double* p, int64_t n, double v, hipStream_t st);
// *out (the float bits of a maximum, zeroed by the caller) raised to max |x[i]| over n floats;
// with the other AMAX_SLOTS - 1 slots zeroed, out is a slot array
bs_status launch_amax_f32(const float* x, int64_t n, uint32_t* out, hipStream_t st);
bs_status launch_amax_bf16(const u16* x, int64_t n, uint32_t* out, hipStream_t st);
bs_status launch_init_diag(bs_diag* diag, hipStream_t st);

// bf16 operand planes. Row-major: out_p[r*ldo + c], c < C (ldo >= C). Transposed:
// out_p[c*ldo + r], r < R, zero for R <= r < ldo. p = 0..nterms-1 (terms of the
// split of each fp32 value; bf16 inputs with nterms == 1 are copied).
bs_status launch_planes(const void* in, bs_dtype dt, int64_t R, int64_t C, int64_t ldi, bool transpose,
                        u16* const* out, int nterms, int64_t ldo, float scale, hipStream_t st);
// The scale 2^e of a two-term fp16 split (bsp_common.h f16_scale_exp) from maxima held as
// slots (AMAX_SLOTS words AMAX_STRIDE apart, float bits): the bound is amax_a's, or with amax_b
// the larger of the two and e one lower, so that a sum of the two tensors (and each alone)
// fits; inv_out (nullable) receives 2^-e, the contraction's multiplier.
struct F16Scale {
  const uint32_t* amax_a = nullptr;
  const uint32_t* amax_b = nullptr;
  float* inv_out = nullptr;
};
// A move tensor seen as a token-major [R][C] fp32 matrix: rows[t*ldi + c], or (rows null) the
// head-major [B][H][S][64] arrays heads[c / d] (Q, K, V gradients; d = 64 H, R = B S).
struct MoveSrc {
  const float* rows = nullptr;
  int64_t ldi = 0;
  const float* heads[3] = {nullptr, nullptr, nullptr};
  int64_t S = 0, H = 0, d = 0;
};
// The scaled two-term fp16 planes (scale from sc, F16Scale) of a move m, from one read: tM =
// transposed planes of m (tM_p[c*ldo + r], rows R..ldo zero), tS (with base non-null) those of
// base + m (base [R][C] with leading dimension ldb), rows (nullable) the row-major planes
// rows_p[r*ldr + c]. Needs C and the leading dimensions multiples of 4 (ldo of 64, ldo >= R),
// 16-byte aligned inputs and transposed planes, 8-byte aligned row planes (BS_EINVAL otherwise).
bs_status launch_split_move(const MoveSrc& m, const float* base, int64_t ldb, int64_t R, int64_t C, F16Scale sc,
                            u16* const* tM, u16* const* tS, int64_t ldo, u16* const* rows, int64_t ldr,
                            hipStream_t st);
// out = fp16(in 2^e) of a bf16 tensor with e = f16_scale_exp of the max held in slots (an
// AMAX_SLOTS array), 2^-e to inv_out (nullable). Exact where |in| 2^e >= 2^-17 (fp16 subnormal
// spacing); below, the error is at most 2^-25 2^-e.
bs_status launch_scale_f16(const u16* in, int64_t n, const uint32_t* slots, u16* out, float* inv_out, hipStream_t st);

// Trial statistics over per-trial rows (App. C.4, App. D.4).
bs_status launch_policy_bias(const float* delta, int K, int64_t m, const float* g_ref, float* mean_err, float* se,
                             double* summary, double* ws, hipStream_t st);

}  // namespace bsp
