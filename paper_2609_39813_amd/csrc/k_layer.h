// Launchers of the decoder layer's elementwise kernels.
#pragma once
#include "bsp_kernels.h"

namespace bsp {

bs_status launch_qkv_heads(const float* qkv, int B, int S, int H, int dh, u16* Q, u16* K, u16* V, hipStream_t st);
bs_status launch_heads_tokens_f32(const float* in, float* out, int B, int S, int H, int dh, bool to_tokens,
                                  hipStream_t st);
bs_status launch_heads_tokens_u8(const uint8_t* in, uint8_t* out, int B, int S, int H, int dh, hipStream_t st);
bs_status launch_dqkv_tokens(const float* dQ, const float* dK, const float* dV, float* out, int B, int S, int H,
                             int dh, hipStream_t st);
bs_status launch_bf16_to_f32(const u16* in, float* out, int64_t n, hipStream_t st);
bs_status launch_concat_cols(const u16* A, const u16* B, u16* out, int64_t rows, int64_t c1, int64_t c2,
                             hipStream_t st);
bs_status launch_split_cols(const float* in, float* A, float* B, int64_t rows, int64_t c, hipStream_t st);
bs_status launch_swiglu_fwd(const float* gh, float* a, int64_t T, int64_t F, hipStream_t st);
bs_status launch_swiglu_bwd(const float* da, const float* gh, float* dgh, int64_t T, int64_t F, hipStream_t st);
bs_status launch_add(const void* a, bs_dtype at, const float* b, float* out, int64_t n, hipStream_t st);
// Batched sums of squares (fp64, fixed order): job i writes sum x^2 over n floats to out, or
// NaN (x == nullptr, n == 0) or 0 (x == nullptr, n == 1). Two launches for the whole batch.
constexpr int SUMSQ_MAX = 96, SUMSQ_BLOCKS = 256;
struct SumsqJob {
  const float* x;
  int64_t n;
  double* out;
};
struct SumsqBatch {
  SumsqJob job[SUMSQ_MAX];
  int count;
  int row[SUMSQ_MAX];  // set by launch_sumsq_batch: the partial-sum row of each job (jobs on the
                       // same array and length share one)
};
inline size_t sumsq_part_size() { return (size_t)SUMSQ_MAX * SUMSQ_BLOCKS; }  // doubles
bs_status launch_sumsq_batch(const SumsqBatch& b, double* part, hipStream_t st);

}  // namespace bsp
