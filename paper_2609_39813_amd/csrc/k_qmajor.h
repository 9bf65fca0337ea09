// The query-major scaffold of the attention passes that re-form P tile by tile (dh = 64): the
// lane of a 64-query block that owns one query and 16 keys of each key block, P and dP of those
// keys by MFMA, and the element / tile indexing. The argument block A provides Q, dO, m, l (the
// forward's row max of c log2(e) S and row sum), S, Sp, causal, scale and scale_mul.
#pragma once
#include "k_attn_tiles.h"

namespace bsp {

// 64 x 64 tiles per head of a tile-major array: on or below the diagonal when causal
inline __host__ __device__ int64_t causal_tiles(int nqb, int causal) {
  return causal ? (int64_t)nqb * (nqb + 1) / 2 : (int64_t)nqb * nqb;
}

// grid value (code's value) of an OCP FP8 code by the conversion instruction
template <int FMT>
__device__ __forceinline__ float f8_val(uint32_t word, int byte) {
  switch (byte) {
    case 0: return FMT == BS_E5M2 ? __builtin_amdgcn_cvt_f32_bf8((int)word, 0) : __builtin_amdgcn_cvt_f32_fp8((int)word, 0);
    case 1: return FMT == BS_E5M2 ? __builtin_amdgcn_cvt_f32_bf8((int)word, 1) : __builtin_amdgcn_cvt_f32_fp8((int)word, 1);
    case 2: return FMT == BS_E5M2 ? __builtin_amdgcn_cvt_f32_bf8((int)word, 2) : __builtin_amdgcn_cvt_f32_fp8((int)word, 2);
    default: return FMT == BS_E5M2 ? __builtin_amdgcn_cvt_f32_bf8((int)word, 3) : __builtin_amdgcn_cvt_f32_fp8((int)word, 3);
  }
}

// Block (bh, query block): wave w's lane (g, c16) owns query q = q0 + 16 w + c16 and, within a
// key block, the keys k0 + 16 t + 4 g + r (t, r < 4).
struct QMajor {
  int bh, qb, q0, q, w, g, c16;
  bool qok;
  int64_t hb, tb, rb;
  float mq, ilq;
  bf16x8 fq[2], fdo[2];
};

template <typename A>
__device__ __forceinline__ QMajor qmajor_setup(const A& a, bool need_do) {
  QMajor z;
  const int lane = threadIdx.x & 63;
  z.w = threadIdx.x >> 6;
  z.g = lane >> 4;
  z.c16 = lane & 15;
  z.bh = blockIdx.x;
  z.qb = a.causal ? (int)gridDim.y - 1 - (int)blockIdx.y : (int)blockIdx.y;  // heaviest first
  z.q0 = z.qb * AT;
  z.q = z.q0 + 16 * z.w + z.c16;
  z.qok = z.q < a.S;
  z.hb = (int64_t)z.bh * a.S * AT;
  z.tb = (int64_t)z.bh * AT * a.Sp;
  z.rb = (int64_t)z.bh * a.S;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int64_t e = z.hb + (int64_t)z.q * AT + 32 * s + 8 * z.g;
    z.fq[s] = __builtin_bit_cast(bf16x8, z.qok ? *(const uint4*)(a.Q + e) : make_uint4(0, 0, 0, 0));
    z.fdo[s] = __builtin_bit_cast(bf16x8, (need_do && z.qok) ? *(const uint4*)(a.dO + e) : make_uint4(0, 0, 0, 0));
  }
  z.mq = z.qok ? a.m[z.rb + z.q] : 0.0f;
  z.ilq = z.qok ? 1.0f / a.l[z.rb + z.q] : 0.0f;
  return z;
}

// p of the lane's 16 keys of key block k0 (tK: K rows of the block in LDS)
template <typename A>
__device__ __forceinline__ void probs(const A& a, const QMajor& z, const u16* tK, int k0, float (&p)[4][4]) {
#pragma clang fp contract(off)  // x = fl(c log2(e) s) is rounded before m is subtracted
  floatx4 sv[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) sv[t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int t = 0; t < 4; ++t) sv[t] = mfma(*(const bf16x8*)(tK + sw(16 * t + z.c16, 32 * s + 8 * z.g)), z.fq[s], sv[t]);
  const float c2 = scores_scale(a.scale, a.scale_mul) * kLog2e;
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int key = k0 + 16 * t + 4 * z.g + r;
      const bool ok = z.qok && key < a.S && (!a.causal || key <= z.q);
      const float x = c2 * sv[t][r];
      p[t][r] = ok ? __builtin_amdgcn_exp2f(x - z.mq) * z.ilq : 0.0f;
    }
}

// dp = dO . v_key of the lane's query and 16 keys (tV: V rows of the block in LDS)
__device__ __forceinline__ void dprobs(const QMajor& z, const u16* tV, float (&dp)[4][4]) {
  floatx4 dv[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) dv[t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int t = 0; t < 4; ++t) dv[t] = mfma(*(const bf16x8*)(tV + sw(16 * t + z.c16, 32 * s + 8 * z.g)), z.fdo[s], dv[t]);
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) dp[t][r] = dv[t][r];
}

// the element index of P[bh][q][key] (a multiple of 4 for key = 16 t + 4 g, since S % 4 == 0)
template <typename A>
__device__ __forceinline__ uint64_t pelem(const A& a, const QMajor& z, int key) {
  return ((uint64_t)z.rb + (uint64_t)z.q) * (uint64_t)a.S + (uint64_t)key;
}

// first element of the tile (query block qb, key block kb) of head bh in a tile-major [BH][tiles][64][64]
// array (causal: the tiles on or below the diagonal, row-major within the triangle)
template <typename A>
__device__ __forceinline__ int64_t fld_tile(const A& a, int bh, int qb, int kb, int nqb) {
  const int64_t per = causal_tiles(nqb, a.causal);
  const int64_t t = a.causal ? (int64_t)qb * (qb + 1) / 2 + kb : (int64_t)qb * nqb + kb;
  return ((int64_t)bh * per + t) * AT * AT;
}

}  // namespace bsp
