// Tile helpers of the attention kernels (dh = 64): LDS tile layouts, MFMA operand fragments,
// exact three-term bf16 splits and the register-staged tile copies.
//
// All tiles are 64 x 64 bf16 in LDS with rows of 128 B whose 16-byte chunks are XOR-swizzled
// by (row & 7); MFMA 16x16x32 bf16 operands are read as 16-byte fragments: lane l takes row
// r0 + (l & 15), columns k0 + 8 (l >> 4) .. + 7. A 16x16 result tile holds D[4 (l >> 4) + r]
// [l & 15] in register r of lane l.
#pragma once
#include "bsp_kernels.h"

namespace bsp {

// the scores' scale c of an argument block with an optional device multiplier (FP8 operands
// whose scales are applied after the products); the same fp32 product wherever P is formed
__device__ __forceinline__ float scores_scale(float c, const float* mul) { return mul ? c * mul[0] : c; }

constexpr int AT = 64;  // block rows / keys, and dh

__device__ __forceinline__ int sw(int row, int col) { return row * AT + ((((col >> 3) ^ (row & 7)) << 3) | (col & 7)); }

__device__ __forceinline__ floatx4 mfma(bf16x8 a, bf16x8 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
// the same product of operands that hold fp16 values
__device__ __forceinline__ floatx4 mfma_h(bf16x8 a, bf16x8 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(halfx8, a), __builtin_bit_cast(halfx8, b), c, 0, 0,
                                                0);
}

// P = 2^(c log2(e) S - m) / l with m the row max of c log2(e) S: one hardware exp2 per
// element (a few ulps; the exponent's rounding adds |m| 2^-24, below 1e-6 for these scores)
constexpr float kLog2e = 1.4426950408889634f;

// Transposed copies X^T [64][Sp] store each 64-column tile in fragment order: column e of a
// tile holds tile row tperm(e) of X, e = 32 s + 8 g + j -> 32 s + 4 g + (j & 3) + 16 (j >> 2).
// The eight k values of an operand fragment built from a 16x16 result tile pair (result rows
// 32 s + 4 g + 0..3 and 32 s + 16 + 4 g + 0..3, lane group g) are then one 16-byte chunk.
__device__ __forceinline__ int tperm(int e) { return (e & 32) | ((e >> 1) & 12) | (e & 3) | ((e & 4) << 2); }

// B operand of X^T stored in LDS (sw layout): row `row`, the k values of half s, lane group g
__device__ __forceinline__ bf16x8 frag_t(const u16* T, int row, int s, int g) {
  return *(const bf16x8*)(T + sw(row, 8 * (4 * s + g)));
}

// the three bf16 terms (round to nearest, then the exact remainders) of eight fp32 values as
// MFMA operands, converted two at a time into packed registers
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pk_bf16(float a, float b) {
  const bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ float lo_f32(uint32_t p) { return __uint_as_float(p << 16); }
__device__ __forceinline__ float hi_f32(uint32_t p) { return __uint_as_float(p & 0xFFFF0000u); }
__device__ __forceinline__ void pack3(const float* v, bf16x8* t) {
  uint32_t w[3][4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float a = v[2 * i], b = v[2 * i + 1];
    const uint32_t p0 = pk_bf16(a, b);
    const float ra = a - lo_f32(p0), rb = b - hi_f32(p0);
    const uint32_t p1 = pk_bf16(ra, rb);
    const float sa = ra - lo_f32(p1), sb = rb - hi_f32(p1);
    w[0][i] = p0;
    w[1][i] = p1;
    w[2][i] = pk_bf16(sa, sb);
  }
#pragma unroll
  for (int p = 0; p < 3; ++p) t[p] = __builtin_bit_cast(bf16x8, make_uint4(w[p][0], w[p][1], w[p][2], w[p][3]));
}

// The same exact three-term split by truncation: each term is the high half of what the
// previous ones leave (a byte permute packs two), no conversions. Terms of one sign, the
// second below 2^-7 and the third below 2^-15 of the value.
__device__ __forceinline__ uint32_t hi_pair(float a, float b) {
  return __builtin_amdgcn_perm(__float_as_uint(b), __float_as_uint(a), 0x07060302u);
}
__device__ __forceinline__ float cut_hi(float a) { return a - __uint_as_float(__float_as_uint(a) & 0xFFFF0000u); }
__device__ __forceinline__ void pack3t(const float* v, bf16x8* t) {
  uint32_t w[3][4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float a = v[2 * i], b = v[2 * i + 1];
    const float ra = cut_hi(a), rb = cut_hi(b);
    w[0][i] = hi_pair(a, b);
    w[1][i] = hi_pair(ra, rb);
    w[2][i] = hi_pair(cut_hi(ra), cut_hi(rb));
  }
#pragma unroll
  for (int p = 0; p < 3; ++p) t[p] = __builtin_bit_cast(bf16x8, make_uint4(w[p][0], w[p][1], w[p][2], w[p][3]));
}

// The two-term fp16 split (bsp_common.h split2_f16) of eight fp32 values below 2^15 in magnitude.
// Pairs go through the packed conversion (hi of two values in one instruction, round to nearest
// even); the remainders are exact in fp32 and rounded as a pair again.
typedef float floatx2_t __attribute__((ext_vector_type(2)));
typedef _Float16 halfx2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void pack2h(const float* v, bf16x8* t) {
  uint32_t w[2][4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const floatx2_t x = {v[2 * i], v[2 * i + 1]};
    const halfx2_t h = __builtin_convertvector(x, halfx2_t);
    halfx2_t l;
    l.x = (_Float16)(x.x - (float)h.x);
    l.y = (_Float16)(x.y - (float)h.y);
    w[0][i] = __builtin_bit_cast(uint32_t, h);
    w[1][i] = __builtin_bit_cast(uint32_t, l);
  }
#pragma unroll
  for (int p = 0; p < 2; ++p) t[p] = __builtin_bit_cast(bf16x8, make_uint4(w[p][0], w[p][1], w[p][2], w[p][3]));
}

// buffer resource over n_bytes from base: loads past the end read as zero
__device__ __forceinline__ __amdgpu_buffer_rsrc_t attn_rsrc(const u16* base, int64_t n_bytes) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, (int)n_bytes, 0x00020000);
}
// s_waitcnt with only a vector-memory count (lgkm and exp counts not awaited)
#define ATTN_WAIT_VM(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (((n) >> 4) << 14) | (7 << 4) | (15 << 8))
// every LDS access of this wave done, then a barrier without a memory fence (a fence would
// drain the loads in flight)
#define ATTN_LDS_BARRIER()                                                       \
  do {                                                                           \
    __builtin_amdgcn_s_waitcnt((15 | (3 << 14)) | (7 << 4)); /* lgkmcnt(0) */   \
    asm volatile("s_barrier" ::: "memory");                                      \
  } while (0)

// a row-major [64][64] bf16 tile (rows r0.. of a [*, 64] matrix with nrow rows, zeros past
// them) as two 16-byte pieces per thread, and its store into LDS
struct TileRegs {
  uint4 v[2];
};
__device__ __forceinline__ void tile_fetch(TileRegs& t, const u16* __restrict__ g, int r0, int nrow) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = (threadIdx.x >> 3) + 32 * i, c = (threadIdx.x & 7) * 8;
    t.v[i] = r0 + r < nrow ? *(const uint4*)(g + (int64_t)(r0 + r) * AT + c) : make_uint4(0, 0, 0, 0);
  }
}
__device__ __forceinline__ void tile_put(u16* T, const TileRegs& t) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = (threadIdx.x >> 3) + 32 * i, c = (threadIdx.x & 7) * 8;
    *(uint4*)(T + sw(r, c)) = t.v[i];
  }
}
// columns c0 .. c0 + 63 of a transposed [64][ld] matrix (ld a multiple of 64, zero padded)
__device__ __forceinline__ void tile_fetch_t(TileRegs& t, const u16* __restrict__ g, int c0, int ld) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = (threadIdx.x >> 3) + 32 * i, c = (threadIdx.x & 7) * 8;
    t.v[i] = *(const uint4*)(g + (int64_t)r * ld + c0 + c);
  }
}
__device__ __forceinline__ void tile_put_t(u16* T, const TileRegs& t) { tile_put(T, t); }

}  // namespace bsp
