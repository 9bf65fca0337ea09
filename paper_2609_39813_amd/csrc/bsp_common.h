// Device helpers shared by the gfx950 kernels: Philox4x32-10, the FP8 codec, bf16
// splitting, wave reductions and the workspace carver. Everything here is written for
// CDNA4 (64-wide wavefronts); nothing is shared with the CPU oracle.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "../../include/bsp.h"

#define BS_WAVE 64

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16;

namespace bsp {

// ---------------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two 32x32->64
// multiplies and xors, key bumped by the Weyl constants between rounds. The counter is
// (element >> 2 lo, element >> 2 hi, trial, use); the key is the 64-bit seed.
// ---------------------------------------------------------------------------------
struct Philox4 {
  uint32_t w0, w1, w2, w3;
};

__device__ __forceinline__ Philox4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                                 uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
    // three-input xor in one v_bitop3_b32 (truth table 0x96 = a ^ b ^ c)
    const uint32_t n0 = __builtin_amdgcn_bitop3_b32((uint32_t)(p1 >> 32), c1, k0, 0x96);
    const uint32_t n2 = __builtin_amdgcn_bitop3_b32((uint32_t)(p0 >> 32), c3, k1, 0x96);
    c1 = (uint32_t)p1;
    c3 = (uint32_t)p0;
    c0 = n0;
    c2 = n2;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return {c0, c1, c2, c3};
}

// Words for the 4 consecutive elements of group g = element >> 2.
__device__ __forceinline__ Philox4 philox_group(uint64_t seed, uint64_t g, uint32_t trial, uint32_t use) {
  return philox4x32_10((uint32_t)g, (uint32_t)(g >> 32), trial, use, (uint32_t)seed, (uint32_t)(seed >> 32));
}

__device__ __forceinline__ uint32_t philox_word(const Philox4& p, int q) {
  return q == 0 ? p.w0 : (q == 1 ? p.w1 : (q == 2 ? p.w2 : p.w3));
}

// ---------------------------------------------------------------------------------
// FP8 codec. For a magnitude a <= FMAX the bracketing grid values are lo = mi * step
// and hi = lo + step, with v = a / step exact (step is a power of two), mi = floor(v)
// and frac = v - mi exact. The code of magnitude m*step is base + m, where base is
// (e + bias - 1) << mbits in the normal range (e = exponent of a) and 0 below it; a
// carry of m into the next binade lands on the right code by construction.
// Everything is taken from the fp32 bit pattern with integer operations: with a = M 2^(e-23)
// (M the 24-bit significand) and q = max(e, 1 - bias) the binade of the grid step
// 2^(q - mbits), v = M / 2^w with w = 23 - mbits + q - e, so mi = M >> w and the fraction is
// the low w bits of M; F = floor(frac 2^32) is those bits moved to the top of a 32-bit word
// (exact for w <= 32, truncated beyond).
// ---------------------------------------------------------------------------------
struct F8 {
  int mbits;
  int bias;
  float fmax;
};

__host__ __device__ __forceinline__ F8 f8_format(int fmt) {
  return fmt == BS_E5M2 ? F8{2, 15, 57344.0f} : F8{3, 7, 448.0f};
}

struct Bracket {
  uint32_t base;  // code of 0 * step in a's binade
  uint32_t mi;    // floor(a / step)
  uint32_t F;     // floor((a / step - mi) * 2^32)
  int sh;         // a / step = a * 2^sh
};

// 0 <= a <= fmax, finite
__device__ __forceinline__ Bracket f8_bracket(float a, F8 f) {
  const uint32_t bits = __float_as_uint(a);
  const int E = (int)(bits >> 23);
  const uint32_t M = (bits & 0x7FFFFFu) | (E ? 0x800000u : 0u);
  const int e = E ? E - 127 : -126;
  const int q = max(e, 1 - f.bias);
  const int w = 23 - f.mbits + q - e;  // >= 20
  Bracket b;
  b.sh = f.mbits - q;
  b.base = (uint32_t)(q + f.bias - 1) << f.mbits;
  b.mi = w < 32 ? M >> w : 0u;
  const uint32_t D = w < 32 ? M & ((1u << w) - 1u) : M;
  b.F = w <= 32 ? (w == 32 ? D : D << (32 - w)) : (w < 64 ? D >> (w - 32) : 0u);
  return b;
}

// y = fl32(x / s) as the fp64 product x * fl64(1 / s) rounded once to fp32 (rs = 1.0 / (double)s,
// computed once). Identical to the IEEE fp32 quotient: the product is within 2^-52 relative of
// x / s, while the quotient of two floats is never a rounding midpoint and, when inexact, is at
// least 2^-49 relative away from every midpoint (x - s m is a nonzero multiple of the smaller
// operand grid; m needs 25 significant bits). Subnormal and overflowing quotients round the same
// way from the fp64 value.
__device__ __forceinline__ float div_scale(float x, double rs) { return (float)((double)x * rs); }

// Round up iff R + F >= 2^32 (so P(up) = F / 2^32): the carry out of the 32-bit add.
__device__ __forceinline__ uint32_t sr_up(uint32_t F, uint32_t R) {
  return (uint32_t)(((uint64_t)R + (uint64_t)F) >> 32);
}

__device__ __forceinline__ uint32_t rne_up(const Bracket& b) {
  return (b.F > 0x80000000u) | ((b.F == 0x80000000u) & (b.mi & 1u));
}

// Step (hi - lo) of a bracket, as a float power of two.
__device__ __forceinline__ float f8_step(const Bracket& b) { return __uint_as_float((uint32_t)(127 - b.sh) << 23); }

// Real value of a finite FP8 code.
__device__ __forceinline__ float f8_value(uint32_t code, F8 f) {
  const uint32_t mag = code & 0x7Fu;
  const int ef = (int)(mag >> f.mbits);
  const int mf = (int)(mag & ((1u << f.mbits) - 1u));
  const float v = ef ? ldexpf((float)((1 << f.mbits) + mf), ef - f.bias - f.mbits)
                     : ldexpf((float)mf, 1 - f.bias - f.mbits);
  return (code & 0x80u) ? -v : v;
}

// ---------------------------------------------------------------------------------
// bf16: exact conversions of values with at most 8 significant bits, and the split of
// an fp32 value into up to three bf16 terms whose sum is the value (each term rounds the
// remainder to nearest; three terms carry all 24 bits).
// ---------------------------------------------------------------------------------
// fp16 bits of x, round to nearest even
__device__ __forceinline__ u16 f16_bits(float x) { return __builtin_bit_cast(u16, (_Float16)x); }

// The two-term fp16 split of fp32 operands: a tensor bounded by `bound` in magnitude is scaled by
// 2^e with bound 2^e in [2^14, 2^15) (no fp16 overflow), then x 2^e = hi + lo + err with hi =
// fp16(x 2^e), lo = fp16(x 2^e - hi), |err| <= 2^-22 |x 2^e| where lo is a normal fp16 number
// and <= 2^-25 (2^-40 of the bound) below; a contraction undoes the scale with 2^-e. e = 0 for
// a bound of zero or not finite (finite values beyond the fp16 range then become infinite);
// -113 <= e <= 100, so 2^e and 2^-e are normal fp32 numbers.
__device__ __forceinline__ int f16_scale_exp(float bound) {
  if (!(bound > 0.0f) || !__builtin_isfinite(bound)) return 0;
  int k;
  (void)frexpf(bound, &k);  // bound in [2^(k-1), 2^k), k <= 128
  const int e = 15 - k;
  return e > 100 ? 100 : e;
}
__device__ __forceinline__ void split2_f16(float xs, u16& hi, u16& lo) {
  const _Float16 h = (_Float16)xs;
  hi = __builtin_bit_cast(u16, h);
  lo = f16_bits(xs - (float)h);
}

__device__ __forceinline__ u16 bf16_bits(float x) {
  __bf16 h = (__bf16)x;
  return __builtin_bit_cast(u16, h);
}
__device__ __forceinline__ float bf16_to_f32(u16 b) { return __uint_as_float((uint32_t)b << 16); }

__device__ __forceinline__ void split3(float x, u16& h0, u16& h1, u16& h2) {
  h0 = bf16_bits(x);
  const float r1 = x - bf16_to_f32(h0);
  h1 = bf16_bits(r1);
  const float r2 = r1 - bf16_to_f32(h1);
  h2 = bf16_bits(r2);
}

template <typename T>
__device__ __forceinline__ float load_f32(const T* p, int64_t i);
template <>
__device__ __forceinline__ float load_f32<float>(const float* p, int64_t i) {
  return p[i];
}
template <>
__device__ __forceinline__ float load_f32<u16>(const u16* p, int64_t i) {
  return bf16_to_f32(p[i]);
}

// ---------------------------------------------------------------------------------
// Wave and block reductions (wave64).
// ---------------------------------------------------------------------------------
__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_down(v, off, BS_WAVE);
  return v;  // valid in lane 0
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint32_t o = __shfl_down(v, off, BS_WAVE);
    v = v > o ? v : o;
  }
  return v;
}
// A maximum raised by many blocks lives in AMAX_SLOTS words AMAX_STRIDE words apart (block b,
// the linear index of a 1-D or 2-D grid, raises slot b % AMAX_SLOTS): device-scope atomics on
// one word serialize, on words in different memory channels they do not. Its value is the max
// over the slots.
constexpr int AMAX_SLOTS = 32, AMAX_STRIDE = 64;
// The block's max of v (float bits of non-negative values; all threads of the block call it)
// raised into its slot of `slots` by one atomic.
__device__ __forceinline__ void block_amax_to_slot(float v, uint32_t* slots) {
  __shared__ uint32_t red[16];
  const uint32_t m = wave_max_u32(__float_as_uint(v));
  if ((threadIdx.x & (BS_WAVE - 1)) == 0) red[threadIdx.x / BS_WAVE] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t b = 0;
    for (int w = 0; w < (int)((blockDim.x + BS_WAVE - 1) / BS_WAVE); ++w) b = b > red[w] ? b : red[w];
    if (b) atomicMax(slots + ((blockIdx.x + gridDim.x * blockIdx.y) % AMAX_SLOTS) * AMAX_STRIDE, b);
  }
}
// The same, one atomic per wave and no LDS (every lane of the wave calls it): for kernels whose
// direct-to-LDS loads the compiler tracks only while they own every LDS variable.
__device__ __forceinline__ void wave_amax_to_slot(float v, uint32_t* slots) {
  const uint32_t m = wave_max_u32(__float_as_uint(v));
  if ((threadIdx.x & (BS_WAVE - 1)) == 0 && m)
    atomicMax(slots + ((blockIdx.x + gridDim.x * blockIdx.y) % AMAX_SLOTS) * AMAX_STRIDE, m);
}
__device__ __forceinline__ float amax_of_slots(const uint32_t* slots) {
  uint32_t m = 0;
#pragma unroll 8
  for (int i = 0; i < AMAX_SLOTS; ++i) m = max(m, slots[i * AMAX_STRIDE]);
  return __uint_as_float(m);
}
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_down(v, off, BS_WAVE);
  return v;
}

}  // namespace bsp

// ---------------------------------------------------------------------------------
// Host side: workspace carving and launch checking.
// ---------------------------------------------------------------------------------
namespace bsp {

struct Carver {
  char* base;
  size_t off = 0;
  size_t cap;
  explicit Carver(void* p = nullptr, size_t c = 0) : base((char*)p), cap(c) {}
  template <typename T>
  T* take(size_t count) {
    off = (off + 255) & ~(size_t)255;
    T* p = base ? (T*)(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
  size_t used() const { return (off + 255) & ~(size_t)255; }
};

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

}  // namespace bsp

#define BS_CHECK_LAUNCH()                                   \
  do {                                                      \
    if (hipGetLastError() != hipSuccess) return BS_EHIP;    \
  } while (0)
