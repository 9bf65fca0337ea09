// Normalization store (RMSNorm -> FP8 store -> Linear) kernels: forward in the fixed
// fp32 order, operand planes for the contractions, the gain use's column reductions,
// the gain use's per-trial standard error, and the normalization input gradient.
#include "bsp_kernels.h"
#include "k_norm.h"

namespace bsp {

// One wave64 per row. Lane l accumulates x_j^2 for j = l, l + 64, ... in ascending j,
// the 64 partials are combined pairwise with offsets 32, 16, ..., 1, then
// ms = ss / d, r = 1 / sqrt(ms + eps), z = x r, u = gain z; every operation rounded to
// fp32 with no contraction. max |u| goes to amax_bits (see amax_kernel).
template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_fwd_kernel(const T* __restrict__ X, const float* __restrict__ gain,
                                                          int64_t Tn, int64_t d, float eps, float* __restrict__ u,
                                                          float* __restrict__ rstd, uint32_t* __restrict__ amax_bits) {
#pragma clang fp contract(off)
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t t = (int64_t)blockIdx.x * 4 + w;
  uint32_t m = 0;
  if (t < Tn) {
    const T* xr = X + t * d;
    float p = 0.0f;
    for (int64_t j = lane; j < d; j += 64) {
      const float x = load_f32(xr, j);
      const float sq = x * x;
      p = p + sq;
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const float o = __shfl_down(p, off, 64);
      if (lane < off) p = p + o;
    }
    const float ss = __shfl(p, 0, 64);
    const float ms = __fdiv_rn(ss, (float)d);
    const float r = 1.0f / sqrtf(ms + eps);  // both correctly rounded (built with -fhip-fp32-correctly-rounded-divide-sqrt)
    float* ur = u + t * d;
    for (int64_t j = lane; j < d; j += 64) {
      const float z = load_f32(xr, j) * r;
      const float uv = gain[j] * z;
      ur[j] = uv;
      const uint32_t b = __float_as_uint(fabsf(uv));
      m = m > b ? m : b;
    }
    if (lane == 0) rstd[t] = r;
  }
  m = wave_max_u32(m);
  __shared__ uint32_t red[4];
  if (lane == 0) red[w] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t b = red[0];
    for (int i = 1; i < 4; ++i) b = b > red[i] ? b : red[i];
    if (b) atomicMax(amax_bits, b);
  }
}

// The same forward with vector accesses (d a multiple of 8; X, gain and u 16-byte aligned) and
// the same fixed fp32 order: each 512-element chunk of a row is loaded 8 elements per lane, its
// squares pass through LDS, and lane l adds the entries l, l + 64, ... of the chunk, chunks in
// order, so partial l still takes j = l, l + 64, ... ascending. A wave takes RMS_RPW rows (the
// same trip count in every wave, so the block barriers are uniform); one amax atomic per block.
constexpr int RMS_RPW = 4;

template <typename T>
__device__ __forceinline__ void load8_f32(const T* p, float (&x)[8]);
template <>
__device__ __forceinline__ void load8_f32<float>(const float* p, float (&x)[8]) {
  const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}
template <>
__device__ __forceinline__ void load8_f32<u16>(const u16* p, float (&x)[8]) {
  const uint4 v = *(const uint4*)p;
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_fwd8_kernel(const T* __restrict__ X, const float* __restrict__ gain,
                                                           int64_t Tn, int64_t d, float eps, float* __restrict__ u,
                                                           float* __restrict__ rstd, uint32_t* __restrict__ amax_bits) {
#pragma clang fp contract(off)
  __shared__ float sq[4][512];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint32_t m = 0;
  for (int k = 0; k < RMS_RPW; ++k) {
    const int64_t t = ((int64_t)blockIdx.x * RMS_RPW + k) * 4 + w;
    const bool ok = t < Tn;
    const T* xr = X + (ok ? t : 0) * d;
    float p = 0.0f;
    for (int64_t c0 = 0; c0 < d; c0 += 512) {
      const int64_t j8 = c0 + 8 * lane;
      if (ok && j8 < d) {
        float x[8];
        load8_f32(xr + j8, x);
#pragma unroll
        for (int i = 0; i < 8; ++i) sq[w][8 * lane + i] = x[i] * x[i];
      }
      __syncthreads();
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (ok && c0 + lane + 64 * i < d) p = p + sq[w][lane + 64 * i];
      __syncthreads();
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const float o = __shfl_down(p, off, 64);
      if (lane < off) p = p + o;
    }
    const float ss = __shfl(p, 0, 64);
    if (!ok) continue;
    const float ms = __fdiv_rn(ss, (float)d);
    const float r = 1.0f / sqrtf(ms + eps);
    float* ur = u + t * d;
    for (int64_t j8 = 8 * lane; j8 < d; j8 += 512) {
      float x[8], g[8], o[8];
      load8_f32(xr + j8, x);
      load8_f32(gain + j8, g);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float z = x[i] * r;
        o[i] = g[i] * z;
        const uint32_t b = __float_as_uint(fabsf(o[i]));
        m = m > b ? m : b;
      }
      *(float4*)(ur + j8) = make_float4(o[0], o[1], o[2], o[3]);
      *(float4*)(ur + j8 + 4) = make_float4(o[4], o[5], o[6], o[7]);
    }
    if (lane == 0) rstd[t] = r;
  }
  m = wave_max_u32(m);
  __shared__ uint32_t red[4];
  if (lane == 0) red[w] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t b = red[0];
    for (int i = 1; i < 4; ++i) b = b > red[i] ? b : red[i];
    if (b) atomicMax(amax_bits, b);
  }
}

// Transposed planes [d][ldo] of per-element operands of the weight-use contractions.
//   NP_VAL : val(C_u)                                      (1 term, exact)
//   NP_RESU: u - s * val(C_u)  (= minus the forward's rounding error; 3 terms)
//   NP_RESN: sign * (n_up - K * [C_u rounded up]) * step   (1 term if K <= 256, else 2)
// split2_f16 of x as one word (hi | lo << 16); kept out of line: inlined into the vector plane
// kernel's packing it trips the compiler's instruction selection
__device__ __attribute__((noinline)) uint32_t split2_f16_word(float x) {
  u16 h, l;
  split2_f16(x, h, l);
  return (uint32_t)h | ((uint32_t)l << 16);
}

// 2^e of the fp16 split of the U residual u - s val(C) (its bound max(max|u|, s FMAX) doubled),
// with 2^-e stored by the first thread of the grid
__device__ __forceinline__ float resu_f16_scale(const NormPlaneArgs& a, float s) {
  const float bound = fmaxf(a.amax_u ? *a.amax_u : 0.0f, s * a.f.fmax);
  const int e = f16_scale_exp(bound) - 1;
  if (a.inv_out && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) *a.inv_out = ldexpf(1.0f, -e);
  return ldexpf(1.0f, e);
}

template <int MODE>
__global__ __launch_bounds__(256) void norm_planes_t_kernel(NormPlaneArgs a) {
  __shared__ u16 tile[3][64][66];
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
  const float s = *a.scale;
  const double rs = 1.0 / (double)s;
  const float rsc = MODE == NP_RESU && a.f16 ? resu_f16_scale(a, s) : 1.0f;
#pragma unroll 2
  for (int i = 0; i < 16; ++i) {
    const int rr = ty + 4 * i;
    const int64_t t = r0 + rr, j = c0 + tx;
    u16 o[3] = {0, 0, 0};
    if (t < a.T && j < a.d) {
      const int64_t e = t * a.d + j;
      const uint32_t code = a.codes[e];
      if (MODE == NP_VAL) {
        {
          const float v = f8_value(code, a.f);
          o[0] = a.f16 ? f16_bits(v) : bf16_bits(v);
        }
      } else if (MODE == NP_RESU) {
        const float r = fmaf(-s, f8_value(code, a.f), a.u[e]);
        if (a.f16)
          split2_f16(r * rsc, o[0], o[1]);
        else
          split3(r, o[0], o[1], o[2]);
      } else {
        const float y = div_scale(a.u[e], rs);
        const Bracket b = f8_bracket(fminf(fabsf(y), a.f.fmax), a.f);
        const int h = (code & 0x7Fu) != b.base + b.mi;
        const float v = (float)((int)a.counts[e] - a.K * h) * f8_step(b);
        if (a.f16)
          o[0] = f16_bits((signbit(y) ? -v : v) * a.resn_scale);
        else
          split3(signbit(y) ? -v : v, o[0], o[1], o[2]);
      }
    }
    for (int p = 0; p < a.nterms; ++p) tile[p][rr][tx] = o[p];
  }
  __syncthreads();
#pragma unroll 2
  for (int i = 0; i < 16; ++i) {
    const int cc = ty + 4 * i;
    const int64_t j = c0 + cc, t = r0 + tx;
    if (j < a.d && t < a.ldo)
      for (int p = 0; p < a.nterms; ++p) a.out[p][j * a.ldo + t] = tile[p][tx][cc];
  }
}

// LDS tile [j][t] of 64 x 64 16-bit values: rows 34 words apart, the words of row r rotated by
// 2 ((r >> 4) & 3), so that 8-byte stores of a thread's four consecutive t of one column and
// 8-byte reads along a row leave every 16-lane pass on distinct banks.
__device__ __forceinline__ int tp_word(int r, int w) { return r * 34 + ((w + 2 * ((r >> 4) & 3)) & 31); }

// The same planes with vector accesses (d a multiple of 4, ldo of 64, 16-byte aligned u, 4-byte
// aligned codes, 8-byte aligned counts): a thread forms 4 consecutive columns of a row, and each
// output row (one column j) leaves the LDS tile as 16-byte stores of 8 consecutive t.
template <int MODE>
__global__ __launch_bounds__(256) void norm_planes_t4_kernel(NormPlaneArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t tile[3][64 * 34];
  const int cg = threadIdx.x & 15, rg = threadIdx.x >> 4;  // 4 columns, 4 consecutive rows
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
  const float s = *a.scale;
  const double rs = 1.0 / (double)s;
  const float rsc = MODE == NP_RESU && a.f16 ? resu_f16_scale(a, s) : 1.0f;
  u16 o[3][4][4];  // [plane][column c][row i]
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t t = r0 + 4 * rg + i, j = c0 + 4 * cg;
#pragma unroll
    for (int p = 0; p < 3; ++p)
#pragma unroll
      for (int c = 0; c < 4; ++c) o[p][c][i] = 0;
    if (t < a.T && j < a.d) {
      const int64_t e = t * a.d + j;
      const uint32_t cw = *(const uint32_t*)(a.codes + e);
      float uv[4] = {0.f, 0.f, 0.f, 0.f};
      if (MODE != NP_VAL) {
        const float4 u4 = *(const float4*)(a.u + e);
        uv[0] = u4.x;
        uv[1] = u4.y;
        uv[2] = u4.z;
        uv[3] = u4.w;
      }
      uint32_t cn[4] = {0, 0, 0, 0};
      if (MODE == NP_RESN) {
        const uint2 c2 = *(const uint2*)(a.counts + e);
        cn[0] = c2.x & 0xFFFFu;
        cn[1] = c2.x >> 16;
        cn[2] = c2.y & 0xFFFFu;
        cn[3] = c2.y >> 16;
      }
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint32_t code = (cw >> (8 * c)) & 0xFFu;
        if (MODE == NP_VAL) {
          const float v = f8_value(code, a.f);
          o[0][c][i] = a.f16 ? f16_bits(v) : bf16_bits(v);
        } else if (MODE == NP_RESU) {
          const float r = fmaf(-s, f8_value(code, a.f), uv[c]);
          if (a.f16) {
            const uint32_t hl = split2_f16_word(r * rsc);
            o[0][c][i] = (u16)(hl & 0xFFFFu);
            o[1][c][i] = (u16)(hl >> 16);
          } else {
            split3(r, o[0][c][i], o[1][c][i], o[2][c][i]);
          }
        } else {
          const float y = div_scale(uv[c], rs);
          const Bracket b = f8_bracket(fminf(fabsf(y), a.f.fmax), a.f);
          const int h = (code & 0x7Fu) != b.base + b.mi;
          const float v = (float)((int)cn[c] - a.K * h) * f8_step(b);
          if (a.f16)
            o[0][c][i] = f16_bits((signbit(y) ? -v : v) * a.resn_scale);
          else
            split3(signbit(y) ? -v : v, o[0][c][i], o[1][c][i], o[2][c][i]);
        }
      }
    }
  }
#pragma unroll
  for (int p = 0; p < 3; ++p)
    if (p < a.nterms)
#pragma unroll
      for (int c = 0; c < 4; ++c)
        *(uint2*)&tile[p][tp_word(4 * cg + c, 2 * rg)] =
            make_uint2((uint32_t)o[p][c][0] | ((uint32_t)o[p][c][1] << 16), (uint32_t)o[p][c][2] | ((uint32_t)o[p][c][3] << 16));
  __syncthreads();
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    const int ch = threadIdx.x + 256 * pass, cc = ch >> 3, k8 = ch & 7;
    const int64_t j = c0 + cc;
    if (j >= a.d) continue;
    const int w0 = tp_word(cc, 4 * k8), w1 = tp_word(cc, 4 * k8 + 2);
#pragma unroll
    for (int p = 0; p < 3; ++p) {
      if (p >= a.nterms) break;
      const uint2 x0 = *(const uint2*)&tile[p][w0], x1 = *(const uint2*)&tile[p][w1];
      *(uint4*)(a.out[p] + j * a.ldo + r0 + 8 * k8) = make_uint4(x0.x, x0.y, x1.x, x1.y);
    }
  }
}

// Per-trial residual planes of the weight use (the per-trial contraction path): a block covers
// 64 rows t x 64 columns j; a thread holds 4 consecutive rows x 4 consecutive columns (one Philox
// call per row and trial). A trial's values go through an LDS tile [j][t] to rows of the plane
// [j][t] and leave as 16-byte pieces. A thread's four rows of a column enter the tile as one
// 8-byte store. Tile rows are 34 words apart, and the words of row r are rotated by
// 2 ((r >> 4) & 3) (tp_word), so that the 16 lanes of a store pass and of a read pass fall on
// distinct banks.
__global__ __launch_bounds__(256) void trial_planes_kernel(TrialPlaneArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t tile[64 * 34];
  __shared__ __attribute__((aligned(16))) uint32_t tileW[64 * 34];
  const int64_t t0 = (int64_t)blockIdx.y * 64, j0 = (int64_t)blockIdx.x * 64;
  const int cg = threadIdx.x & 15, rg = threadIdx.x >> 4;  // column group, row group
  const int64_t jg = j0 + 4 * cg, tb = t0 + 4 * rg;          // first column, first row
  const double rs = 1.0 / (double)*a.scale;
  uint32_t F[4][4];
  u16 sv[4][4];    // bf16 of sign * step
  float ov[4][4], stp[4][4];  // the forward's value and sign * step (outW)
  uint32_t h[4];   // bit c: the forward's code was rounded up
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t t = tb + q;
    h[q] = 0;
    // the row's four columns in one 16-byte and one 4-byte load (d % 4 == 0)
    const bool ok = t < a.T && jg < a.d;
    const float4 uv = ok ? *(const float4*)(a.u + t * a.d + jg) : make_float4(0.f, 0.f, 0.f, 0.f);
    const uint32_t cw = ok ? *(const uint32_t*)(a.codes + t * a.d + jg) : 0u;
    const float u4[4] = {uv.x, uv.y, uv.z, uv.w};
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      F[q][c] = 0;
      sv[q][c] = 0;
      ov[q][c] = stp[q][c] = 0.0f;
      if (ok) {
        const float y = div_scale(u4[c], rs);
        const Bracket b = f8_bracket(fminf(fabsf(y), a.f.fmax), a.f);
        F[q][c] = b.F;
        const float st = signbit(y) ? -f8_step(b) : f8_step(b);
        sv[q][c] = a.f16 ? f16_bits(st) : bf16_bits(st);
        ov[q][c] = f8_value((cw >> (8 * c)) & 0xFFu, a.f);
        stp[q][c] = st;
        h[q] |= (uint32_t)(((cw >> (8 * c)) & 0x7Fu) != b.base + b.mi) << c;
      }
    }
  }
  for (int b = 0; b < a.nb; ++b) {
    const uint32_t k = (uint32_t)(a.k0 + b);
    u16 dv[4][4], wv[4][4];  // [c][q]: the difference and the new rounding's value
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t t = tb + q;
      const Philox4 p = philox_group(a.seed, (uint64_t)((t * a.d + jg) >> 2), k, a.use);
      const uint32_t R[4] = {p.w0, p.w1, p.w2, p.w3};
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint32_t up = sr_up(F[q][c], R[c]), hb = (h[q] >> c) & 1u;
        dv[c][q] = up == hb ? (u16)0 : (up ? sv[q][c] : (u16)(sv[q][c] ^ 0x8000u));
        // the new rounding's value: exact (an FP8 value)
        const float nv = up == hb ? ov[q][c] : (up ? ov[q][c] + stp[q][c] : ov[q][c] - stp[q][c]);
        wv[c][q] = a.f16 ? f16_bits(nv) : bf16_bits(nv);
      }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int wd = tp_word(4 * cg + c, 2 * rg);  // words 2 rg, 2 rg + 1 of row 4 cg + c
      *(uint2*)&tile[wd] = make_uint2((uint32_t)dv[c][0] | ((uint32_t)dv[c][1] << 16),
                                      (uint32_t)dv[c][2] | ((uint32_t)dv[c][3] << 16));
      if (a.outW)
        *(uint2*)&tileW[wd] = make_uint2((uint32_t)wv[c][0] | ((uint32_t)wv[c][1] << 16),
                                         (uint32_t)wv[c][2] | ((uint32_t)wv[c][3] << 16));
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int ch = threadIdx.x + 256 * i, cc = ch >> 3, k8 = ch & 7;
      const int64_t j = j0 + cc;
      const int64_t o = (int64_t)b * a.d * a.ldo + j * a.ldo + t0 + 8 * k8;
      const int w0 = tp_word(cc, 4 * k8), w1 = tp_word(cc, 4 * k8 + 2);
      if (j < a.d && a.out) {
        const uint2 x0 = *(const uint2*)&tile[w0], x1 = *(const uint2*)&tile[w1];
        *(uint4*)(a.out + o) = make_uint4(x0.x, x0.y, x1.x, x1.y);
      }
      if (j < a.d && a.outW) {
        const uint2 x0 = *(const uint2*)&tileW[w0], x1 = *(const uint2*)&tileW[w1];
        *(uint4*)(a.outW + o) = make_uint4(x0.x, x0.y, x1.x, x1.y);
      }
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void trial_accum_kernel(const float* __restrict__ delta, int nb, int k0, int64_t m,
                                                          float* __restrict__ d1, double* __restrict__ S1,
                                                          double* __restrict__ S2) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m; i += (int64_t)gridDim.x * blockDim.x) {
    float shift = k0 == 1 ? delta[i] : d1[i];
    double a1 = k0 == 1 ? 0.0 : S1[i], a2 = k0 == 1 ? 0.0 : S2[i];
    for (int b = (k0 == 1 ? 1 : 0); b < nb; ++b) {
      const double x = (double)delta[(int64_t)b * m + i] - (double)shift;
      a1 += x;
      a2 += x * x;
    }
    if (k0 == 1) d1[i] = shift;
    S1[i] = a1;
    S2[i] = a2;
  }
}

// The same over four consecutive elements per thread (m % 4 == 0, 16-byte aligned arrays): 16-byte
// loads, and the trial loop unrolled so that several trials' loads are in flight; each element's
// trials are still added in order.
__global__ __launch_bounds__(256) void trial_accum4_kernel(const float4* __restrict__ delta, int nb, int k0, int64_t m4,
                                                           float4* __restrict__ d1, double2* __restrict__ S1,
                                                           double2* __restrict__ S2) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m4; i += (int64_t)gridDim.x * blockDim.x) {
    const float4 sh = k0 == 1 ? delta[i] : d1[i];
    const float shift[4] = {sh.x, sh.y, sh.z, sh.w};
    double a1[4] = {0.0, 0.0, 0.0, 0.0}, a2[4] = {0.0, 0.0, 0.0, 0.0};
    if (k0 != 1) {
      const double2 p0 = S1[2 * i], p1 = S1[2 * i + 1], q0 = S2[2 * i], q1 = S2[2 * i + 1];
      a1[0] = p0.x; a1[1] = p0.y; a1[2] = p1.x; a1[3] = p1.y;
      a2[0] = q0.x; a2[1] = q0.y; a2[2] = q1.x; a2[3] = q1.y;
    }
#pragma unroll 4
    for (int b = (k0 == 1 ? 1 : 0); b < nb; ++b) {
      const float4 v = delta[(int64_t)b * m4 + i];
      const float xv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const double x = (double)xv[c] - (double)shift[c];
        a1[c] += x;
        a2[c] += x * x;
      }
    }
    if (k0 == 1) d1[i] = sh;
    S1[2 * i] = make_double2(a1[0], a1[1]);
    S1[2 * i + 1] = make_double2(a1[2], a1[3]);
    S2[2 * i] = make_double2(a2[0], a2[1]);
    S2[2 * i + 1] = make_double2(a2[2], a2[3]);
  }
}

__global__ __launch_bounds__(256) void trial_se_kernel(const double* __restrict__ S1, const double* __restrict__ S2,
                                                       int K, int64_t m, float* __restrict__ se) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m; i += (int64_t)gridDim.x * blockDim.x) {
    const double a1 = S1[i];
    se[i] = K > 1 ? (float)sqrt(fmax(S2[i] - a1 * a1 / K, 0.0) / (K - 1) / K) : 0.0f;
  }
}

// Row-major plane of val(C) (exact bf16), the A operand of the Linear forward.
__global__ __launch_bounds__(256) void val_rows_kernel(const uint8_t* __restrict__ codes, int64_t n, F8 f,
                                                       u16* __restrict__ out) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    out[i] = bf16_bits(f8_value(codes[i], f));
}

// Gain use, partial column sums over a tile of 64 rows (fp64):
//   q0: z du                      (reference)
//   q1: (s val(C_u) - gain z) / gain * du          (R: reads deq(C_u) / gain)
//   q2: (s mean_k val(C_k) - gain z) / gain * du   (N: reads a new rounding; mean over
//       the K trials = sign (lo + n_up step / K))
// z = fl32(x r) is recomputed exactly as in the forward.
template <typename T>
__global__ __launch_bounds__(256) void gain_partials_kernel(GainArgs<T> a) {
#pragma clang fp contract(off)
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t rt = blockIdx.y;
  if (j >= a.d) return;
  const double s = *a.scale;
  const float sf = *a.scale;
  const double rsf = 1.0 / (double)sf;
  const double g = a.gain[j], ig = 1.0 / g;
  double q0 = 0.0, q1 = 0.0, q2 = 0.0;
  const int64_t tend = (rt + 1) * GAIN_RT < a.T ? (rt + 1) * GAIN_RT : a.T;
  for (int64_t t = rt * GAIN_RT; t < tend; ++t) {
    const int64_t e = t * a.d + j;
    const float z = load_f32(a.X, e) * a.rstd[t];
    const double du = a.du[e];
    const double gz = g * (double)z;
    q0 += (double)z * du;
    if (a.want_r) q1 += (s * (double)f8_value(a.codes[e], a.f) - gz) * ig * du;
    if (a.counts) {
      const float y = div_scale(a.u[e], rsf);
      const Bracket b = f8_bracket(fminf(fabsf(y), a.f.fmax), a.f);
      const double step = f8_step(b);
      double mv = (double)b.mi * step + (double)a.counts[e] * step / a.K;
      if (signbit(y)) mv = -mv;
      q2 += (s * mv - gz) * ig * du;
    }
  }
  const int64_t nrt = gridDim.y;
  a.part[(0 * nrt + rt) * a.d + j] = q0;
  a.part[(1 * nrt + rt) * a.d + j] = q1;
  a.part[(2 * nrt + rt) * a.d + j] = q2;
}

// Sums the row-tile partials of each column: 16 segments of row tiles per column, each summed
// in order, then the segments by a fixed tree (deterministic). 16 columns per block.
__global__ __launch_bounds__(256) void gain_final_kernel(const double* __restrict__ part, int64_t nrt, int64_t d,
                                                         float* __restrict__ ref, float* __restrict__ bias_r,
                                                         float* __restrict__ bias_n) {
  __shared__ double red[3][16][17];
  const int c = threadIdx.x & 15, sgi = threadIdx.x >> 4;
  const int64_t j = (int64_t)blockIdx.x * 16 + c;
  const int64_t per = (nrt + 15) / 16;
  const int64_t r0 = sgi * per, r1 = (r0 + per) < nrt ? (r0 + per) : nrt;
  // only the arrays asked for are read; eight rows' loads in flight ahead of their (ordered) adds
  const int na = bias_n ? 3 : (bias_r ? 2 : 1);
  double q[3] = {0.0, 0.0, 0.0};
  if (j < d) {
    int64_t rt = r0;
    for (; rt + 8 <= r1; rt += 8) {
      double v[3][8];
#pragma unroll
      for (int i = 0; i < 3; ++i)
#pragma unroll
        for (int u = 0; u < 8; ++u) v[i][u] = i < na ? part[(i * nrt + rt + u) * d + j] : 0.0;
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int i = 0; i < 3; ++i) q[i] += v[i][u];
    }
    for (; rt < r1; ++rt)
#pragma unroll
      for (int i = 0; i < 3; ++i)
        if (i < na) q[i] += part[(i * nrt + rt) * d + j];
  }
#pragma unroll
  for (int i = 0; i < 3; ++i) red[i][sgi][c] = q[i];
  __syncthreads();
  for (int h = 8; h >= 1; h >>= 1) {
    if (sgi < h)
#pragma unroll
      for (int i = 0; i < 3; ++i) red[i][sgi][c] += red[i][sgi + h][c];
    __syncthreads();
  }
  if (sgi == 0 && j < d) {
    ref[j] = (float)red[0][0][c];
    if (bias_r) bias_r[j] = (float)red[1][0][c];
    if (bias_n) bias_n[j] = (float)red[2][0][c];
  }
}

// se of the gain use under N: the per-trial gradient is const + (s / gain) S_k with
// S_k = sum over row tiles of the new-rounding counter's partials. First S_k[j] for every
// (trial, column) (row tiles summed in order), then Welford over k in order per column.
__global__ __launch_bounds__(256) void gain_trial_sum_kernel(const float* __restrict__ part, int64_t nrt, int64_t d,
                                                             double* __restrict__ S) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t k = blockIdx.y;
  if (j >= d) return;
  const float* p = part + k * nrt * d + j;
  double acc = 0.0;
  int64_t rt = 0;
  for (; rt + 8 <= nrt; rt += 8) {  // eight loads in flight, added in row-tile order
    float v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = p[(rt + q) * d];
#pragma unroll
    for (int q = 0; q < 8; ++q) acc += v[q];
  }
  for (; rt < nrt; ++rt) acc += p[rt * d];
  S[k * d + j] = acc;
}

// se of the gain use under N: 16 lanes per column, each over trials k = lane, lane + 16, ...
// of the shifted values S_k - S_0 (sum and sum of squares, fp64), folded over the 16 lanes
// in a fixed tree; sample variance over the K trials, se = |s / gain| sqrt(var / K).
__global__ __launch_bounds__(256) void gain_se_kernel(const double* __restrict__ S, int K, int64_t d,
                                                      const float* __restrict__ scale, const float* __restrict__ gain,
                                                      float* __restrict__ se) {
  const int64_t j = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
  const int sub = threadIdx.x & 15;
  const bool ok = j < d;
  const double s0 = ok ? S[j] : 0.0;
  double a1 = 0.0, a2 = 0.0;
  if (ok)
    for (int k = sub; k < K; k += 16) {
      const double v = S[(int64_t)k * d + j] - s0;
      a1 += v;
      a2 += v * v;
    }
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) {
    a1 += __shfl_xor(a1, o, 64);
    a2 += __shfl_xor(a2, o, 64);
  }
  if (!ok || sub != 0) return;
  const double var = K > 1 ? fmax(a2 - a1 * a1 / K, 0.0) / (K - 1) : 0.0;
  const double f = fabs((double)*scale / (double)gain[j]);
  se[j] = (float)(f * sqrt(var / K));
}

// Normalization input gradient, one wave64 per row:
//   dz = gain du; dx = r (dz - zhat (sum_j dz zhat) / d), zhat = z (U) or s val(C_u) / gain (R).
template <typename T>
__global__ __launch_bounds__(256) void norm_dx_kernel(DxArgs<T> a) {
#pragma clang fp contract(off)
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t t = (int64_t)blockIdx.x * 4 + w;
  if (t >= a.T) return;
  const float r = a.rstd[t];
  const double s = a.scale ? (double)*a.scale : 1.0;
  double dot_u = 0.0, dot_r = 0.0;
  for (int64_t j = lane; j < a.d; j += 64) {
    const int64_t e = t * a.d + j;
    const double z = (double)(load_f32(a.X, e) * r);
    const double g = a.gain[j];
    const double dz = g * (double)a.du[e];
    dot_u += dz * z;
    if (a.dx_r) dot_r += dz * (s * (double)f8_value(a.codes[e], a.f) / g);
  }
  dot_u = wave_sum_f64(dot_u);
  dot_r = wave_sum_f64(dot_r);
  dot_u = __shfl(dot_u, 0, 64) / (double)a.d;
  dot_r = __shfl(dot_r, 0, 64) / (double)a.d;
  for (int64_t j = lane; j < a.d; j += 64) {
    const int64_t e = t * a.d + j;
    const double z = (double)(load_f32(a.X, e) * r);
    const double g = a.gain[j];
    const double dz = g * (double)a.du[e];
    a.dx_ref[e] = (float)((double)r * (dz - z * dot_u));
    if (a.dx_r) {
      const double zr = s * (double)f8_value(a.codes[e], a.f) / g;
      a.dx_r[e] = (float)((double)r * (dz - zr * dot_r));
    }
  }
}

// mean = ref + bias, bias, se (each output nullable; bias / se inputs nullable = 0).
__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ ref, const float* __restrict__ bias,
                                                      const float* __restrict__ se, int64_t n, float* __restrict__ mean_out,
                                                      float* __restrict__ bias_out, float* __restrict__ se_out) {
  // 16-byte vectors when every pointer allows them, then the scalar tail
  bool vec = true;
  for (const void* p : {(const void*)ref, (const void*)bias, (const void*)se, (const void*)mean_out,
                        (const void*)bias_out, (const void*)se_out})
    vec = vec && ((uintptr_t)p & 15) == 0;
  const int64_t n4 = vec ? n / 4 : 0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
    const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
    const float4 b = bias ? ((const float4*)bias)[i] : z;
    if (mean_out) {
      const float4 r = ((const float4*)ref)[i];
      ((float4*)mean_out)[i] = bias ? make_float4(r.x + b.x, r.y + b.y, r.z + b.z, r.w + b.w) : r;
    }
    if (bias_out) ((float4*)bias_out)[i] = b;
    if (se_out) ((float4*)se_out)[i] = se ? ((const float4*)se)[i] : z;
  }
  for (int64_t i = 4 * n4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const float b = bias ? bias[i] : 0.0f;
    if (mean_out) mean_out[i] = bias ? ref[i] + b : ref[i];
    if (bias_out) bias_out[i] = b;
    if (se_out) se_out[i] = se ? se[i] : 0.0f;
  }
}

// mean = alt, bias = alt - ref (a use whose reading is computed in full).
__global__ __launch_bounds__(256) void combine_alt_kernel(const float* __restrict__ ref, const float* __restrict__ alt,
                                                          int64_t n, float* __restrict__ mean_out,
                                                          float* __restrict__ bias_out, float* __restrict__ se_out) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    if (mean_out) mean_out[i] = alt[i];
    if (bias_out) bias_out[i] = alt[i] - ref[i];
    if (se_out) se_out[i] = 0.0f;
  }
}

// ------------------------------------------------------------------------------------
// launchers
// ------------------------------------------------------------------------------------
static unsigned grid1d(int64_t n, int64_t cap = 8192) {
  const int64_t want = (n + 255) / 256;
  return (unsigned)(want < 1 ? 1 : (want < cap ? want : cap));
}

bs_status launch_rmsnorm_fwd(const void* X, bs_dtype dt, const float* gain, int64_t T, int64_t d, float eps, float* u,
                             float* rstd, bs_diag* diag, hipStream_t st) {
  if (T > 0) {
    const unsigned blocks = (unsigned)((T + 3) / 4);
    ProfScope prof("rmsnorm_fwd", st);
    const bool vec = d % 8 == 0 && ((uintptr_t)X & 15) == 0 && ((uintptr_t)gain & 15) == 0 && ((uintptr_t)u & 15) == 0;
    const unsigned blocks8 = (unsigned)((T + 4 * RMS_RPW - 1) / (4 * RMS_RPW));
    if (vec && dt == BS_F32)
      rmsnorm_fwd8_kernel<float><<<blocks8, 256, 0, st>>>((const float*)X, gain, T, d, eps, u, rstd,
                                                          (uint32_t*)&diag->amax);
    else if (vec)
      rmsnorm_fwd8_kernel<u16><<<blocks8, 256, 0, st>>>((const u16*)X, gain, T, d, eps, u, rstd,
                                                        (uint32_t*)&diag->amax);
    else if (dt == BS_F32)
      rmsnorm_fwd_kernel<float><<<blocks, 256, 0, st>>>((const float*)X, gain, T, d, eps, u, rstd,
                                                        (uint32_t*)&diag->amax);
    else
      rmsnorm_fwd_kernel<u16><<<blocks, 256, 0, st>>>((const u16*)X, gain, T, d, eps, u, rstd,
                                                      (uint32_t*)&diag->amax);
  }
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status launch_norm_planes(int mode, const NormPlaneArgs& a, hipStream_t st) {
  if (a.f16 && ((mode == NP_RESU) != (a.nterms == 2) || a.nterms > 2 || (mode == NP_RESN && a.K > 256)))
    return BS_EINVAL;
  if (a.d <= 0 || a.ldo <= 0) return BS_OK;
  dim3 grid((unsigned)((a.d + 63) / 64), (unsigned)((a.ldo + 63) / 64));
  bool vec = a.d % 4 == 0 && a.ldo % 64 == 0 && ((uintptr_t)a.u & 15) == 0 && ((uintptr_t)a.codes & 3) == 0 &&
             ((uintptr_t)a.counts & 7) == 0;
  for (int p = 0; p < a.nterms; ++p) vec = vec && ((uintptr_t)a.out[p] & 15) == 0;
  if (vec) {
    if (mode == NP_VAL)
      norm_planes_t4_kernel<NP_VAL><<<grid, 256, 0, st>>>(a);
    else if (mode == NP_RESU)
      norm_planes_t4_kernel<NP_RESU><<<grid, 256, 0, st>>>(a);
    else
      norm_planes_t4_kernel<NP_RESN><<<grid, 256, 0, st>>>(a);
  } else if (mode == NP_VAL)
    norm_planes_t_kernel<NP_VAL><<<grid, 256, 0, st>>>(a);
  else if (mode == NP_RESU)
    norm_planes_t_kernel<NP_RESU><<<grid, 256, 0, st>>>(a);
  else
    norm_planes_t_kernel<NP_RESN><<<grid, 256, 0, st>>>(a);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status launch_trial_planes(const TrialPlaneArgs& a, hipStream_t st) {
  if (a.nb <= 0 || a.d <= 0) return BS_OK;
  // whole 16-byte pieces of padded rows out, four columns per load in
  if (a.ldo % 64 || ((uintptr_t)a.out & 15) || ((uintptr_t)a.outW & 15) || (a.d & 3) || ((uintptr_t)a.u & 15) ||
      ((uintptr_t)a.codes & 3))
    return BS_EINVAL;
  dim3 grid((unsigned)((a.d + 63) / 64), (unsigned)((a.ldo + 63) / 64));
  ProfScope prof("trial_planes", st);
  trial_planes_kernel<<<grid, 256, 0, st>>>(a);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
bs_status launch_trial_accum(const float* delta, int nb, int k0, int64_t m, float* d1, double* S1, double* S2,
                             hipStream_t st) {
  if (m <= 0 || nb <= 0) return BS_OK;
  const bool vec = m % 4 == 0 && ((uintptr_t)delta & 15) == 0 && ((uintptr_t)d1 & 15) == 0 && ((uintptr_t)S1 & 15) == 0 &&
                   ((uintptr_t)S2 & 15) == 0;
  if (vec)
    trial_accum4_kernel<<<grid1d(m / 4), 256, 0, st>>>((const float4*)delta, nb, k0, m / 4, (float4*)d1, (double2*)S1,
                                                       (double2*)S2);
  else
    trial_accum_kernel<<<grid1d(m), 256, 0, st>>>(delta, nb, k0, m, d1, S1, S2);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
bs_status launch_trial_se(const double* S1, const double* S2, int K, int64_t m, float* se, hipStream_t st) {
  if (m <= 0) return BS_OK;
  trial_se_kernel<<<grid1d(m), 256, 0, st>>>(S1, S2, K, m, se);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
bs_status launch_val_rows(const uint8_t* codes, int64_t n, int fmt, u16* out, hipStream_t st) {
  if (n > 0) val_rows_kernel<<<grid1d(n), 256, 0, st>>>(codes, n, f8_format(fmt), out);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

template <typename T>
bs_status launch_gain_t(const GainArgs<T>& a, float* ref, float* bias_r, float* bias_n, hipStream_t st) {
  if (a.d <= 0) return BS_OK;
  const int64_t nrt = (a.T + GAIN_RT - 1) / GAIN_RT;
  if (nrt == 0) {
    if (ref) launch_fill2d(ref, 1, a.d, a.d, 0.0f, st);
    if (bias_r) launch_fill2d(bias_r, 1, a.d, a.d, 0.0f, st);
    if (bias_n) launch_fill2d(bias_n, 1, a.d, a.d, 0.0f, st);
    BS_CHECK_LAUNCH();
    return BS_OK;
  }
  dim3 grid((unsigned)((a.d + 255) / 256), (unsigned)nrt);
  gain_partials_kernel<T><<<grid, 256, 0, st>>>(a);
  gain_final_kernel<<<(unsigned)((a.d + 15) / 16), 256, 0, st>>>(a.part, nrt, a.d, ref, bias_r, bias_n);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
template bs_status launch_gain_t<float>(const GainArgs<float>&, float*, float*, float*, hipStream_t);
template bs_status launch_gain_t<u16>(const GainArgs<u16>&, float*, float*, float*, hipStream_t);

bs_status launch_gain_se(const float* part, int K, int64_t T, int64_t d, const float* scale, const float* gain,
                         double* S, float* se, hipStream_t st) {
  if (d <= 0) return BS_OK;
  const int64_t nrt = (T + 31) / 32;
  gain_trial_sum_kernel<<<dim3((unsigned)((d + 255) / 256), (unsigned)K), 256, 0, st>>>(part, nrt, d, S);
  gain_se_kernel<<<(unsigned)((d + 15) / 16), 256, 0, st>>>(S, K, d, scale, gain, se);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

template <typename T>
bs_status launch_dx_t(const DxArgs<T>& a, hipStream_t st) {
  if (a.T > 0) norm_dx_kernel<T><<<(unsigned)((a.T + 3) / 4), 256, 0, st>>>(a);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
template bs_status launch_dx_t<float>(const DxArgs<float>&, hipStream_t);
template bs_status launch_dx_t<u16>(const DxArgs<u16>&, hipStream_t);

// Every policy's estimate of one gradient in one pass over ref: policy p writes mean_p = ref +
// bias_p (or alt_p, with bias_p = alt_p - ref, when alt_p is set), bias_p and se_p (bias_p / se_p
// inputs nullable = 0) at offset p n of the nullable output bases.
// a 16-byte non-temporal store (p 16-byte aligned)
__device__ __forceinline__ void store4_nt(float* p, float4 v) {
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  const f32x4 w = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(w, (f32x4*)p);
}

__global__ __launch_bounds__(256) void combine_multi_kernel(CombineMulti c, int64_t n) {
  const int64_t n4 = c.vec ? n / 4 : 0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
    const float4 r = ((const float4*)c.ref)[i];
    for (int p = 0; p < c.n_pol; ++p) {
      const int64_t o = (int64_t)p * n4 + i;
      float4 m, b;
      if (c.alt[p]) {
        m = ((const float4*)c.alt[p])[i];
        b = make_float4(m.x - r.x, m.y - r.y, m.z - r.z, m.w - r.w);
      } else {
        b = c.bias[p] ? ((const float4*)c.bias[p])[i] : z;
        m = c.bias[p] ? make_float4(r.x + b.x, r.y + b.y, r.z + b.z, r.w + b.w) : r;
      }
      // streaming outputs: non-temporal stores keep them from displacing the inputs in the caches
      if (c.mean) store4_nt(c.mean + 4 * o, m);
      if (c.bias_out) store4_nt(c.bias_out + 4 * o, b);
      if (c.se_out) store4_nt(c.se_out + 4 * o, c.se[p] ? ((const float4*)c.se[p])[i] : z);
    }
  }
  for (int64_t i = 4 * n4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const float r = c.ref[i];
    for (int p = 0; p < c.n_pol; ++p) {
      const int64_t o = (int64_t)p * n + i;
      const float m = c.alt[p] ? c.alt[p][i] : (c.bias[p] ? r + c.bias[p][i] : r);
      const float b = c.alt[p] ? m - r : (c.bias[p] ? c.bias[p][i] : 0.0f);
      if (c.mean) c.mean[o] = m;
      if (c.bias_out) c.bias_out[o] = b;
      if (c.se_out) c.se_out[o] = c.se[p] ? c.se[p][i] : 0.0f;
    }
  }
}

bs_status launch_gain_final(const double* part, int64_t nrt, int64_t d, float* ref, float* bias_r, float* bias_n,
                            hipStream_t st) {
  if (d <= 0 || nrt <= 0) return BS_OK;
  gain_final_kernel<<<(unsigned)((d + 15) / 16), 256, 0, st>>>(part, nrt, d, ref, bias_r, bias_n);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status launch_combine_multi(CombineMulti c, int64_t n, hipStream_t st) {
  if (n <= 0 || c.n_pol < 1 || (!c.mean && !c.bias_out && !c.se_out)) return BS_OK;
  if (c.n_pol > COMBINE_MAX_POL) return BS_EINVAL;
  // the float4 path needs every array 16-byte aligned, including each policy's output slice
  bool vec = n % 4 == 0;
  for (const void* q : {(const void*)c.ref, (const void*)c.mean, (const void*)c.bias_out, (const void*)c.se_out})
    vec = vec && ((uintptr_t)q & 15) == 0;
  for (int p = 0; p < c.n_pol; ++p)
    for (const void* q : {(const void*)c.bias[p], (const void*)c.se[p], (const void*)c.alt[p]})
      vec = vec && ((uintptr_t)q & 15) == 0;
  c.vec = vec ? 1 : 0;
  combine_multi_kernel<<<grid1d((n + 3) / 4, 4096), 256, 0, st>>>(c, n);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status launch_combine(const float* ref, const float* bias, const float* se, int64_t n, float* mean_out,
                         float* bias_out, float* se_out, hipStream_t st) {
  if (n <= 0 || (!mean_out && !bias_out && !se_out)) return BS_OK;
  combine_kernel<<<grid1d((n + 3) / 4, 4096), 256, 0, st>>>(ref, bias, se, n, mean_out, bias_out, se_out);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status launch_combine_alt(const float* ref, const float* alt, int64_t n, float* mean_out, float* bias_out,
                             float* se_out, hipStream_t st) {
  if (n <= 0 || (!mean_out && !bias_out && !se_out)) return BS_OK;
  combine_alt_kernel<<<grid1d(n), 256, 0, st>>>(ref, alt, n, mean_out, bias_out, se_out);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

}  // namespace bsp
