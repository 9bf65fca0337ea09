// Utility kernels: fills, bf16 operand planes (copy / split / transpose), and the trial
// statistics reducer.
#include "bsp_kernels.h"

namespace bsp {

__global__ void init_diag_only(bs_diag* diag) {
  if (threadIdx.x == 0) {
    diag->nonfinite = 0;
    diag->n_saturated = 0;
    diag->amax = 0.0f;
    diag->scale = 1.0f;
  }
}

bs_status launch_init_diag(bs_diag* diag, hipStream_t st) {
  init_diag_only<<<1, 64, 0, st>>>(diag);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

__global__ void fill2d_kernel(float* p, int64_t rows, int64_t cols, int64_t ld, float v) {
  const int64_t n = rows * cols;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[(i / cols) * ld + (i % cols)] = v;
}
__global__ void fill_f64_kernel(double* p, int64_t n, double v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) p[i] = v;
}

bs_status launch_fill2d(float* p, int64_t rows, int64_t cols, int64_t ld, float v, hipStream_t st) {
  const int64_t n = rows * cols;
  if (n <= 0) return BS_OK;
  const int64_t want = (n + 255) / 256;
  fill2d_kernel<<<(unsigned)(want < 4096 ? want : 4096), 256, 0, st>>>(p, rows, cols, ld, v);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
bs_status launch_fill_f64(double* p, int64_t n, double v, hipStream_t st) {
  if (n <= 0) return BS_OK;
  const int64_t want = (n + 255) / 256;
  fill_f64_kernel<<<(unsigned)(want < 4096 ? want : 4096), 256, 0, st>>>(p, n, v);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

// ------------------------------------------------------------------------------------
// bf16 planes of a [R, C] matrix: value * scale split into nterms bf16 terms.
// ------------------------------------------------------------------------------------
struct PlaneOut {
  u16* p[3];
};

__device__ __forceinline__ void split_to(float v, int nterms, u16 (&o)[3]) {
  if (nterms == 1) {
    o[0] = bf16_bits(v);
    o[1] = o[2] = 0;
  } else {
    split3(v, o[0], o[1], o[2]);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void planes_rows_kernel(const T* __restrict__ in, int64_t R, int64_t C, int64_t ldi,
                                                          PlaneOut out, int nterms, int64_t ldo, float scale) {
  const int64_t n = R * ldo;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / ldo, c = i - r * ldo;
    const float v = c < C ? load_f32(in, r * ldi + c) * scale : 0.0f;
    u16 o[3];
    split_to(v, nterms, o);
    for (int p = 0; p < nterms; ++p) out.p[p][i] = o[p];
  }
}

// The same planes of an fp32 matrix 4 elements per thread (C, ldi and ldo multiples of 4, 16-byte
// aligned input rows, 8-byte aligned planes): one index division per 4 elements, 16-byte loads,
// 8-byte stores per plane.
__global__ __launch_bounds__(256) void planes_rows4_kernel(const float* __restrict__ in, int64_t R, int64_t C,
                                                           int64_t ldi, PlaneOut out, int nterms, int64_t ldo,
                                                           float scale) {
  const int64_t q = ldo / 4, n = R * q;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / q, c = 4 * (i - r * q);
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (c < C) v = *(const float4*)(in + r * ldi + c);
    const float x[4] = {v.x * scale, v.y * scale, v.z * scale, v.w * scale};
    u16 o[4][3];
#pragma unroll
    for (int k = 0; k < 4; ++k) split_to(x[k], nterms, o[k]);
#pragma unroll
    for (int p = 0; p < 3; ++p)
      if (p < nterms)
        *(uint2*)(out.p[p] + 4 * i) = make_uint2((uint32_t)o[0][p] | ((uint32_t)o[1][p] << 16),
                                                 (uint32_t)o[2][p] | ((uint32_t)o[3][p] << 16));
  }
}

// Transposed: out_p[c * ldo + r] for r < ldo (zero for r >= R). Tile 64 x 64 through LDS.
template <typename T>
__global__ __launch_bounds__(256) void planes_t_kernel(const T* __restrict__ in, int64_t R, int64_t C, int64_t ldi,
                                                       PlaneOut out, int nterms, int64_t ldo, float scale) {
  __shared__ u16 tile[3][64][66];
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int rr = ty + 4 * i;
    const int64_t r = r0 + rr, c = c0 + tx;
    const float v = (r < R && c < C) ? load_f32(in, r * ldi + c) * scale : 0.0f;
    u16 o[3];
    split_to(v, nterms, o);
    for (int p = 0; p < nterms; ++p) tile[p][rr][tx] = o[p];
  }
  __syncthreads();
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int cc = ty + 4 * i;
    const int64_t c = c0 + cc, r = r0 + tx;
    if (c < C && r < ldo)
      for (int p = 0; p < nterms; ++p) out.p[p][c * ldo + r] = tile[p][tx][cc];
  }
}

// The transpose of a bf16 [R, C] matrix (C and ldi multiples of 8, 16-byte aligned rows) into
// [C][ldo] with zeros in rows R .. ldo - 1 of every output row: one 64 x 64 tile per block,
// 16-byte loads and stores, the tile held in LDS with rows padded to 144 bytes.
__global__ __launch_bounds__(256) void transpose_bf16_kernel(const u16* __restrict__ in, int64_t R, int64_t C,
                                                             int64_t ldi, u16* __restrict__ out, int64_t ldo) {
  __shared__ __attribute__((aligned(16))) u16 tile[64][72];
  const int t = threadIdx.x, q = (t & 7) * 8;
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    const int rr = (t >> 3) + 32 * pass;
    const int64_t r = r0 + rr, c = c0 + q;
    const uint4 v = (r < R && c < C) ? *(const uint4*)(in + r * ldi + c) : make_uint4(0, 0, 0, 0);
    *(uint4*)&tile[rr][q] = v;
  }
  __syncthreads();
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    const int cc = (t >> 3) + 32 * pass;
    const int64_t c = c0 + cc;
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = (uint32_t)tile[q + 2 * i][cc] | ((uint32_t)tile[q + 2 * i + 1][cc] << 16);
    if (c < C) *(uint4*)(out + c * ldo + r0 + q) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// The transposed planes of an fp32 [R, C] matrix (C and ldi multiples of 4, 16-byte aligned rows,
// ldo a multiple of 64) split into nterms bf16 terms per value (the split of planes_t_kernel): a
// 64 x 64 tile goes into LDS as fp32 (rows padded to 65 words, so both the row writes and the
// column reads below fall on distinct banks); a thread then splits 8 consecutive rows of one
// column and stores them as one 16-byte piece per plane, eight threads covering 128 bytes of an
// output row. Optional: add (nullable, same layout as in) is added before the split, and the
// row-major planes (rows.p[0] non-null, leading dimension ldr; three bf16 terms) are written from
// the same read. F16T: the transposed planes are the two-term fp16 split at the scale 2^e that
// scale sc gives (F16Scale), and 2^-e is stored to *sc.inv_out by the first thread (nullable).
template <bool F16T>
__global__ __launch_bounds__(256) void transpose_split_f32_kernel(const float* __restrict__ in, const float* __restrict__ add,
                                                                  int64_t R, int64_t C, int64_t ldi, PlaneOut out,
                                                                  int nterms, int64_t ldo, float scale, PlaneOut rows,
                                                                  int64_t ldr, F16Scale sc) {
  __shared__ float tile[64][65];
  const int c4 = threadIdx.x & 15, rq = threadIdx.x >> 4;
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int rr = rq + 16 * i;
    const int64_t r = r0 + rr, c = c0 + 4 * c4;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (r < R && c < C) {
      v = *(const float4*)(in + r * ldi + c);
      if (add) {
        const float4 b = *(const float4*)(add + r * ldi + c);
        v = make_float4(v.x + b.x, v.y + b.y, v.z + b.z, v.w + b.w);
      }
    }
    const float x[4] = {v.x * scale, v.y * scale, v.z * scale, v.w * scale};
#pragma unroll
    for (int q = 0; q < 4; ++q) tile[rr][4 * c4 + q] = x[q];
    if (rows.p[0] && r < R && c < C) {
      u16 o[4][3];
#pragma unroll
      for (int q = 0; q < 4; ++q) split_to(x[q], 3, o[q]);
#pragma unroll
      for (int p = 0; p < 3; ++p)
        *(uint2*)(rows.p[p] + r * ldr + c) = make_uint2((uint32_t)o[0][p] | ((uint32_t)o[1][p] << 16),
                                                        (uint32_t)o[2][p] | ((uint32_t)o[3][p] << 16));
    }
  }
  __syncthreads();
  float scl = 1.0f;
  if constexpr (F16T) {
    const float a = amax_of_slots(sc.amax_a), b = sc.amax_b ? amax_of_slots(sc.amax_b) : 0.0f;
    const int e = f16_scale_exp(fmaxf(a, b)) - (sc.amax_b ? 1 : 0);
    scl = ldexpf(1.0f, e);
    if (sc.inv_out && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) *sc.inv_out = ldexpf(1.0f, -e);
  }
  const int rg = threadIdx.x & 7;
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    const int cc = (threadIdx.x >> 3) + 32 * pass;
    const int64_t c = c0 + cc;
    if (c >= C) continue;
    u16 o[8][3];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if constexpr (F16T) {
        split2_f16(tile[8 * rg + i][cc] * scl, o[i][0], o[i][1]);
        o[i][2] = 0;
      } else {
        split_to(tile[8 * rg + i][cc], nterms, o[i]);
      }
    }
#pragma unroll
    for (int p = 0; p < 3; ++p) {
      if (p >= nterms) break;
      uint32_t w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = (uint32_t)o[2 * i][p] | ((uint32_t)o[2 * i + 1][p] << 16);
      *(uint4*)(out.p[p] + c * ldo + r0 + 8 * rg) = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

// The row-major planes of an fp32 matrix, 8 elements per thread (C and ldi multiples of 4, ldo a
// multiple of 8, 16-byte aligned input rows and planes): grid x over 2048-column pieces of a row,
// grid y over rows; two 16-byte loads, one 16-byte store per plane, no index division.
__global__ __launch_bounds__(256) void planes_rows8_kernel(const float* __restrict__ in, int64_t R, int64_t C,
                                                           int64_t ldi, PlaneOut out, int nterms, int64_t ldo,
                                                           float scale) {
  const int64_t c = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 8;
  if (c >= ldo) return;
  for (int64_t r = blockIdx.y; r < R; r += gridDim.y) {
    float4 v0 = make_float4(0.f, 0.f, 0.f, 0.f), v1 = v0;
    if (c < C) v0 = *(const float4*)(in + r * ldi + c);
    if (c + 4 < C) v1 = *(const float4*)(in + r * ldi + c + 4);
    const float x[8] = {v0.x * scale, v0.y * scale, v0.z * scale, v0.w * scale,
                        v1.x * scale, v1.y * scale, v1.z * scale, v1.w * scale};
    u16 o[8][3];
#pragma unroll
    for (int k = 0; k < 8; ++k) split_to(x[k], nterms, o[k]);
#pragma unroll
    for (int p = 0; p < 3; ++p) {
      if (p >= nterms) break;
      uint32_t w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = (uint32_t)o[2 * i][p] | ((uint32_t)o[2 * i + 1][p] << 16);
      *(uint4*)(out.p[p] + r * ldo + c) = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

bs_status launch_planes(const void* in, bs_dtype dt, int64_t R, int64_t C, int64_t ldi, bool transpose,
                        u16* const* outp, int nterms, int64_t ldo, float scale, hipStream_t st) {
  if (nterms < 1 || nterms > 3) return BS_EINVAL;
  PlaneOut out{{outp[0], nterms > 1 ? outp[1] : nullptr, nterms > 2 ? outp[2] : nullptr}};
  if (transpose) {
    if (C <= 0 || ldo <= 0) return BS_OK;
    dim3 grid((unsigned)((C + 63) / 64), (unsigned)((ldo + 63) / 64));
    const bool vec = dt == BS_BF16 && nterms == 1 && scale == 1.0f && C % 8 == 0 && ldi % 8 == 0 && ldo % 64 == 0 &&
                     ((uintptr_t)in & 15) == 0 && ((uintptr_t)outp[0] & 15) == 0;
    bool vecf = dt == BS_F32 && C % 4 == 0 && ldi % 4 == 0 && ldo % 64 == 0 && ((uintptr_t)in & 15) == 0;
    for (int p = 0; p < nterms; ++p) vecf = vecf && ((uintptr_t)outp[p] & 15) == 0;
    if (vec)
      transpose_bf16_kernel<<<grid, 256, 0, st>>>((const u16*)in, R, C, ldi, outp[0], ldo);
    else if (vecf)
      transpose_split_f32_kernel<false><<<grid, 256, 0, st>>>((const float*)in, nullptr, R, C, ldi, out, nterms, ldo,
                                                              scale, PlaneOut{{nullptr, nullptr, nullptr}}, 0,
                                                              F16Scale{});
    else if (dt == BS_F32)
      planes_t_kernel<float><<<grid, 256, 0, st>>>((const float*)in, R, C, ldi, out, nterms, ldo, scale);
    else
      planes_t_kernel<u16><<<grid, 256, 0, st>>>((const u16*)in, R, C, ldi, out, nterms, ldo, scale);
  } else {
    const int64_t n = R * ldo;
    if (n <= 0) return BS_OK;
    const int64_t want = (n + 255) / 256;
    const unsigned blocks = (unsigned)(want < 8192 ? want : 8192);
    bool vec8 = dt == BS_F32 && C % 4 == 0 && ldi % 4 == 0 && ldo % 8 == 0 && ((uintptr_t)in & 15) == 0;
    for (int p = 0; p < nterms; ++p) vec8 = vec8 && ((uintptr_t)outp[p] & 15) == 0;
    bool vec4 = dt == BS_F32 && C % 4 == 0 && ldi % 4 == 0 && ldo % 4 == 0 && ((uintptr_t)in & 15) == 0;
    for (int p = 0; p < nterms; ++p) vec4 = vec4 && ((uintptr_t)outp[p] & 7) == 0;
    if (vec8) {
      const dim3 grid((unsigned)((ldo / 8 + 255) / 256), (unsigned)(R < 65535 ? R : 65535));
      planes_rows8_kernel<<<grid, 256, 0, st>>>((const float*)in, R, C, ldi, out, nterms, ldo, scale);
    } else if (vec4) {
      const int64_t want4 = (n / 4 + 255) / 256;
      planes_rows4_kernel<<<(unsigned)(want4 < 8192 ? want4 : 8192), 256, 0, st>>>((const float*)in, R, C, ldi, out,
                                                                                   nterms, ldo, scale);
    } else if (dt == BS_F32)
      planes_rows_kernel<float><<<blocks, 256, 0, st>>>((const float*)in, R, C, ldi, out, nterms, ldo, scale);
    else
      planes_rows_kernel<u16><<<blocks, 256, 0, st>>>((const u16*)in, R, C, ldi, out, nterms, ldo, scale);
  }
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status launch_planes_t2(const float* in, const float* add, int64_t R, int64_t C, int64_t ldi, u16* const* outT,
                           int nterms, int64_t ldo, u16* const* outR, int64_t ldr, hipStream_t st, F16Scale sc) {
  if (nterms < 1 || nterms > 3 || (sc.amax_a && nterms != 2)) return BS_EINVAL;
  if (C <= 0 || ldo <= 0) return BS_OK;
  bool ok = C % 4 == 0 && ldi % 4 == 0 && ldo % 64 == 0 && ((uintptr_t)in & 15) == 0 && ((uintptr_t)add & 15) == 0 &&
            (!outR || (ldr % 4 == 0 && ldr >= C));
  for (int p = 0; p < nterms; ++p) ok = ok && outT[p] && ((uintptr_t)outT[p] & 15) == 0;
  // the row-major planes are always the three bf16 terms, whatever nterms
  for (int p = 0; outR && p < 3; ++p) ok = ok && outR[p] && ((uintptr_t)outR[p] & 7) == 0;
  if (!ok) return BS_EINVAL;
  const PlaneOut out{{outT[0], nterms > 1 ? outT[1] : nullptr, nterms > 2 ? outT[2] : nullptr}};
  const PlaneOut rows{{outR ? outR[0] : nullptr, outR ? outR[1] : nullptr, outR ? outR[2] : nullptr}};
  const dim3 grid((unsigned)((C + 63) / 64), (unsigned)((ldo + 63) / 64));
  if (sc.amax_a)
    transpose_split_f32_kernel<true><<<grid, 256, 0, st>>>(in, add, R, C, ldi, out, nterms, ldo, 1.0f, rows, ldr, sc);
  else
    transpose_split_f32_kernel<false><<<grid, 256, 0, st>>>(in, add, R, C, ldi, out, nterms, ldo, 1.0f, rows, ldr, sc);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

// ------------------------------------------------------------------------------------
// Trial statistics: per column j of delta [K][m], mean over trials (fp64, trials in
// order), sample variance by a second pass, se = sd / sqrt(K); block partial sums of
// mean^2, ref^2 and se^2 (fp64), combined in block order by one more kernel.
// ------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void trial_stats_kernel(const float* __restrict__ delta, int K, int64_t m,
                                                          const float* __restrict__ g_ref, float* __restrict__ mean_err,
                                                          float* __restrict__ se, double* __restrict__ part) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  double mean = 0.0, var = 0.0, ref = 0.0;
  if (j < m) {
    // mean = d_1 + (1/K) sum_k (d_k - d_1): exactly d_1 when every trial agrees
    const double d1 = delta[j];
    double s = 0.0;
    for (int k = 1; k < K; ++k) s += (double)delta[(int64_t)k * m + j] - d1;
    mean = d1 + s / K;
    double q = 0.0;
    for (int k = 0; k < K; ++k) {
      const double e = (double)delta[(int64_t)k * m + j] - mean;
      q += e * e;
    }
    var = K > 1 ? q / (K - 1) / K : 0.0;
    mean_err[j] = (float)mean;
    if (se) se[j] = (float)sqrt(var);
    if (g_ref) ref = g_ref[j];
  }
  __shared__ double red[3][4];
  double v[3] = {mean * mean, ref * ref, var};
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int i = 0; i < 3; ++i) {
    const double s = wave_sum_f64(v[i]);
    if (lane == 0) red[i][w] = s;
  }
  __syncthreads();
  if (threadIdx.x < 3) {
    const int i = threadIdx.x;
    part[(int64_t)blockIdx.x * 3 + i] = ((red[i][0] + red[i][1]) + red[i][2]) + red[i][3];
  }
}

// One block of 256 threads: thread i adds the partials of blocks i, i + 256, ... in order, then a
// fixed pairwise tree (offsets 128, 64, ..., 1) combines the threads (deterministic).
__global__ __launch_bounds__(256) void trial_summary_kernel(const double* __restrict__ part, int64_t nblk,
                                                            double* __restrict__ summary) {
  __shared__ double red[3][256];
  double s[3] = {0.0, 0.0, 0.0};
  for (int64_t b = threadIdx.x; b < nblk; b += 256)
    for (int i = 0; i < 3; ++i) s[i] += part[b * 3 + i];
  for (int i = 0; i < 3; ++i) red[i][threadIdx.x] = s[i];
  __syncthreads();
  for (int off = 128; off >= 1; off >>= 1) {
    if ((int)threadIdx.x < off)
      for (int i = 0; i < 3; ++i) red[i][threadIdx.x] += red[i][threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    summary[0] = sqrt(red[0][0]);
    summary[1] = sqrt(red[1][0]);
    summary[2] = red[2][0] > 0.0 ? red[0][0] / red[2][0] : __builtin_nan("");
  }
}

bs_status launch_policy_bias(const float* delta, int K, int64_t m, const float* g_ref, float* mean_err, float* se,
                             double* summary, double* ws, hipStream_t st) {
  const int64_t nblk = (m + 255) / 256;
  if (nblk > 0)
    trial_stats_kernel<<<(unsigned)nblk, 256, 0, st>>>(delta, K, m, g_ref, mean_err, se, ws);
  if (summary) trial_summary_kernel<<<1, 256, 0, st>>>(ws, nblk, summary);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

}  // namespace bsp
