// E5M2-gradient Linear backward: residual operand planes of the policy biases and the
// coupling statistic between the two uses of a rounded incoming gradient.
#include "k_linear.h"

namespace bsp {

// Mean over the K trials of a use's new roundings minus the incoming gradient:
// E = s sign (lo + n_up step / K) - dY = s sign (mi K + n_up) step / K - dY, evaluated in
// fp64 (the integer and the power-of-two step are exact) and rounded once to fp32, then
// split into three exact bf16 terms.
__device__ __forceinline__ float resid_value(const ResidArgs& a, int64_t e, float s) {
  const float g = bf16_to_f32(a.dY[e]);
  const float y = div_scale(g, 1.0 / (double)s);
  const Bracket b = f8_bracket(fminf(fabsf(y), a.f.fmax), a.f);
  const double num = ((double)b.mi * a.K + (double)a.counts[e]) * (double)f8_step(b);
  double mv = num / a.K;
  if (signbit(y)) mv = -mv;
  return (float)((double)s * mv - (double)g);
}

__global__ __launch_bounds__(256) void resid_planes_kernel(ResidArgs a) {
  __shared__ u16 tile[3][64][66];
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
  const float s = *a.scale;
#pragma unroll 2
  for (int i = 0; i < 16; ++i) {
    const int rr = ty + 4 * i;
    const int64_t r = r0 + rr, c = c0 + tx;
    u16 o[3] = {0, 0, 0};
    if (r < a.M && c < a.n) {
      split3(resid_value(a, r * a.n + c, s), o[0], o[1], o[2]);
      if (a.rows[0])
        for (int p = 0; p < 3; ++p) a.rows[p][r * a.n + c] = o[p];
    }
    if (a.cols[0])
      for (int p = 0; p < 3; ++p) tile[p][rr][tx] = o[p];
  }
  if (!a.cols[0]) return;
  __syncthreads();
#pragma unroll 2
  for (int i = 0; i < 16; ++i) {
    const int cc = ty + 4 * i;
    const int64_t c = c0 + cc, r = r0 + tx;
    if (c < a.n && r < a.ldo)
      for (int p = 0; p < 3; ++p) a.cols[p][c * a.ldo + r] = tile[p][tx][cc];
  }
}

bs_status launch_resid_planes(const ResidArgs& a, hipStream_t st) {
  if (a.n <= 0) return BS_OK;
  const int64_t rows = a.cols[0] ? (a.ldo > a.M ? a.ldo : a.M) : a.M;
  if (rows <= 0) return BS_OK;
  dim3 grid((unsigned)((a.n + 63) / 64), (unsigned)((rows + 63) / 64));
  resid_planes_kernel<<<grid, 256, 0, st>>>(a);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

__global__ __launch_bounds__(256) void kappa_fixed_kernel(const u16* __restrict__ dY, const float* __restrict__ scale,
                                                          F8 f, int64_t n_el, const float* __restrict__ AW,
                                                          const float* __restrict__ XB, double* __restrict__ part) {
  const float s = *scale;
  const double rs = 1.0 / (double)s;
  double a0 = 0.0, b0 = 0.0;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < n_el; e += (int64_t)gridDim.x * 256) {
    const float g = bf16_to_f32(dY[e]);
    const float y = div_scale(g, rs);
    const Bracket b = f8_bracket(fminf(fabsf(y), f.fmax), f);
    double lo = (double)b.mi * (double)f8_step(b);
    if (signbit(y)) lo = -lo;
    const double r = (double)s * lo - (double)g;
    a0 += r * (double)AW[e];
    b0 += r * (double)XB[e];
  }
  __shared__ double red[2][4];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  a0 = wave_sum_f64(a0);
  b0 = wave_sum_f64(b0);
  if (lane == 0) {
    red[0][w] = a0;
    red[1][w] = b0;
  }
  __syncthreads();
  if (threadIdx.x < 2) {
    const int i = threadIdx.x;
    part[(int64_t)blockIdx.x * 2 + i] = ((red[i][0] + red[i][1]) + red[i][2]) + red[i][3];
  }
}

__global__ void kappa_fixed_final(const double* __restrict__ part, int nblk, double* __restrict__ out) {
  if (threadIdx.x >= 2) return;
  double v = 0.0;
  for (int b = 0; b < nblk; ++b) v += part[b * 2 + threadIdx.x];
  out[threadIdx.x] = v;
}

bs_status launch_kappa_fixed(const u16* dY, const float* scale, int fmt, int64_t M, int64_t n, const float* AW,
                             const float* XB, double* part, double* out, hipStream_t st) {
  const int nblk = 1024;
  kappa_fixed_kernel<<<nblk, 256, 0, st>>>(dY, scale, f8_format(fmt), M * n, AW, XB, part);
  kappa_fixed_final<<<1, 64, 0, st>>>(part, nblk, out);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

// one wave: trial sums of the block partials (blocks in order, per trial), then the mean
// of the per-trial products in trial order
__global__ void kappa_final_kernel(const double* __restrict__ fixed, const double* __restrict__ pa, int ia,
                                   const double* __restrict__ pb, int ib, int64_t nblk, int K,
                                   const float* __restrict__ scale, double* __restrict__ kappa) {
  __shared__ double prod[4096];
  const double s = *scale;
  for (int k = threadIdx.x; k < K; k += blockDim.x) {
    double sa = 0.0, sb = 0.0;
    const double* qa = pa + ((int64_t)k * 2 + ia) * nblk;
    const double* qb = pb + ((int64_t)k * 2 + ib) * nblk;
    for (int64_t b = 0; b < nblk; ++b) {
      sa += qa[b];
      sb += qb[b];
    }
    prod[k] = (fixed[0] + s * sa) * (fixed[1] + s * sb);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double m = 0.0;
    for (int k = 0; k < K; ++k) m += prod[k];
    *kappa = m / K;
  }
}

bs_status launch_kappa_final(const double* fixed, const double* pa, int ia, const double* pb, int ib, int64_t nblk,
                             int K, const float* scale, double* kappa, hipStream_t st) {
  if (K > 4096) return BS_EINVAL;
  kappa_final_kernel<<<1, 256, 0, st>>>(fixed, pa, ia, pb, ib, nblk, K, scale, kappa);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

}  // namespace bsp
