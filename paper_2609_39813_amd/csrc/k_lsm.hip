// The log-softmax operator test (Sec. 4.3; App. C.5) on the GPU, in fp64 as the paper's test:
// the operator's backward h - exp(S) (1^T h) reads a saved output S = l + r (r_j = +-eps) under
// reuse, or l + r' with r' drawn anew; per trial the statistic is the mean over rows and classes
// of (g - g*) / p under the likelihood (h = -e_y) and the constructed loss (h = r).
//
// One wave per (row, chunk of trials); a lane takes groups of 4 consecutive classes (one Philox
// call per group, draw and trial). Per trial the wave first sums r over the row (the constructed
// loss's 1^T h), then forms the four errors literally (g and g* in fp64, then / p). Per-trial
// row sums go to the workspace; a second kernel sums them over rows in row order and takes the
// mean and se over trials.
#include "bsp_kernels.h"

namespace bsp {

namespace {

constexpr int LSM_TCH = 32;  // trials per wave

__device__ __forceinline__ double wsum(double v) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// l = z - max - log(sum exp(z - max)) per row, one wave per row, and the three values every
// trial's exponentials take (the saved output is l + r with r = +eps or -eps exactly):
// p = exp(l), ep = exp(l + eps) / cal and em = exp(l - eps) / cal
__global__ __launch_bounds__(64) void lsm_prep_kernel(const double* __restrict__ z, int64_t rows, int C, double eps,
                                                      double cal, double* __restrict__ p, double* __restrict__ ep,
                                                      double* __restrict__ em) {
  const int64_t row = blockIdx.x;
  const int lane = threadIdx.x;
  const double* zr = z + row * C;
  double m = -INFINITY;
  for (int j = lane; j < C; j += 64) m = fmax(m, zr[j]);
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) m = fmax(m, __shfl_xor(m, off, 64));
  double se = 0.0;
  for (int j = lane; j < C; j += 64) se += exp(zr[j] - m);
  const double lse = m + log(wsum(se));
  for (int j = lane; j < C; j += 64) {
    const double lj = zr[j] - lse;
    const int64_t e = row * C + j;
    p[e] = exp(lj);
    ep[e] = exp(lj + eps) / cal;
    em[e] = exp(lj + -eps) / cal;
  }
}

// per (row, trial): the row sums of the four entry errors, [4][K][rows]
__global__ __launch_bounds__(64) void lsm_trial_kernel(const double* __restrict__ pv, const double* __restrict__ epv,
                                                       const double* __restrict__ emv, const int32_t* __restrict__ y,
                                                       int64_t rows, int C, double eps, int K, uint64_t seed,
                                                       uint32_t use_r, uint32_t use_p, double* __restrict__ part) {
  const int64_t row = blockIdx.x;
  const int lane = threadIdx.x;
  const int yt = y[row];
  const double sh = (yt >= 0 && yt < C) ? -1.0 : 0.0;
  const int ngroups = C / 4;
  const int k_end = min(K, (int)(blockIdx.y + 1) * LSM_TCH);
  for (int k = blockIdx.y * LSM_TCH; k < k_end; ++k) {
    const uint32_t trial = (uint32_t)(k + 1);
    // 1^T r over the row
    double sr = 0.0;
    for (int gi = lane; gi < ngroups; gi += 64) {
      const Philox4 pr = philox_group(seed, (uint64_t)(row * C) / 4 + gi, trial, use_r);
      const uint32_t R[4] = {pr.w0, pr.w1, pr.w2, pr.w3};
#pragma unroll
      for (int q = 0; q < 4; ++q) sr += R[q] >= 0x80000000u ? eps : -eps;
    }
    sr = wsum(sr);
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    for (int gi = lane; gi < ngroups; gi += 64) {
      const uint64_t grp = (uint64_t)(row * C) / 4 + gi;
      const Philox4 pr = philox_group(seed, grp, trial, use_r);
      const Philox4 pp = philox_group(seed, grp, trial, use_p);
      const uint32_t R[4] = {pr.w0, pr.w1, pr.w2, pr.w3}, Rp[4] = {pp.w0, pp.w1, pp.w2, pp.w3};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int j = 4 * gi + q;
        const int64_t e = row * C + j;
        const double p = pv[e];
        const bool ur = R[q] >= 0x80000000u, urp = Rp[q] >= 0x80000000u;
        const double r = ur ? eps : -eps;
        const double er = ur ? epv[e] : emv[e], erp = urp ? epv[e] : emv[e];
        // likelihood: h = -e_y, 1^T h = sh (-1, or 0 for a target outside the classes)
        const double hl = j == yt ? -1.0 : 0.0;
        const double gl_star = hl - p * sh;
        acc[0] += ((hl - er * sh) - gl_star) / p;
        acc[1] += ((hl - erp * sh) - gl_star) / p;
        // constructed: h = r, 1^T h = sr
        const double gc_star = r - p * sr;
        acc[2] += ((r - er * sr) - gc_star) / p;
        acc[3] += ((r - erp * sr) - gc_star) / p;
      }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const double v = wsum(acc[c]);
      if (lane == 0) part[((int64_t)c * K + k) * rows + row] = v;
    }
  }
}

// per statistic: t_k = sum over rows (row order) / (rows C); mean and se over trials
constexpr int LSM_RT = 64;  // trials per block of the first reduction stage

// mean over rows and classes of statistic c in trial k: one wave, rows lane-strided, combined by
// a fixed xor tree (every lane ends with the total)
__device__ __forceinline__ double lsm_trial_mean(const double* __restrict__ part, int64_t rows, int C, int K, int c,
                                                 int k) {
  const int lane = threadIdx.x & 63;
  double t = 0.0;
  for (int64_t i = lane; i < rows; i += 64) t += part[((int64_t)c * K + k) * rows + i];
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) t += __shfl_xor(t, off, 64);
  return t / ((double)rows * C);
}

// first stage: block (j, c) takes trials 64 j .. 64 j + 63 of statistic c and writes their sums of
// d_k = m_k - m_0 and d_k^2 (shifted by trial 0's mean m_0, which block (0, c) also writes)
__global__ __launch_bounds__(256) void lsm_reduce_kernel(const double* __restrict__ part, int64_t rows, int C, int K,
                                                         double* __restrict__ acc, double* __restrict__ m0) {
  const int c = blockIdx.y, w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const double t0 = lsm_trial_mean(part, rows, C, K, c, 0);
  double s1 = 0.0, s2 = 0.0;
  for (int j = w; j < LSM_RT; j += 4) {
    const int k = blockIdx.x * LSM_RT + j;
    if (k >= K) break;  // wave-uniform
    const double d = lsm_trial_mean(part, rows, C, K, c, k) - t0;
    s1 += d;
    s2 += d * d;
  }
  __shared__ double red[2][4];
  if (lane == 0) {
    red[0][w] = s1;
    red[1][w] = s2;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double* o = acc + 2 * ((int64_t)c * gridDim.x + blockIdx.x);
    o[0] = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
    o[1] = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
    if (blockIdx.x == 0) m0[c] = t0;
  }
}

// second stage: block c sums its nb partials (thread-strided, then a fixed tree) into the mean
// and its standard error over the K trials
__global__ __launch_bounds__(256) void lsm_final_kernel(const double* __restrict__ acc, const double* __restrict__ m0,
                                                        int nb, int K, double* __restrict__ stats) {
  const int c = blockIdx.x;
  __shared__ double red[2][256];
  double s1 = 0.0, s2 = 0.0;
  for (int j = threadIdx.x; j < nb; j += 256) {
    s1 += acc[2 * ((int64_t)c * nb + j)];
    s2 += acc[2 * ((int64_t)c * nb + j) + 1];
  }
  red[0][threadIdx.x] = s1;
  red[1][threadIdx.x] = s2;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off) {
      red[0][threadIdx.x] += red[0][threadIdx.x + off];
      red[1][threadIdx.x] += red[1][threadIdx.x + off];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double S1 = red[0][0], S2 = red[1][0];
    const double var = K > 1 ? fmax(S2 - S1 * S1 / K, 0.0) / (K - 1) : 0.0;
    stats[2 * c] = m0[c] + S1 / K;
    stats[2 * c + 1] = sqrt(var / K);
  }
}

}  // namespace

size_t lsm_ws_size(int64_t rows, int C, int K) {
  if (rows < 1 || C < 4 || (C & 3) || K < 1) return 0;
  Carver c;
  for (int i = 0; i < 3; ++i) c.take<double>(rows * C);
  c.take<double>((int64_t)4 * K * rows);
  c.take<double>((int64_t)8 * ((K + LSM_RT - 1) / LSM_RT));
  c.take<double>(4);
  return c.used();
}

}  // namespace bsp

using namespace bsp;

extern "C" {

size_t bs_logsoftmax_check_workspace_size(int64_t rows, int C, int K) { return lsm_ws_size(rows, C, K); }

bs_status bs_logsoftmax_reuse_check(const double* logits, const int32_t* target, int64_t rows, int C, double eps,
                                    int K, uint64_t seed, uint32_t store_id, int calibrate, double* stats, void* ws,
                                    size_t ws_bytes, void* stream) {
  if (!logits || !target || !stats) return BS_EINVAL;
  if (rows < 1 || K < 1 || K > (1 << 20) || !(eps > 0.0) || !(eps < 1.0)) return BS_EINVAL;
  if (C < 4 || (C & 3) || rows > 0x7FFFFFFF) return BS_ESHAPE;
  const size_t need = lsm_ws_size(rows, C, K);
  if (!ws || ((uintptr_t)ws & 255) || ws_bytes < need) return BS_EWORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  Carver c(ws, ws_bytes);
  double* pv = c.take<double>(rows * C);
  double* epv = c.take<double>(rows * C);
  double* emv = c.take<double>(rows * C);
  double* part = c.take<double>((int64_t)4 * K * rows);
  const int nb = (K + LSM_RT - 1) / LSM_RT;
  double* acc = c.take<double>((int64_t)8 * nb);
  double* m0 = c.take<double>(4);
  {
    ProfScope prof("lsm_prep", st);
    lsm_prep_kernel<<<(unsigned)rows, 64, 0, st>>>(logits, rows, C, eps, calibrate ? cosh(eps) : 1.0, pv, epv, emv);
    BS_CHECK_LAUNCH();
  }
  const uint32_t base = store_id * 256u;
  {
    ProfScope prof("lsm_trial", st);
    const dim3 grid((unsigned)rows, (unsigned)((K + LSM_TCH - 1) / LSM_TCH));
    lsm_trial_kernel<<<grid, 64, 0, st>>>(pv, epv, emv, target, rows, C, eps, K, seed, base, base + 1, part);
    BS_CHECK_LAUNCH();
  }
  {
    ProfScope prof("lsm_reduce", st);
    lsm_reduce_kernel<<<dim3((unsigned)nb, 4), 256, 0, st>>>(part, rows, C, K, acc, m0);
    lsm_final_kernel<<<4, 256, 0, st>>>(acc, m0, nb, K, stats);
    BS_CHECK_LAUNCH();
  }
  return BS_OK;
}

}  // extern "C"
