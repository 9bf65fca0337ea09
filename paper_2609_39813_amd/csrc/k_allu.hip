// Kernels of the "every use at once" check of the decoder layer (declared in k_allu.h).
#include "k_allu.h"

namespace bsp {

namespace {

// What a use reads of four consecutive store elements e0 .. e0 + 3 (e0 a multiple of 4): the
// original x (U), the forward's rounding s val(C) (R), or a new stochastic rounding of fl32(x / s)
// at the same scale (N; Philox word e & 3 of the call keyed (seed; e0 >> 2, trial, use)). fp64.
__device__ __forceinline__ void read4(const StoreRead& r, int64_t e0, const float (&x)[4], double rs, float s,
                                      double (&v)[4]) {
  if (r.letter == LETTER_U) {
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = x[i];
  } else if (r.letter == LETTER_R) {
    const uint32_t w = *(const uint32_t*)(r.codes + e0);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = (double)s * (double)f8_value((w >> (8 * i)) & 0xFFu, r.f);
  } else {
    const Philox4 p = philox_group(r.seed, (uint64_t)(e0 >> 2), r.trial, r.use);
    const uint32_t R[4] = {p.w0, p.w1, p.w2, p.w3};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float y = div_scale(x[i], rs);
      const Bracket b = f8_bracket(fminf(fabsf(y), r.f.fmax), r.f);
      const double mag = (double)(b.mi + sr_up(b.F, R[i])) * (double)f8_step(b);
      v[i] = (signbit(y) ? -mag : mag) * (double)s;
    }
  }
}

__device__ __forceinline__ void load4(const float* p, int64_t e, float (&v)[4]) {
  const float4 q = *(const float4*)(p + e);
  v[0] = q.x;
  v[1] = q.y;
  v[2] = q.z;
  v[3] = q.w;
}
__device__ __forceinline__ void load4(const u16* p, int64_t e, float (&v)[4]) {
  const uint2 q = *(const uint2*)(p + e);
  v[0] = bf16_to_f32((u16)(q.x & 0xFFFF));
  v[1] = bf16_to_f32((u16)(q.x >> 16));
  v[2] = bf16_to_f32((u16)(q.y & 0xFFFF));
  v[3] = bf16_to_f32((u16)(q.y >> 16));
}

constexpr int ALLU_RT = 16;  // rows per tile of the gain use's partial sums

// block: 256 threads x 4 consecutive columns (1024 columns), rows [16 y, 16 y + 16)
template <typename XT>
__global__ __launch_bounds__(256) void allu_gain_kernel(AlluGainArgs<XT> a) {
  const int64_t j0 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (j0 >= a.d) return;
  const int64_t t0 = (int64_t)blockIdx.y * ALLU_RT;
  const float s = a.rd.scale ? *a.rd.scale : 1.0f;
  const double rs = 1.0 / (double)s;
  float g[4];
  load4(a.gain, j0, g);
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  for (int i = 0; i < ALLU_RT; ++i) {
    const int64_t t = t0 + i;
    if (t >= a.T) break;
    const int64_t e = t * a.d + j0;
    const float r = a.rstd[t];
    float x[4], u[4], du[4], ddu[4] = {0.f, 0.f, 0.f, 0.f};
    load4(a.X, e, x);
    load4(a.rd.x, e, u);
    load4(a.du, e, du);
    if (a.ddu) load4(a.ddu, e, ddu);
    double v[4];
    read4(a.rd, e, u, rs, s, v);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const float z = x[c] * r;  // the forward's fp32 z
      const double zg = a.rd.letter == LETTER_U ? (double)z : v[c] / (double)g[c];
      // z_g (du + ddu) - z du = (z_g - z)(du + ddu) + z ddu
      acc[c] += (zg - (double)z) * ((double)du[c] + (double)ddu[c]) + (double)z * (double)ddu[c];
    }
  }
#pragma unroll
  for (int c = 0; c < 4; ++c) a.part[(int64_t)blockIdx.y * a.d + j0 + c] = acc[c];
}

// one wave per row, 4 rows per block; columns in groups of 4 per lane
// NI > 0: the row's columns in NI chunks of 256 (d <= 256 NI), each lane keeping x, z_x and
// gain ddu of the first pass in registers for the second (the letter's read, a Philox draw and
// an fp64 division per element, is taken once); NI == 0: any d, the second pass reads and
// computes again.
// GAIN: also the gain use's terms (z_g - z)(du + ddu) + z ddu of this row, z_g from the gain use's
// read rd_g, added to accg[4 lane + 256 it + c] (LDS) for the lane's columns (NI > 0 only).
template <typename XT, int NI, bool GAIN = false>
__device__ __forceinline__ float allu_dx_row(const AlluDxArgs<XT>& a, int64_t t, int lane,
                                             const StoreRead* rd_g = nullptr, double* accg = nullptr) {
  static_assert(!GAIN || NI > 0, "the gain terms need the kept columns");
  const float s = a.rd.scale ? *a.rd.scale : 1.0f;
  const double rs = 1.0 / (double)s;
  const float r = a.rstd[t];
  const int64_t rowe = t * a.d;
  constexpr int NK = NI > 0 ? NI : 1;
  float xk[NK][4], dk[NK][4];  // x and ddu, kept for the second pass (NI > 0)
  double zk[NK][4];
  double dref = 0.0, dl = 0.0;
  // first pass: the two row sums (and, NI > 0, the kept values)
  auto first = [&](int64_t j0, int it) {
    float x[4], u[4], du[4], ddu[4] = {0.f, 0.f, 0.f, 0.f}, g[4];
    load4(a.X, rowe + j0, x);
    load4(a.rd.x, rowe + j0, u);
    load4(a.du, rowe + j0, du);
    load4(a.gain, j0, g);
    if (a.ddu) load4(a.ddu, rowe + j0, ddu);
    double v[4];
    read4(a.rd, rowe + j0, u, rs, s, v);
    double vg[4];
    if constexpr (GAIN) {
      if (rd_g->letter == LETTER_N) {
        read4(*rd_g, rowe + j0, u, rs, s, vg);
      } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) vg[c] = v[c];  // U and R read the same at both uses
      }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const double z = (double)(x[c] * r);
      // GAIN: the two uses' reads over one reciprocal of the gain (v / g as v (1 / g), within an
      // fp64 ulp); else the division
      const double ig = GAIN ? 1.0 / (double)g[c] : 0.0;
      const double zx = a.rd.letter == LETTER_U ? z : GAIN ? v[c] * ig : v[c] / (double)g[c];
      dref += (double)g[c] * (double)du[c] * z;
      dl += (double)g[c] * ((double)du[c] + (double)ddu[c]) * zx;
      if constexpr (NI > 0) {
        xk[it][c] = x[c];
        zk[it][c] = zx;
        dk[it][c] = ddu[c];
      }
      if constexpr (GAIN) {
        const double zg = rd_g->letter == LETTER_U ? z : vg[c] * ig;
        accg[4 * lane + 256 * it + c] += (zg - z) * ((double)du[c] + (double)ddu[c]) + z * (double)ddu[c];
      }
    }
  };
  if constexpr (NI > 0) {
#pragma unroll
    for (int it = 0; it < NI; ++it)
      if (4 * (int64_t)lane + 256 * it < a.d) first(4 * (int64_t)lane + 256 * it, it);
  } else {
    for (int64_t j0 = 4 * (int64_t)lane; j0 < a.d; j0 += 256) first(j0, 0);
  }
  dref = __shfl(wave_sum_f64(dref), 0, 64);  // the wave sum is valid in lane 0: broadcast it
  dl = __shfl(wave_sum_f64(dl), 0, 64);
  const double inv_d = 1.0 / (double)a.d;
  float mx = 0.0f;
  // second pass: out = r (gain ddu - (z_x dl - z dref) / d) + add
  auto second = [&](int64_t j0, const float (&x)[4], const double (&zx)[4], const float (&ddu)[4]) {
    float ad[4] = {0.f, 0.f, 0.f, 0.f}, g[4];
    if (a.add) load4(a.add, rowe + j0, ad);
    load4(a.gain, j0, g);
    float o[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const double z = (double)(x[c] * r);
      const double gd = (double)g[c] * (double)ddu[c];
      o[c] = (float)((double)r * (gd - (zx[c] * dl - z * dref) * inv_d) + (double)ad[c]);
      mx = fmaxf(mx, fabsf(o[c]));
    }
    *(float4*)(a.out + rowe + j0) = make_float4(o[0], o[1], o[2], o[3]);
  };
  if constexpr (NI > 0) {
#pragma unroll
    for (int it = 0; it < NI; ++it)
      if (4 * (int64_t)lane + 256 * it < a.d) second(4 * (int64_t)lane + 256 * it, xk[it], zk[it], dk[it]);
  } else {
    for (int64_t j0 = 4 * (int64_t)lane; j0 < a.d; j0 += 256) {
      float x[4], u[4], ddu[4] = {0.f, 0.f, 0.f, 0.f}, g[4];
      load4(a.X, rowe + j0, x);
      load4(a.rd.x, rowe + j0, u);
      load4(a.gain, j0, g);
      if (a.ddu) load4(a.ddu, rowe + j0, ddu);
      double v[4], zx[4];
      read4(a.rd, rowe + j0, u, rs, s, v);
#pragma unroll
      for (int c = 0; c < 4; ++c) zx[c] = a.rd.letter == LETTER_U ? (double)(x[c] * r) : v[c] / (double)g[c];
      second(j0, x, zx, ddu);
    }
  }
  return mx;
}
template <typename XT, int NI>
__global__ __launch_bounds__(256) void allu_dx_kernel(AlluDxArgs<XT> a) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const float mx = t < a.T ? allu_dx_row<XT, NI>(a, t, lane) : 0.0f;  // uniform per wave
  if (a.amax) block_amax_to_slot(mx, a.amax);
}

// 16 rows per block (the gain use's tile), 4 consecutive rows per wave; the gain terms of a column
// summed over the wave's rows in order, then over the 4 waves in order through LDS
template <typename XT, int NI>
__global__ __launch_bounds__(256, 3) void allu_gain_dx_kernel(AlluGainDxArgs<XT> a) {
  __shared__ double red[4][256 * NI];  // per wave, the gain terms of its rows by column
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int j = lane; j < 256 * NI; j += 64) red[w][j] = 0.0;  // each lane's own columns below
  float mx = 0.0f;
  for (int i = 0; i < 4; ++i) {
    const int64_t t = (int64_t)blockIdx.x * ALLU_RT + 4 * w + i;
    if (t < a.dx.T) mx = fmaxf(mx, allu_dx_row<XT, NI, true>(a.dx, t, lane, &a.rd_g, red[w]));  // uniform per wave
  }
  __syncthreads();
  for (int j = threadIdx.x; j < a.dx.d; j += 256)
    a.part[(int64_t)blockIdx.x * a.dx.d + j] = ((red[0][j] + red[1][j]) + red[2][j]) + red[3][j];
  if (a.dx.amax) block_amax_to_slot(mx, a.dx.amax);
}

// 16 lanes per row of 64, 4 elements each; 16 rows per block
__global__ __launch_bounds__(256) void allu_d_kernel(AlluDArgs a) {
  const int64_t row = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
  const int sub = threadIdx.x & 15;
  const bool ok = row < a.rows;
  double acc = 0.0;
  if (ok) {
    const float s = *a.rd.scale;
    const double rs = 1.0 / (double)s;
    const int64_t e = row * 64 + 4 * sub;
    int64_t ed = e;  // ddO's element
    if (a.ddo_heads > 0) {
      const int64_t bh = row / a.ddo_S, s = row - bh * a.ddo_S;
      ed = (((bh / a.ddo_heads) * a.ddo_S + s) * a.ddo_heads + bh % a.ddo_heads) * 64 + 4 * sub;
    }
    float o[4], dO[4], ddO[4] = {0.f, 0.f, 0.f, 0.f};
    load4(a.rd.x, e, o);
    load4(a.dO, e, dO);
    if (a.ddO) load4(a.ddO, ed, ddO);
    double v[4];
    read4(a.rd, e, o, rs, s, v);
#pragma unroll
    for (int c = 0; c < 4; ++c) acc += (double)ddO[c] * v[c] + (double)dO[c] * (v[c] - (double)o[c]);
  }
#pragma unroll
  for (int m = 1; m < 16; m <<= 1) acc += __shfl_xor(acc, m, 64);
  if (ok && sub == 0) a.out[row] = (float)acc;
  if (a.amax) block_amax_to_slot(ok ? fabsf((float)acc) : 0.0f, a.amax);
}

__global__ __launch_bounds__(256) void trial_mean_kernel(const float* __restrict__ d1, const double* __restrict__ S1,
                                                         int K, int64_t m, float* __restrict__ out) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m; i += (int64_t)gridDim.x * blockDim.x)
    out[i] = (float)((double)d1[i] + S1[i] / (double)K);
}

__global__ __launch_bounds__(256) void fill_kernel(float* __restrict__ out, int64_t n, float v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    out[i] = v;
}

unsigned blocks1d(int64_t n) {
  const int64_t b = (n + 255) / 256;
  return (unsigned)(b < 8192 ? (b > 0 ? b : 1) : 8192);
}

}  // namespace

template <typename XT>
bs_status launch_allu_gain(const AlluGainArgs<XT>& a, hipStream_t st) {
  if (a.T <= 0 || a.d <= 0) return BS_OK;
  if (a.d & 3) return BS_ESHAPE;
  const dim3 grid((unsigned)((a.d + 1023) / 1024), (unsigned)((a.T + ALLU_RT - 1) / ALLU_RT));
  allu_gain_kernel<XT><<<grid, 256, 0, st>>>(a);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
template bs_status launch_allu_gain<float>(const AlluGainArgs<float>&, hipStream_t);
template bs_status launch_allu_gain<u16>(const AlluGainArgs<u16>&, hipStream_t);

template <typename XT>
bs_status launch_allu_dx(const AlluDxArgs<XT>& a, hipStream_t st) {
  if (a.T <= 0 || a.d <= 0) return BS_OK;
  if (a.d & 3) return BS_ESHAPE;
  const unsigned grid = (unsigned)((a.T + 3) / 4);
  if (a.d <= 256)
    allu_dx_kernel<XT, 1><<<grid, 256, 0, st>>>(a);
  else if (a.d <= 512)
    allu_dx_kernel<XT, 2><<<grid, 256, 0, st>>>(a);
  else if (a.d <= 1024)
    allu_dx_kernel<XT, 4><<<grid, 256, 0, st>>>(a);
  else
    allu_dx_kernel<XT, 0><<<grid, 256, 0, st>>>(a);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
template bs_status launch_allu_dx<float>(const AlluDxArgs<float>&, hipStream_t);
template bs_status launch_allu_dx<u16>(const AlluDxArgs<u16>&, hipStream_t);

template <typename XT>
bs_status launch_allu_gain_dx(const AlluGainDxArgs<XT>& a, hipStream_t st) {
  const AlluDxArgs<XT>& x = a.dx;
  if (x.T <= 0 || x.d <= 0) return BS_OK;
  if (x.d & 3) return BS_ESHAPE;
  if (a.rd_g.x != x.rd.x || a.rd_g.codes != x.rd.codes || a.rd_g.scale != x.rd.scale || a.rd_g.letter != x.rd.letter)
    return BS_EINVAL;
  if (x.d > 1024) {
    const AlluGainArgs<XT> g{x.X, x.rstd, x.gain, a.rd_g, x.du, x.ddu, x.T, x.d, a.part};
    const bs_status e = launch_allu_gain(g, st);
    return e != BS_OK ? e : launch_allu_dx(x, st);
  }
  const unsigned grid = (unsigned)((x.T + ALLU_RT - 1) / ALLU_RT);
  if (x.d <= 256)
    allu_gain_dx_kernel<XT, 1><<<grid, 256, 0, st>>>(a);
  else if (x.d <= 512)
    allu_gain_dx_kernel<XT, 2><<<grid, 256, 0, st>>>(a);
  else
    allu_gain_dx_kernel<XT, 4><<<grid, 256, 0, st>>>(a);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
template bs_status launch_allu_gain_dx<float>(const AlluGainDxArgs<float>&, hipStream_t);
template bs_status launch_allu_gain_dx<u16>(const AlluGainDxArgs<u16>&, hipStream_t);

bs_status launch_allu_d(const AlluDArgs& a, hipStream_t st) {
  if (a.ddo_heads < 0 || (a.ddo_heads > 0 && (a.ddo_S <= 0 || a.rows % a.ddo_S))) return BS_EINVAL;
  if (a.rows <= 0) return BS_OK;
  allu_d_kernel<<<(unsigned)((a.rows + 15) / 16), 256, 0, st>>>(a);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status launch_trial_mean(const float* d1, const double* S1, int K, int64_t m, float* out, hipStream_t st) {
  if (m <= 0) return BS_OK;
  trial_mean_kernel<<<blocks1d(m), 256, 0, st>>>(d1, S1, K, m, out);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status launch_fill(float* out, int64_t n, float v, hipStream_t st) {
  if (n <= 0) return BS_OK;
  fill_kernel<<<blocks1d(n), 256, 0, st>>>(out, n, v);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

}  // namespace bsp
