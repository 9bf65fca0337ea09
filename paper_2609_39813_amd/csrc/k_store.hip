// FP8 store kernels: amax, scale, quantize (RNE / stochastic), and the K-trial
// stochastic-rounding counter of a store's new roundings.
#include "bsp_kernels.h"

namespace bsp {

__global__ void init_diag_kernel(bs_diag* diag) {
  if (threadIdx.x == 0) {
    diag->nonfinite = 0;
    diag->n_saturated = 0;
    diag->amax = 0.0f;
    diag->scale = 1.0f;
  }
}

// max |x| as the bit pattern of a non-negative float: the integer order of such
// patterns is the float order, and NaN/Inf patterns (>= 0x7F800000) sort above every
// finite value, so one atomicMax also detects non-finite input.
template <typename T>
__global__ __launch_bounds__(256) void amax_kernel(const T* __restrict__ x, int64_t n,
                                                   uint32_t* __restrict__ amax_bits) {
  uint32_t m = 0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const uint32_t b = __float_as_uint(fabsf(load_f32(x, i)));
    m = m > b ? m : b;
  }
  m = wave_max_u32(m);
  __shared__ uint32_t red[4];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (lane == 0) red[w] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t b = red[0];
    for (int i = 1; i < (int)(blockDim.x >> 6); ++i) b = b > red[i] ? b : red[i];
    if (b) atomicMax(amax_bits, b);
  }
}

__global__ void finalize_scale_kernel(bs_diag* diag, const float* scale_in, float* scale_out, float fmax) {
  if (threadIdx.x != 0) return;
  const uint32_t bits = __float_as_uint(diag->amax);
  const bool bad = bits >= 0x7F800000u;
  diag->nonfinite = bad ? 1u : 0u;
  float s;
  if (scale_in) {
    s = *scale_in;
  } else {
    const float amax = diag->amax;
    s = (amax == 0.0f || bad) ? 1.0f : __fdiv_rn(amax, fmax);
  }
  diag->scale = s;
  if (scale_out) *scale_out = s;
}

// One thread per group of 4 consecutive elements (one Philox call).
template <typename T, int MODE>
__global__ __launch_bounds__(256) void quantize_kernel(const T* __restrict__ x, int64_t n, F8 f,
                                                       bs_diag* __restrict__ diag, uint8_t* __restrict__ codes,
                                                       uint64_t seed, uint32_t trial, uint32_t use) {
  if (diag->nonfinite) return;
  const float s = diag->scale;
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t e0 = g * 4;
  uint32_t nsat = 0;
  if (e0 < n) {
    Philox4 p{0, 0, 0, 0};
    if (MODE == BS_SR) p = philox_group(seed, (uint64_t)g, trial, use);
    uint32_t packed = 0;
    const int cnt = (int)((n - e0) < 4 ? (n - e0) : 4);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (q < cnt) {
        const float y = __fdiv_rn(load_f32(x, e0 + q), s);
        float a = fabsf(y);
        if (a > f.fmax) {
          a = f.fmax;
          ++nsat;
        }
        const Bracket b = f8_bracket(a, f);
        const uint32_t up = MODE == BS_SR ? sr_up(sr_threshold(b.frac), philox_word(p, q)) : rne_up(b);
        const uint32_t code = (b.base + b.mi + up) | (signbit(y) ? 0x80u : 0u);
        packed |= code << (8 * q);
      }
    }
    if (cnt == 4 && ((uintptr_t)(codes + e0) & 3) == 0) {
      *(uint32_t*)(codes + e0) = packed;
    } else {
      for (int q = 0; q < cnt; ++q) codes[e0 + q] = (uint8_t)(packed >> (8 * q));
    }
  }
  nsat = wave_sum_u32(nsat);
  if ((threadIdx.x & 63) == 0 && nsat) atomicAdd(&diag->n_saturated, nsat);
}

// K-trial counter of new roundings of a [T, d] store y = fl32(u / s) (d % 4 == 0).
// counts[t, j] = number of trials k in 1..K whose rounding of element t*d + j goes up.
// With PARTIALS, also the per-trial column sums
//   partial[k-1][rt][j] = sum over the block's rows t of up_k(t, j) * sign(y) * step(t, j) * w(t, j)
// (fp64) for a weight w (the gain use's du), one row tile rt = 32 rows per block.
// Block: 256 threads = 64 column groups (4 columns each) x 4 row lanes; 8 rows per thread.
template <bool PARTIALS>
__global__ __launch_bounds__(256) void fresh_count_kernel(const float* __restrict__ u, int64_t T, int64_t d, F8 f,
                                                          const float* __restrict__ scale, uint64_t seed,
                                                          uint32_t use, int K, u16* __restrict__ counts,
                                                          const float* __restrict__ w,
                                                          double* __restrict__ partial) {
  constexpr int RT = 32, RPT = 8;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int64_t j0 = (int64_t)blockIdx.x * 256 + 4 * tx;
  const int64_t t0 = (int64_t)blockIdx.y * RT;
  const bool colok = j0 < d;
  const float s = *scale;
  uint32_t F[RPT][4];
  float c[RPT][4];
  uint32_t cnt[RPT][4];
#pragma unroll
  for (int r = 0; r < RPT; ++r) {
    const int64_t t = t0 + ty + 4 * r;
    const bool ok = colok && t < T;
    float4 uv = ok ? *(const float4*)(u + t * d + j0) : make_float4(0.f, 0.f, 0.f, 0.f);
    float4 wv = make_float4(0.f, 0.f, 0.f, 0.f);
    if (PARTIALS && ok) wv = *(const float4*)(w + t * d + j0);
    const float uu[4] = {uv.x, uv.y, uv.z, uv.w};
    const float ww[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float y = __fdiv_rn(uu[q], s);
      const float a = fminf(fabsf(y), f.fmax);
      const Bracket b = f8_bracket(a, f);
      F[r][q] = ok ? sr_threshold(b.frac) : 0u;
      c[r][q] = PARTIALS ? (signbit(y) ? -1.0f : 1.0f) * f8_step(b) * ww[q] : 0.0f;
      cnt[r][q] = 0;
    }
  }
  __shared__ double red[PARTIALS ? 4 : 1][PARTIALS ? 256 : 1];
  const int64_t nrt = (T + RT - 1) / RT;
  for (int k = 1; k <= K; ++k) {
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
      const int64_t t = t0 + ty + 4 * r;
      const uint64_t g = (uint64_t)((t * d + j0) >> 2);
      const Philox4 p = philox_group(seed, g, (uint32_t)k, use);
      const uint32_t R[4] = {p.w0, p.w1, p.w2, p.w3};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t up = sr_up(F[r][q], R[q]);
        cnt[r][q] += up;
        if (PARTIALS) acc[q] += up ? (double)c[r][q] : 0.0;
      }
    }
    if (PARTIALS) {
#pragma unroll
      for (int q = 0; q < 4; ++q) red[ty][4 * tx + q] = acc[q];
      __syncthreads();
      if (ty == 0) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int col = 4 * tx + q;
          const double v = ((red[0][col] + red[1][col]) + red[2][col]) + red[3][col];
          if (colok) partial[((int64_t)(k - 1) * nrt + blockIdx.y) * d + j0 + q] = v;
        }
      }
      __syncthreads();
    }
  }
#pragma unroll
  for (int r = 0; r < RPT; ++r) {
    const int64_t t = t0 + ty + 4 * r;
    if (colok && t < T) {
      const uint32_t lo = cnt[r][0] | (cnt[r][1] << 16);
      const uint32_t hi = cnt[r][2] | (cnt[r][3] << 16);
      *(uint2*)(counts + t * d + j0) = make_uint2(lo, hi);
    }
  }
}

// ------------------------------------------------------------------------------------
// launchers
// ------------------------------------------------------------------------------------
bs_status launch_store(const void* x, bs_dtype xt, int64_t n, int fmt, int mode, uint64_t seed, uint32_t trial,
                       uint32_t use, const float* scale_in, uint8_t* codes, float* scale_out, bs_diag* diag,
                       hipStream_t st, bool amax_done) {
  const F8 f = f8_format(fmt);
  if (!amax_done) {
    init_diag_kernel<<<1, 64, 0, st>>>(diag);
    if (n > 0 && !scale_in) {
      const int64_t want = (n + 255) / 256;
      const int blocks = (int)(want < 2048 ? want : 2048);
      if (xt == BS_F32)
        amax_kernel<float><<<blocks, 256, 0, st>>>((const float*)x, n, (uint32_t*)&diag->amax);
      else
        amax_kernel<u16><<<blocks, 256, 0, st>>>((const u16*)x, n, (uint32_t*)&diag->amax);
    }
  }
  finalize_scale_kernel<<<1, 64, 0, st>>>(diag, scale_in, scale_out, f.fmax);
  if (n > 0) {
    const int64_t groups = (n + 3) / 4;
    const unsigned blocks = (unsigned)((groups + 255) / 256);
    ProfScope prof("quantize", st);
#define QK(T, M) quantize_kernel<T, M><<<blocks, 256, 0, st>>>((const T*)x, n, f, diag, codes, seed, trial, use)
    if (xt == BS_F32) {
      if (mode == BS_SR) QK(float, BS_SR); else QK(float, BS_RNE);
    } else {
      if (mode == BS_SR) QK(u16, BS_SR); else QK(u16, BS_RNE);
    }
#undef QK
  }
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status launch_fresh_count(const float* u, int64_t T, int64_t d, int fmt, const float* scale, uint64_t seed,
                             uint32_t use, int K, u16* counts, const float* w, double* partial, hipStream_t st) {
  if (T == 0) return BS_OK;
  const F8 f = f8_format(fmt);
  dim3 grid((unsigned)((d + 255) / 256), (unsigned)((T + 31) / 32));
  ProfScope prof(partial ? "fresh_count_se" : "fresh_count", st);
  if (partial)
    fresh_count_kernel<true><<<grid, 256, 0, st>>>(u, T, d, f, scale, seed, use, K, counts, w, partial);
  else
    fresh_count_kernel<false><<<grid, 256, 0, st>>>(u, T, d, f, scale, seed, use, K, counts, nullptr, nullptr);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

}  // namespace bsp
