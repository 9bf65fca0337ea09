// FP8 store kernels: amax, scale, quantize (RNE / stochastic), and the K-trial
// stochastic-rounding counter of a store's new roundings.
#include <type_traits>

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
// finite value, so one atomicMax also detects non-finite input. Each thread streams
// 16-byte vectors (8 bf16 or 4 fp32) in a grid-stride loop; the scalar tail is done once.
template <typename T>
__device__ __forceinline__ uint32_t vec_absmax(uint4 v);
template <>
__device__ __forceinline__ uint32_t vec_absmax<float>(uint4 v) {
  const uint32_t a = v.x & 0x7FFFFFFFu, b = v.y & 0x7FFFFFFFu, c = v.z & 0x7FFFFFFFu, d = v.w & 0x7FFFFFFFu;
  return max(max(a, b), max(c, d));
}
template <>
__device__ __forceinline__ uint32_t vec_absmax<u16>(uint4 v) {
  // bf16 -> fp32 bit patterns are the bf16 bits shifted by 16, order preserved
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t lo = (w[i] << 16) & 0x7FFFFFFFu, hi = w[i] & 0x7FFF0000u;
    m = max(m, max(lo, hi));
  }
  return m;
}

template <typename T>
__global__ __launch_bounds__(256) void amax_kernel(const T* __restrict__ x, int64_t n,
                                                   uint32_t* __restrict__ amax_bits) {
  constexpr int PER = 16 / sizeof(T);
  uint32_t m = 0;
  const int64_t nvec = ((uintptr_t)x & 15) ? 0 : n / PER;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const uint4* xv = (const uint4*)x;
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  // Each block streams its own contiguous range of vectors, eight 16-byte non-temporal loads in
  // flight per thread (read once, not kept in cache); the remainder goes grid-strided.
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  constexpr int U = 8;
  {
    const int64_t per = ((nvec / gridDim.x) / (U * blockDim.x)) * (U * blockDim.x);
    const int64_t b0 = (int64_t)blockIdx.x * per;
    for (int64_t j = 0; j < per; j += U * blockDim.x) {
      uint4 v[U];
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const u32x4 t = __builtin_nontemporal_load((const u32x4*)(xv + b0 + j + k * blockDim.x + threadIdx.x));
        v[k] = make_uint4(t.x, t.y, t.z, t.w);
      }
#pragma unroll
      for (int k = 0; k < U; ++k) m = max(m, vec_absmax<T>(v[k]));
    }
    i = per * gridDim.x + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  }
  for (; i + (U - 1) * stride < nvec; i += U * stride) {
    uint4 v[U];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const u32x4 t = __builtin_nontemporal_load((const u32x4*)(xv + i + k * stride));
      v[k] = make_uint4(t.x, t.y, t.z, t.w);
    }
#pragma unroll
    for (int k = 0; k < U; ++k) m = max(m, vec_absmax<T>(v[k]));
  }
  for (; i < nvec; i += stride) m = max(m, vec_absmax<T>(xv[i]));
  for (int64_t j = nvec * PER + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n; j += stride)
    m = max(m, __float_as_uint(fabsf(load_f32(x, j))));
  m = wave_max_u32(m);
  __shared__ uint32_t red[4];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (lane == 0) red[w] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t b = red[0];
    for (int k = 1; k < (int)(blockDim.x >> 6); ++k) b = b > red[k] ? b : red[k];
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

// gfx950's conversion instructions to the OCP formats ("fp8" = E4M3, "bf8" = E5M2), on values
// clamped to +-FMAX first. The packed conversion rounds to nearest even: the codec above, bit for
// bit (negative values that round to zero keep the sign bit). The stochastic one rounds up iff
// R + F >= 2^32 with its 32-bit operand R for every normal FP8 magnitude (there F has at most 21
// significant bits); below the smallest normal magnitude it does not resolve F to all 32 bits
// (at R + F = 2^32 exactly it stays down), so nonzero values there take the integer path.
template <int FMT, bool HI>
__device__ __forceinline__ uint32_t cvt_rne2(float a, float b, uint32_t old) {
  return FMT == BS_E5M2 ? (uint32_t)__builtin_amdgcn_cvt_pk_bf8_f32(a, b, (int)old, HI)
                        : (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a, b, (int)old, HI);
}
template <int FMT, int BYTE>
__device__ __forceinline__ uint32_t cvt_sr1(float a, uint32_t R, uint32_t old) {
  return FMT == BS_E5M2 ? (uint32_t)__builtin_amdgcn_cvt_sr_bf8_f32(a, (int)R, (int)old, BYTE)
                        : (uint32_t)__builtin_amdgcn_cvt_sr_fp8_f32(a, (int)R, (int)old, BYTE);
}

// y = fl32(x / s) clamped to [-FMAX, FMAX] (sign of zero kept); counts the wave's clamped
// values (a ballot and a scalar popcount: the count is wave-uniform)
__device__ __forceinline__ float scaled_clamped(float x, double rs, float fmax, uint32_t& nsat) {
  const float y = div_scale(x, rs);
  nsat += (uint32_t)__popcll(__ballot(fabsf(y) > fmax));
  return __builtin_amdgcn_fmed3f(y, -fmax, fmax);
}

// stochastic rounding of one clamped value by the integer codec
__device__ __forceinline__ uint32_t sr_code(float y, uint32_t R, F8 f) {
  const Bracket b = f8_bracket(fabsf(y), f);
  return (b.base + b.mi + sr_up(b.F, R)) | (signbit(y) ? 0x80u : 0u);
}

// Four codes packed into a word from four scaled values (R: the Philox words, SR only).
template <int FMT, int MODE>
__device__ __forceinline__ uint32_t codes4(const float* y, const uint32_t* R) {
  if (MODE == BS_SR) {
    uint32_t w = cvt_sr1<FMT, 0>(y[0], R[0], 0u);
    w = cvt_sr1<FMT, 1>(y[1], R[1], w);
    w = cvt_sr1<FMT, 2>(y[2], R[2], w);
    w = cvt_sr1<FMT, 3>(y[3], R[3], w);
    const F8 f = f8_format(FMT);
    const float min_normal = __uint_as_float((uint32_t)(128 - f.bias) << 23);
    bool sub = false;
#pragma unroll
    for (int q = 0; q < 4; ++q) sub |= fabsf(y[q]) < min_normal && y[q] != 0.0f;
    if (sub) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (fabsf(y[q]) < min_normal && y[q] != 0.0f)
          w = (w & ~(0xFFu << (8 * q))) | (sr_code(y[q], R[q], f) << (8 * q));
    }
    return w;
  }
  return cvt_rne2<FMT, true>(y[2], y[3], cvt_rne2<FMT, false>(y[0], y[1], 0u));
}

// Groups of eight consecutive elements (two Philox groups), grid-stride: one 16- or 32-byte load
// and an 8-byte store of the codes per group. The last group of a ragged tensor takes the
// element-wise path. A thread takes several groups, so that the per-wave set-up is paid once
// per several groups.
template <typename T, int FMT, int MODE>
__global__ __launch_bounds__(256) void quantize_kernel(const T* __restrict__ x, int64_t n, float fmax,
                                                       bs_diag* __restrict__ diag, uint8_t* __restrict__ codes,
                                                       uint64_t seed, uint32_t trial, uint32_t use) {
  if (diag->nonfinite) return;
  const double rs = 1.0 / (double)diag->scale;
  const int64_t ngroups = (n + 7) / 8, stride = (int64_t)gridDim.x * blockDim.x;
  uint32_t nsat = 0;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < ngroups; t += stride) {
    const int64_t e0 = t * 8;
    float xv[8];
    const int cnt = (int)((n - e0) < 8 ? (n - e0) : 8);
    const bool vec = cnt == 8 && (((uintptr_t)(x + e0)) & 15) == 0 && (((uintptr_t)(codes + e0)) & 7) == 0;
    if (vec) {
      if (sizeof(T) == 2) {
        const uint4 v = *(const uint4*)(x + e0);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          xv[2 * i] = __uint_as_float(w[i] << 16);
          xv[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
        }
      } else {
        const float4 a = *(const float4*)(x + e0), b = *(const float4*)(x + e0 + 4);
        xv[0] = a.x; xv[1] = a.y; xv[2] = a.z; xv[3] = a.w;
        xv[4] = b.x; xv[5] = b.y; xv[6] = b.z; xv[7] = b.w;
      }
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) xv[q] = q < cnt ? load_f32(x, e0 + q) : 0.0f;
    }
    uint32_t R[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (MODE == BS_SR) {
      const Philox4 p0 = philox_group(seed, (uint64_t)(2 * t), trial, use);
      const Philox4 p1 = philox_group(seed, (uint64_t)(2 * t + 1), trial, use);
      R[0] = p0.w0; R[1] = p0.w1; R[2] = p0.w2; R[3] = p0.w3;
      R[4] = p1.w0; R[5] = p1.w1; R[6] = p1.w2; R[7] = p1.w3;
    }
    float y[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) y[q] = scaled_clamped(xv[q], rs, fmax, nsat);  // padding zeros never clamp
    const uint32_t lo = codes4<FMT, MODE>(y, R), hi = codes4<FMT, MODE>(y + 4, R + 4);
    if (vec) {
      *(uint2*)(codes + e0) = make_uint2(lo, hi);
    } else {
      for (int q = 0; q < cnt; ++q) codes[e0 + q] = (uint8_t)((q < 4 ? lo >> (8 * q) : hi >> (8 * (q - 4))));
    }
  }
  // nsat is the wave's count here: lane 0 has the smallest group index of its wave, so it takes
  // part in every ballot of the wave
  if ((threadIdx.x & 63) == 0 && nsat) atomicAdd(&diag->n_saturated, nsat);
}

// K-trial counter of new roundings of a [T, d] store y = fl32(x / s) (d % 4 == 0).
// counts[t, j] = number of trials k in 1..K whose rounding of element t*d + j goes up.
// Block: 256 threads = 64 column groups (4 columns each) x 4 row lanes, 8 rows per thread,
// so one block covers 32 rows x 256 columns. The row lane is the wave, except for FC_COLSUM,
// where a wave holds 16 column groups x 4 row lanes so that the column sums reduce inside the
// wave (cross-lane adds in a fixed order, no barrier). With c = sign(y) step (t, j) w(t, j):
//   FC_COLSUM: colsum[k-1][rt][j] = sum over the block's 32 rows of up_k c (w = w1), fp32
//   FC_BLOCKSUM: partial[k-1][i][b] = sum over the block's elements of up_k c_i (w1, w2), fp64
// FC_BLOCKSUM reduces through LDS four trials at a time, in a fixed order. The column sums feed only a
// sample variance over trials: they hold no trial-independent term (an element whose
// rounding never goes up adds nothing), so fp32 rounding of a 32-row sum perturbs each trial
// by a few ulps of values of the size of the trial-to-trial spread, far below the 1e-5 of the
// statistic, and the sums over row blocks are taken in fp64.
template <typename X, int MODE>
__device__ __forceinline__ void fresh_count_body(const FreshArgs<X>& a) {
  constexpr int RT = 32, RPT = 8, TB = MODE == FC_COLSUM ? 1 : 4;
  const int lane = threadIdx.x & 63;
  const int tx = MODE == FC_COLSUM ? (threadIdx.x >> 6) * 16 + (lane & 15) : lane;
  const int ty = MODE == FC_COLSUM ? lane >> 4 : threadIdx.x >> 6;
  const int64_t j0 = (int64_t)blockIdx.x * 256 + 4 * tx;
  const int64_t t0 = (int64_t)blockIdx.y * RT;
  const bool colok = j0 < a.d;
  const double rs = 1.0 / (double)*a.scale;
  uint32_t F[RPT][4], cnt[RPT][4];
  float c1[RPT][4], c2[RPT][4];
#pragma unroll
  for (int r = 0; r < RPT; ++r) {
    const int64_t t = t0 + ty + 4 * r;
    const bool ok = colok && t < a.T;
    float xv[4] = {0.f, 0.f, 0.f, 0.f}, w1v[4] = {0.f, 0.f, 0.f, 0.f}, w2v[4] = {0.f, 0.f, 0.f, 0.f};
    if (ok) {
      const int64_t e = t * a.d + j0;
#pragma unroll
      for (int q = 0; q < 4; ++q) xv[q] = load_f32(a.x, e + q);
      if (MODE != FC_COUNT) {
        const float4 v = *(const float4*)(a.w1 + e);
        w1v[0] = v.x; w1v[1] = v.y; w1v[2] = v.z; w1v[3] = v.w;
      }
      if (MODE == FC_BLOCKSUM && a.w2) {
        const float4 v = *(const float4*)(a.w2 + e);
        w2v[0] = v.x; w2v[1] = v.y; w2v[2] = v.z; w2v[3] = v.w;
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float y = div_scale(xv[q], rs);
      const Bracket b = f8_bracket(fminf(fabsf(y), a.f.fmax), a.f);
      F[r][q] = ok ? b.F : 0u;
      const float sc = (signbit(y) ? -1.0f : 1.0f) * f8_step(b);
      c1[r][q] = sc * w1v[q];
      c2[r][q] = sc * w2v[q];
      cnt[r][q] = 0;
      // opaque from here on: keeps the row-validity test out of the trial loop
      asm volatile("" : "+v"(F[r][q]), "+v"(c1[r][q]));
    }
  }
  using Acc = typename std::conditional<MODE == FC_COLSUM, float, double>::type;
  __shared__ double red[MODE == FC_BLOCKSUM ? TB : 1][2 * 4];
  const int64_t nrt = gridDim.y;
  const int64_t nblk = (int64_t)gridDim.x * gridDim.y, bid = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;
  for (int k0 = 1; k0 <= a.K; k0 += TB) {
    Acc acc[TB][4];
#pragma unroll
    for (int i = 0; i < TB; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[i][q] = 0;
#pragma unroll
    for (int i = 0; i < TB; ++i) {
      const int k = k0 + i;
      if (k > a.K) break;
#pragma unroll
      for (int r = 0; r < RPT; ++r) {
        const int64_t t = t0 + ty + 4 * r;
        const uint64_t g = (uint64_t)((t * a.d + j0) >> 2);
        const Philox4 p = philox_group(a.seed, g, (uint32_t)(k - 1 + a.trial0), a.use);
        const uint32_t R[4] = {p.w0, p.w1, p.w2, p.w3};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t up = sr_up(F[r][q], R[q]);
          cnt[r][q] += up;
          if (MODE == FC_COLSUM) acc[i][q] += up ? c1[r][q] : 0.0f;
          if (MODE == FC_BLOCKSUM) {
            acc[i][0] += up ? (double)c1[r][q] : 0.0;
            acc[i][1] += up ? (double)c2[r][q] : 0.0;
          }
        }
        // column sums: at most four Philox groups in flight (register budget of three waves)
        if (MODE == FC_COLSUM && (r & 3) == 3) __builtin_amdgcn_sched_barrier(0);
      }
    }
    if (MODE == FC_COLSUM) {
      // sum over the 4 row lanes (lane bits 4 and 5): (l + l^16) + (l^32 + l^48)
#pragma unroll
      for (int i = 0; i < TB; ++i) {
        float v[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          v[q] = (float)acc[i][q];
          v[q] += __shfl_xor(v[q], 16, 64);
          v[q] += __shfl_xor(v[q], 32, 64);
        }
        const int k = k0 + i;
        if (ty == 0 && colok && k <= a.K)
          *(float4*)(a.colsum + ((int64_t)(k - 1) * nrt + blockIdx.y) * a.d + j0) = make_float4(v[0], v[1], v[2], v[3]);
      }
    }
    if (MODE == FC_BLOCKSUM) {
      const int wv = threadIdx.x >> 6;
#pragma unroll
      for (int i = 0; i < TB; ++i) {
        const double v1 = wave_sum_f64(acc[i][0]);
        const double v2 = wave_sum_f64(acc[i][1]);
        if (lane == 0) {
          red[i][2 * wv] = v1;
          red[i][2 * wv + 1] = v2;
        }
      }
      __syncthreads();
      if (threadIdx.x < 2 * TB) {
        const int i = threadIdx.x >> 1, u = threadIdx.x & 1;
        const int k = k0 + i;
        const double v = ((red[i][u] + red[i][2 + u]) + red[i][4 + u]) + red[i][6 + u];
        if (k <= a.K) a.partial[((int64_t)(k - 1) * 2 + u) * nblk + bid] = v;
      }
      __syncthreads();
    }
  }
  if (a.counts) {
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
      const int64_t t = t0 + ty + 4 * r;
      if (colok && t < a.T) {
        const uint32_t lo = cnt[r][0] | (cnt[r][1] << 16);
        const uint32_t hi = cnt[r][2] | (cnt[r][3] << 16);
        *(uint2*)(a.counts + t * a.d + j0) = make_uint2(lo, hi);
      }
    }
  }
}

// The column-sum variant holds the per-element weights too; it is held to 168 registers so that
// three waves share each SIMD (the Philox latency needs them).
template <typename X, int MODE>
__global__ __launch_bounds__(256) void fresh_count_kernel(FreshArgs<X> a) {
  fresh_count_body<X, MODE>(a);
}
template <typename X>
__global__ __launch_bounds__(256) void fresh_colsum_kernel(FreshArgs<X> a) {
  fresh_count_body<X, FC_COLSUM>(a);
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
    // amax runs with a caller's scale too: it flags NaN / infinity (no codes then) and reports the
    // tensor's amax to a delayed-scaling caller's history; the caller's scale replaces only s
    if (n > 0) {
      // four blocks per CU, each streaming a contiguous range with eight 16-byte loads in flight
      // per thread; the per-block atomics stay few (same-address atomics serialize)
      const int64_t want = (n / (16 / (xt == BS_F32 ? 4 : 2)) + 255) / 256 + 1;
      const int blocks = (int)(want < 1024 ? want : 1024);
      ProfScope prof("amax", st);
      if (xt == BS_F32)
        amax_kernel<float><<<blocks, 256, 0, st>>>((const float*)x, n, (uint32_t*)&diag->amax);
      else
        amax_kernel<u16><<<blocks, 256, 0, st>>>((const u16*)x, n, (uint32_t*)&diag->amax);
    }
  }
  finalize_scale_kernel<<<1, 64, 0, st>>>(diag, scale_in, scale_out, f.fmax);
  if (n > 0 && codes) {  // codes == nullptr: the scale only
    // up to 8192 blocks (32 waves per CU), each thread then taking several groups of eight
    const int64_t threads = (n + 7) / 8;
    const unsigned blocks = (unsigned)std::min<int64_t>((threads + 255) / 256, 8192);
    ProfScope prof("quantize", st);
#define QK(T, FM, M) \
  quantize_kernel<T, FM, M><<<blocks, 256, 0, st>>>((const T*)x, n, f.fmax, diag, codes, seed, trial, use)
#define QKF(T)                                              \
  if (fmt == BS_E5M2) {                                     \
    if (mode == BS_SR) QK(T, BS_E5M2, BS_SR); else QK(T, BS_E5M2, BS_RNE); \
  } else {                                                  \
    if (mode == BS_SR) QK(T, BS_E4M3, BS_SR); else QK(T, BS_E4M3, BS_RNE); \
  }
    if (xt == BS_F32) {
      QKF(float);
    } else {
      QKF(u16);
    }
#undef QKF
#undef QK
  }
  BS_CHECK_LAUNCH();
  return BS_OK;
}

template <typename X>
bs_status launch_fresh_count_t(const FreshArgs<X>& a, int mode, hipStream_t st) {
  if (a.T == 0) return BS_OK;
  dim3 grid((unsigned)((a.d + 255) / 256), (unsigned)((a.T + 31) / 32));
  ProfScope prof(mode == FC_COUNT ? "fresh_count" : (mode == FC_COLSUM ? "fresh_count_se" : "fresh_count_kappa"), st);
  if (mode == FC_COUNT)
    fresh_count_kernel<X, FC_COUNT><<<grid, 256, 0, st>>>(a);
  else if (mode == FC_COLSUM)
    fresh_colsum_kernel<X><<<grid, 256, 0, st>>>(a);
  else
    fresh_count_kernel<X, FC_BLOCKSUM><<<grid, 256, 0, st>>>(a);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
template bs_status launch_fresh_count_t<float>(const FreshArgs<float>&, int, hipStream_t);
template bs_status launch_fresh_count_t<u16>(const FreshArgs<u16>&, int, hipStream_t);

bs_status launch_fresh_count(const float* u, int64_t T, int64_t d, int fmt, const float* scale, uint64_t seed,
                             uint32_t use, int K, u16* counts, const float* w, float* colsum, hipStream_t st) {
  FreshArgs<float> a{u, T, d, f8_format(fmt), scale, seed, use, K, counts, w, nullptr, nullptr, colsum};
  return launch_fresh_count_t(a, colsum ? FC_COLSUM : FC_COUNT, st);
}

bs_status launch_amax_f32(const float* x, int64_t n, uint32_t* out, hipStream_t st) {
  if (n < 0 || (n > 0 && (!x || !out))) return BS_EINVAL;
  if (n == 0) return BS_OK;
  const int64_t want = (n / 4 + 255) / 256 + 1;
  amax_kernel<float><<<(int)(want < 1024 ? want : 1024), 256, 0, st>>>(x, n, out);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
bs_status launch_amax_bf16(const u16* x, int64_t n, uint32_t* out, hipStream_t st) {
  if (n < 0 || (n > 0 && (!x || !out))) return BS_EINVAL;
  if (n == 0) return BS_OK;
  const int64_t want = (n / 8 + 255) / 256 + 1;
  amax_kernel<u16><<<(int)(want < 1024 ? want : 1024), 256, 0, st>>>(x, n, out);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

}  // namespace bsp
