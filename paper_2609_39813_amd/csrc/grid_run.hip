// The paper's own normalization store (App. D.4): RMSNorm -> per-token b-bit uniform grid with
// stochastic rounding -> Linear, and the eight policies of its table (gain use first; the weight
// use may also read u_q + (u_f - u)). One new rounding u_f per trial feeds both uses.
//
// Per token t: s_t = fl32(max_j |u_tj| / M), M = 2^(b-1) - 1; y = fl32(u / s_t); a = min(|y|, M)
// (clamps counted); lo = floor(a), F = floor((a - lo) 2^32); the code rounds up iff R + F >= 2^32;
// u_q = fl32(q s_t). Every bias is a contraction (weight use) or an fp64 column sum (gain use) of
// a residual: e_U = u - u_q, e_N = mean_k u_f,k - u_q, e_e = mean_k u_f,k - u, where the mean
// over trials of the grid values is ((K - n) v_lo + n v_hi) / K from the element's up-count n.
#include <algorithm>

#include "bsp_kernels.h"
#include "k_norm.h"

#define BS_TRY(x)               \
  do {                          \
    const bs_status _s = (x);   \
    if (_s != BS_OK) return _s; \
  } while (0)

namespace bsp {

namespace {

struct GridBracket {
  float lo;     // floor(|y|), |y| clamped to M
  uint32_t F;   // floor(frac 2^32)
  bool neg;
  bool sat;
};

__device__ __forceinline__ GridBracket grid_bracket(float u, float s, float M) {
  GridBracket b;
  const float y = u / s;  // IEEE division (correctly rounded)
  const float a = fabsf(y);
  b.sat = a > M;
  const float ac = fminf(a, M);
  b.lo = floorf(ac);
  b.F = (uint32_t)((ac - b.lo) * 4294967296.0f);  // exact: ac - lo has at most 24 bits, < 1
  b.neg = signbit(y);
  return b;
}

// fl32(q s) of the code sign * m
__device__ __forceinline__ float grid_value(float m, bool neg, float s) { return (neg ? -m : m) * s; }

// one wave per token: the step, the forward's codes (trial 0), u_q and e_U = u - u_q
__global__ __launch_bounds__(256) void grid_store_kernel(const float* __restrict__ u, int64_t T, int64_t d, int bits,
                                                         uint64_t seed, uint32_t use, int8_t* __restrict__ codes,
                                                         float* __restrict__ step, float* __restrict__ uq,
                                                         float* __restrict__ eU, bs_diag* __restrict__ diag) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const float M = (float)((1 << (bits - 1)) - 1);
  const float* ur = u + t * d;
  float m = 0.0f;
  for (int64_t j = 4 * lane; j < d; j += 256) {
    const float4 v = *(const float4*)(ur + j);
    m = fmaxf(m, fmaxf(fmaxf(fabsf(v.x), fabsf(v.y)), fmaxf(fabsf(v.z), fabsf(v.w))));
  }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
  const float s = m > 0.0f ? m / M : 1.0f;
  if (lane == 0) step[t] = s;
  uint32_t nsat = 0;
  for (int64_t j = 4 * lane; j < d; j += 256) {
    const float4 v = *(const float4*)(ur + j);
    const float uv[4] = {v.x, v.y, v.z, v.w};
    const Philox4 p = philox_group(seed, (uint64_t)(t * d + j) >> 2, 0u, use);
    const uint32_t R[4] = {p.w0, p.w1, p.w2, p.w3};
    float qv[4], ev[4];
    uint32_t cw = 0;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const GridBracket b = grid_bracket(uv[r], s, M);
      nsat += b.sat ? 1u : 0u;
      const float mag = b.lo + (float)sr_up(b.F, R[r]);
      qv[r] = grid_value(mag, b.neg, s);
      ev[r] = (float)((double)uv[r] - (double)qv[r]);
      const int q = b.neg ? -(int)mag : (int)mag;
      cw |= ((uint32_t)(uint8_t)(int8_t)q) << (8 * r);
    }
    *(uint32_t*)(codes + t * d + j) = cw;
    *(float4*)(uq + t * d + j) = make_float4(qv[0], qv[1], qv[2], qv[3]);
    *(float4*)(eU + t * d + j) = make_float4(ev[0], ev[1], ev[2], ev[3]);
  }
  nsat = wave_sum_u32(nsat);
  if (lane == 0 && nsat) atomicAdd(&diag->n_saturated, nsat);
}

// one thread per 4 elements: up-counts of the new rounding over K trials, then e_N and e_e
__global__ __launch_bounds__(256) void grid_fresh_kernel(const float* __restrict__ u, const float* __restrict__ uq,
                                                         const float* __restrict__ step, int64_t T, int64_t d,
                                                         int bits, uint64_t seed, uint32_t use, int K,
                                                         float* __restrict__ eN, float* __restrict__ eE) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g * 4 >= T * d) return;
  const int64_t e0 = g * 4, t = e0 / d;
  const float M = (float)((1 << (bits - 1)) - 1);
  const float s = step[t];
  const float4 v = *(const float4*)(u + e0);
  const float4 q4 = *(const float4*)(uq + e0);
  const float uv[4] = {v.x, v.y, v.z, v.w}, qv[4] = {q4.x, q4.y, q4.z, q4.w};
  GridBracket b[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) b[r] = grid_bracket(uv[r], s, M);
  uint32_t n[4] = {0u, 0u, 0u, 0u};
  for (int k = 1; k <= K; ++k) {
    const Philox4 p = philox_group(seed, (uint64_t)g, (uint32_t)k, use);
    n[0] += sr_up(b[0].F, p.w0);
    n[1] += sr_up(b[1].F, p.w1);
    n[2] += sr_up(b[2].F, p.w2);
    n[3] += sr_up(b[3].F, p.w3);
  }
  float oN[4], oE[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const double vlo = grid_value(b[r].lo, b[r].neg, s), vhi = grid_value(b[r].lo + 1.0f, b[r].neg, s);
    const double mf = ((double)(K - (int)n[r]) * vlo + (double)n[r] * vhi) / (double)K;
    oN[r] = (float)(mf - (double)qv[r]);
    oE[r] = (float)(mf - (double)uv[r]);
  }
  *(float4*)(eN + e0) = make_float4(oN[0], oN[1], oN[2], oN[3]);
  *(float4*)(eE + e0) = make_float4(oE[0], oE[1], oE[2], oE[3]);
}

// gain use, fp64 column partials over token chunks of 256: [3][nchunk][d]
//   ref  sum z du;  R  sum (u/gain - z - eU/gain) du;  N  sum (u/gain - z + eE/gain) du
// rows per chunk of the gain use's column partial sums: T / 32 chunks (grid x) x d / 64 one-wave
// blocks (grid y)
constexpr int GRID_GAIN_RT = 32;

template <typename XT>
__global__ __launch_bounds__(64) void grid_gain_kernel(const XT* __restrict__ X, const float* __restrict__ rstd,
                                                       const float* __restrict__ gain, const float* __restrict__ u,
                                                       const float* __restrict__ du, const float* __restrict__ eU,
                                                       const float* __restrict__ eE, int64_t T, int64_t d,
                                                       double* __restrict__ part) {
#pragma clang fp contract(off)
  const int64_t j = (int64_t)blockIdx.y * 64 + threadIdx.x;
  const int64_t c = blockIdx.x, nch = gridDim.x;
  if (j >= d) return;
  const double g = gain[j];
  double a0 = 0.0, a1 = 0.0, a2 = 0.0;
  const int64_t t1 = min(T, (c + 1) * GRID_GAIN_RT);
  for (int64_t t = c * GRID_GAIN_RT; t < t1; ++t) {
    const int64_t e = t * d + j;
    const double z = (double)(load_f32(X, e) * rstd[t]);
    const double dd = du[e];
    const double base = (double)u[e] / g - z;
    a0 += z * dd;
    if (eU) a1 += (base - (double)eU[e] / g) * dd;
    if (eE) a2 += (base + (double)eE[e] / g) * dd;
  }
  part[(0 * nch + c) * d + j] = a0;
  part[(1 * nch + c) * d + j] = a1;
  part[(2 * nch + c) * d + j] = a2;
}

struct GridWs {
  float *u, *rstd, *du, *uq, *eU, *eN, *eE, *bias_rg, *bias_ng, *bias_w[3];  // weight biases: U, N, R+e
  u16 *dyT[3], *aT[3], *uq_rows[3], *wT[3], *dy_rows[3], *w_rows[3];
  double* gpart;
  float* gemm_part;
  int64_t gemm_part_cap;
};

GridWs carve_grid(Carver& c, int64_t T, int64_t d, int64_t n, bs_dtype wt, bs_dtype gt, bool want_y) {
  GridWs w{};
  const int64_t Tp = round_up(T > 0 ? T : 1, 64);
  const int nt = gt == BS_F32 ? 3 : 1, ntw = wt == BS_F32 ? 3 : 1;
  for (float** p : {&w.u, &w.du, &w.uq, &w.eU, &w.eN, &w.eE}) *p = c.take<float>(T * d);
  w.rstd = c.take<float>(T > 0 ? T : 1);
  for (int i = 0; i < nt; ++i) w.dyT[i] = c.take<u16>(n * Tp);
  for (int i = 0; i < 3; ++i) w.aT[i] = c.take<u16>(d * Tp);
  if (gt == BS_F32)
    for (int i = 0; i < 3; ++i) w.dy_rows[i] = c.take<u16>(T * n);
  if (wt == BS_F32)
    for (int i = 0; i < 3; ++i) w.w_rows[i] = c.take<u16>(d * n);
  if (want_y) {
    for (int i = 0; i < 3; ++i) w.uq_rows[i] = c.take<u16>(T * d);
    for (int i = 0; i < ntw; ++i) w.wT[i] = c.take<u16>(n * d);
  }
  w.bias_rg = c.take<float>(d);
  w.bias_ng = c.take<float>(d);
  for (int i = 0; i < 3; ++i) w.bias_w[i] = c.take<float>(d * n);
  w.gpart = c.take<double>(3 * ((T + GRID_GAIN_RT - 1) / GRID_GAIN_RT + 1) * d);
  w.gemm_part_cap = 4 * d * std::max<int64_t>(std::max<int64_t>(T, n), 64);
  w.gemm_part = c.take<float>(w.gemm_part_cap);
  return w;
}

}  // namespace

size_t grid_ws_size(int64_t T, int64_t d, int64_t n) {
  if (T < 0 || d < 8 || n < 8) return 0;
  Carver c;
  carve_grid(c, T, d, n, BS_F32, BS_F32, true);
  return c.used();
}

struct GridIO {
  const void *X, *W, *dY;
  const float* gain;
  bs_dtype dt;
  int64_t T, d, n;
  float eps;
  int bits;
  const bs_grid_policy* pol;
  int n_pol, K;
  uint64_t seed;
  uint32_t store_id;
  float* Y;
  int8_t* codes;
  float* step;
  float *dgain_ref, *dW_ref, *dX_ref;
  bs_est dgain, dW;
  bs_diag* diag;
};

bs_status grid_run(const GridIO& io, void* ws, size_t ws_bytes, hipStream_t st) {
  const int64_t T = io.T, d = io.d, n = io.n;
  if (!io.X || !io.W || !io.dY || !io.gain || !io.codes || !io.step || !io.dgain_ref || !io.dW_ref || !io.dX_ref ||
      !io.pol || !io.diag)
    return BS_EINVAL;
  if (io.dt != BS_F32 && io.dt != BS_BF16) return BS_EDTYPE;
  if (io.bits < 2 || io.bits > 8 || io.K < 1 || io.K > 4096 || io.n_pol < 1 || io.n_pol > 16 || !(io.eps >= 0.0f))
    return BS_EINVAL;
  if (T < 1 || d < 8 || d > 8192 || (d & 7) || n < 8 || (n & 7) || T > 65535LL * 256 || n > 0x7FFFFFFF)
    return BS_ESHAPE;
  if (io.dgain.se || io.dW.se) return BS_EUNSUPPORTED;
  for (int i = 0; i < io.n_pol; ++i) {
    if (io.pol[i].gain_use < BS_READ_U || io.pol[i].gain_use > BS_READ_N) return BS_EINVAL;
    if (io.pol[i].weight_use < BS_WREAD_U || io.pol[i].weight_use > BS_WREAD_R_EPS) return BS_EINVAL;
  }
  const bs_dtype wt = io.dt, gt = io.dt, xt = io.dt;
  Carver probe;
  carve_grid(probe, T, d, n, wt, gt, io.Y != nullptr);
  if (!ws || ((uintptr_t)ws & 255) || ws_bytes < probe.used()) return BS_EWORKSPACE;
  Carver c(ws, ws_bytes);
  GridWs w = carve_grid(c, T, d, n, wt, gt, io.Y != nullptr);
  const int64_t Tp = round_up(T, 64);
  const int nt = gt == BS_F32 ? 3 : 1, ntw = wt == BS_F32 ? 3 : 1;
  const uint32_t base = io.store_id * 256u;

  // forward: RMSNorm (fixed fp32 order), the grid store
  BS_TRY(launch_init_diag(io.diag, st));
  BS_TRY(launch_rmsnorm_fwd(io.X, xt, io.gain, T, d, io.eps, w.u, w.rstd, io.diag, st));
  {
    ProfScope prof("grid_store", st);
    grid_store_kernel<<<(unsigned)((T + 3) / 4), 256, 0, st>>>(w.u, T, d, io.bits, io.seed, base, io.codes, io.step,
                                                               w.uq, w.eU, io.diag);
    BS_CHECK_LAUNCH();
  }
  // Y = u_q W (three bf16 terms of u_q)
  if (io.Y) {
    BS_TRY(launch_planes(w.uq, BS_F32, T, d, d, false, w.uq_rows, 3, d, 1.0f, st));
    BS_TRY(launch_planes(io.W, wt, d, n, n, true, w.wT, ntw, d, 1.0f, st));
    GemmArgs g{};
    g.M = (int)T;
    g.N = (int)n;
    g.K = (int)d;
    g.lda = d;
    g.ldb = d;
    g.ldc = n;
    g.alpha = 1.0f;
    g.C = io.Y;
    gemm_add_products(g, w.uq_rows, 3, w.wT, ntw);
    BS_TRY(launch_gemm(g, st));
  }
  // du = dY W^T
  {
    GemmArgs g{};
    g.M = (int)T;
    g.N = (int)d;
    g.K = (int)n;
    g.lda = n;
    g.ldb = n;
    g.ldc = d;
    g.alpha = 1.0f;
    g.C = w.du;
    g.part = w.gemm_part;
    g.part_cap = w.gemm_part_cap;
    u16* A0 = (u16*)io.dY;
    u16* B0 = (u16*)io.W;
    u16* const* Aops = &A0;
    u16* const* Bops = &B0;
    if (gt == BS_F32) {
      BS_TRY(launch_planes(io.dY, gt, T, n, n, false, w.dy_rows, 3, n, 1.0f, st));
      Aops = w.dy_rows;
    }
    if (wt == BS_F32) {
      BS_TRY(launch_planes(io.W, wt, d, n, n, false, w.w_rows, 3, n, 1.0f, st));
      Bops = w.w_rows;
    }
    gemm_add_products(g, Aops, nt, Bops, ntw);
    BS_TRY(launch_gemm(g, st));
  }
  // the new rounding's residuals over K trials
  {
    ProfScope prof("grid_fresh", st);
    const int64_t groups = T * d / 4;
    grid_fresh_kernel<<<(unsigned)((groups + 255) / 256), 256, 0, st>>>(w.u, w.uq, io.step, T, d, io.bits, io.seed,
                                                                       base + 1, io.K, w.eN, w.eE);
    BS_CHECK_LAUNCH();
  }
  // weight use: reference and the U, N and R+e biases, contractions of [d][Tp] planes with dY^T
  BS_TRY(launch_planes(io.dY, gt, T, n, n, true, w.dyT, nt, Tp, 1.0f, st));
  const float* srcs[4] = {w.uq, w.eU, w.eN, w.eE};
  float* dsts[4] = {io.dW_ref, w.bias_w[0], w.bias_w[1], w.bias_w[2]};
  for (int i = 0; i < 4; ++i) {
    BS_TRY(launch_planes(srcs[i], BS_F32, T, d, d, true, w.aT, 3, Tp, 1.0f, st));
    GemmArgs g{};
    g.M = (int)d;
    g.N = (int)n;
    g.K = (int)Tp;
    g.lda = Tp;
    g.ldb = Tp;
    g.ldc = n;
    g.alpha = 1.0f;
    g.C = dsts[i];
    g.part = w.gemm_part;
    g.part_cap = w.gemm_part_cap;
    if (!gemm_add_products(g, w.aT, 3, w.dyT, nt)) return BS_EINVAL;
    BS_TRY(launch_gemm(g, st));
  }
  // gain use: fp64 column sums
  {
    const int64_t nch = (T + GRID_GAIN_RT - 1) / GRID_GAIN_RT;
    const dim3 grid((unsigned)nch, (unsigned)((d + 63) / 64));
    if (xt == BS_F32)
      grid_gain_kernel<float><<<grid, 64, 0, st>>>((const float*)io.X, w.rstd, io.gain, w.u, w.du, w.eU, w.eE, T, d,
                                                   w.gpart);
    else
      grid_gain_kernel<u16><<<grid, 64, 0, st>>>((const u16*)io.X, w.rstd, io.gain, w.u, w.du, w.eU, w.eE, T, d,
                                                 w.gpart);
    BS_CHECK_LAUNCH();
    BS_TRY(launch_gain_final(w.gpart, nch, d, io.dgain_ref, w.bias_rg, w.bias_ng, st));
  }
  // the normalization input gradient with unrounded values
  if (xt == BS_F32) {
    DxArgs<float> da{(const float*)io.X, w.rstd, io.gain, w.du, nullptr, nullptr, F8{}, T, d, io.dX_ref, nullptr};
    BS_TRY(launch_dx_t(da, st));
  } else {
    DxArgs<u16> da{(const u16*)io.X, w.rstd, io.gain, w.du, nullptr, nullptr, F8{}, T, d, io.dX_ref, nullptr};
    BS_TRY(launch_dx_t(da, st));
  }
  // per-policy estimates
  // every policy's estimates, one pass per gradient over its reference
  CombineMulti cg{}, cw{};
  cg.ref = io.dgain_ref;
  cw.ref = io.dW_ref;
  cg.n_pol = cw.n_pol = io.n_pol;
  cg.mean = io.dgain.mean;
  cg.bias_out = io.dgain.bias;
  cw.mean = io.dW.mean;
  cw.bias_out = io.dW.bias;
  for (int i = 0; i < io.n_pol; ++i) {
    const bs_grid_policy& q = io.pol[i];
    cg.bias[i] = q.gain_use == BS_READ_R ? w.bias_rg : (q.gain_use == BS_READ_N ? w.bias_ng : nullptr);
    cw.bias[i] = q.weight_use == BS_WREAD_U       ? w.bias_w[0]
                 : q.weight_use == BS_WREAD_N     ? w.bias_w[1]
                 : q.weight_use == BS_WREAD_R_EPS ? w.bias_w[2]
                                                  : nullptr;
  }
  BS_TRY(launch_combine_multi(cg, d, st));
  BS_TRY(launch_combine_multi(cw, d * n, st));
  return BS_OK;
}

}  // namespace bsp

using namespace bsp;

extern "C" {

size_t bs_rmsnorm_linear_grid_workspace_size(int64_t T, int64_t d, int64_t n) { return grid_ws_size(T, d, n); }

bs_status bs_rmsnorm_linear_grid_fwd_bwd(const void* X, const float* gain, const void* W, const void* dY, bs_dtype dt,
                                         int64_t T, int64_t d, int64_t n, float eps, int bits,
                                         const bs_grid_policy* pol, int n_pol, int K, uint64_t seed,
                                         uint32_t store_id, float* Y, int8_t* u_codes, float* u_step,
                                         float* dgain_ref, float* dW_ref, float* dX_ref, bs_est dgain, bs_est dW,
                                         bs_diag* diag, void* ws, size_t ws_bytes, void* stream) {
  GridIO io{X, W, dY, gain, dt, T, d, n, eps, bits, pol, n_pol, K, seed, store_id, Y, u_codes, u_step, dgain_ref,
            dW_ref, dX_ref, dgain, dW, diag};
  return grid_run(io, ws, ws_bytes, (hipStream_t)stream);
}

}  // extern "C"
