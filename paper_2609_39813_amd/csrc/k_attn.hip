// Attention with an FP8 store of its output and a backward whose correction term D reads
// the original, the forward's rounding or a new rounding of that output (gfx950, dh = 64).
//
// All tiles are 64 x 64 bf16 in LDS with rows of 128 B whose 16-byte chunks are XOR-swizzled
// by (row & 7); MFMA 16x16x32 bf16 operands are read as 16-byte fragments: lane l takes row
// r0 + (l & 15), columns k0 + 8 (l >> 4) .. + 7. A 16x16 result tile holds D[4 (l >> 4) + r]
// [l & 15] in register r of lane l. fp32-valued operands (P, dS, P*dD) enter as three exact
// bf16 terms. Four waves per workgroup; wave w owns rows 16 w .. 16 w + 15 of a 64-row block.
#include "bsp_kernels.h"
#include "k_attn.h"

namespace bsp {

constexpr int AT = 64;  // block rows / keys, and dh

__device__ __forceinline__ int sw(int row, int col) { return row * AT + ((((col >> 3) ^ (row & 7)) << 3) | (col & 7)); }

__device__ __forceinline__ bf16x8 frag(const u16* T, int r0, int k0, int lane) {
  return *(const bf16x8*)(T + sw(r0 + (lane & 15), k0 + ((lane >> 4) << 3)));
}

__device__ __forceinline__ floatx4 mfma(bf16x8 a, bf16x8 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// rows [r0, r0 + 64) of a [S, 64] bf16 matrix into a tile (row-major), zero beyond S
__device__ __forceinline__ void load_tile(u16* T, const u16* __restrict__ g, int r0, int S) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = (tid >> 3) + 32 * i, c = (tid & 7) * 8;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (r0 + r < S) v = *(const uint4*)(g + (int64_t)(r0 + r) * AT + c);
    *(uint4*)(T + sw(r, c)) = v;
  }
}

// the same rows, transposed: T[c][r]
__device__ __forceinline__ void load_tile_t(u16* T, const u16* __restrict__ g, int r0, int S) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = (tid >> 3) + 32 * i, c = (tid & 7) * 8;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (r0 + r < S) v = *(const uint4*)(g + (int64_t)(r0 + r) * AT + c);
    const u16* e = (const u16*)&v;
#pragma unroll
    for (int q = 0; q < 8; ++q) T[sw(c + q, r)] = e[q];
  }
}

// rows [r0, r0 + 64) of a [S, 64] fp32 matrix as three exact bf16 terms (row-major tiles)
__device__ __forceinline__ void load_tile3(u16* const* T, const float* __restrict__ g, int r0, int S) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = (tid >> 3) + 32 * i, c = (tid & 7) * 8;
    float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (r0 + r < S) {
      const float4 a = *(const float4*)(g + (int64_t)(r0 + r) * AT + c);
      const float4 b = *(const float4*)(g + (int64_t)(r0 + r) * AT + c + 4);
      v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    }
    u16 o[3][8];
#pragma unroll
    for (int q = 0; q < 8; ++q) split3(v[q], o[0][q], o[1][q], o[2][q]);
#pragma unroll
    for (int p = 0; p < 3; ++p) *(uint4*)(T[p] + sw(r, c)) = *(const uint4*)o[p];
  }
}

// the same rows transposed: T_p[c][r]
__device__ __forceinline__ void load_tile3_t(u16* const* T, const float* __restrict__ g, int r0, int S) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = (tid >> 3) + 32 * i, c = (tid & 7) * 8;
    float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (r0 + r < S) {
      const float4 a = *(const float4*)(g + (int64_t)(r0 + r) * AT + c);
      const float4 b = *(const float4*)(g + (int64_t)(r0 + r) * AT + c + 4);
      v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      u16 o0, o1, o2;
      split3(v[q], o0, o1, o2);
      const int idx = sw(c + q, r);
      T[0][idx] = o0;
      T[1][idx] = o1;
      T[2][idx] = o2;
    }
  }
}

__device__ __forceinline__ void put3(u16* T0, u16* T1, u16* T2, int row, int col, float v) {
  u16 a, b, c;
  split3(v, a, b, c);
  const int i = sw(row, col);
  T0[i] = a;
  T1[i] = b;
  T2[i] = c;
}

__device__ __forceinline__ float group16_max(float v) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float group16_sum(float v) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// ------------------------------------------------------------------------------------
// forward: row max m, row sum l (P = exp(c S - m) / l) and optionally O = P V
// ------------------------------------------------------------------------------------
template <bool WRITE_O>
__global__ __launch_bounds__(256) void attn_fwd_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) u16 sQ[AT * AT], sK[AT * AT], sVt[AT * AT], sP[3][AT * AT];
  const int qb = blockIdx.x, bh = blockIdx.y;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int q0 = qb * AT;
  const int64_t hb = (int64_t)bh * a.S * AT;
  load_tile(sQ, a.Q + hb, q0, a.S);
  float mr[4], lr[4];
  floatx4 acc[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    mr[r] = -INFINITY;
    lr[r] = 0.0f;
    acc[r] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  const int nkb = a.causal ? qb + 1 : (a.S + AT - 1) / AT;
  for (int kb = 0; kb < nkb; ++kb) {
    __syncthreads();
    load_tile(sK, a.K + hb, kb * AT, a.S);
    load_tile_t(sVt, a.V + hb, kb * AT, a.S);
    __syncthreads();
    floatx4 s[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) s[t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < AT; kk += 32) {
      const bf16x8 fa = frag(sQ, 16 * w, kk, lane);
#pragma unroll
      for (int t = 0; t < 4; ++t) s[t] = mfma(fa, frag(sK, 16 * t, kk, lane), s[t]);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int ql = 16 * w + 4 * (lane >> 4) + r, q = q0 + ql;
      float x[4];
      float mx = -INFINITY;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int key = kb * AT + 16 * t + (lane & 15);
        const bool ok = key < a.S && q < a.S && (!a.causal || key <= q);
        x[t] = ok ? a.scale * s[t][r] : -INFINITY;
        mx = fmaxf(mx, x[t]);
      }
      mx = group16_max(mx);
      const float mn = fmaxf(mr[r], mx);
      const float alpha = mn == -INFINITY ? 0.0f : (mr[r] == -INFINITY ? 0.0f : expf(mr[r] - mn));
      float rs = 0.0f;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const float p = x[t] == -INFINITY ? 0.0f : expf(x[t] - mn);
        rs += p;
        put3(sP[0], sP[1], sP[2], ql, 16 * t + (lane & 15), p);
      }
      rs = group16_sum(rs);
      lr[r] = lr[r] * alpha + rs;
      mr[r] = mn;
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[t][r] *= alpha;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < AT; kk += 32) {
#pragma unroll
      for (int tm = 0; tm < 3; ++tm) {
        const bf16x8 fa = frag(sP[tm], 16 * w, kk, lane);
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] = mfma(fa, frag(sVt, 16 * t, kk, lane), acc[t]);
      }
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int q = q0 + 16 * w + 4 * (lane >> 4) + r;
    if (q >= a.S) continue;
    if ((lane & 15) == 0) {
      a.m[(int64_t)bh * a.S + q] = mr[r];
      a.l[(int64_t)bh * a.S + q] = lr[r];
    }
    if (WRITE_O) {
#pragma unroll
      for (int t = 0; t < 4; ++t) a.O_out[hb + (int64_t)q * AT + 16 * t + (lane & 15)] = acc[t][r] / lr[r];
    }
  }
}

// ------------------------------------------------------------------------------------
// D variants, one row per 16 lanes (4 elements per lane, one Philox call per trial):
//   D_ref = sum dO O; dD_R = sum dO (s val(C_O) - O);
//   dD_k  = sum dO (s val(C_k) - O) for new roundings k = 1..K, = A + s S_k with
//   A = sum dO (s sign lo - O), S_k = sum dO sign step up_k; mean and sample SD over k (fp64).
// ------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void attn_d_kernel(AttnDArgs a) {
  const int64_t row = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
  const int sub = threadIdx.x & 15;
  const bool ok = row < a.rows;
  const int64_t e0 = row * AT + 4 * sub;
  const float s = *a.scale;
  double dref = 0.0, dr = 0.0, A = 0.0;
  uint32_t F[4] = {0, 0, 0, 0};
  double w[4] = {0.0, 0.0, 0.0, 0.0};
  if (ok) {
    const float4 o4 = *(const float4*)(a.O + e0);
    const uint32_t c4 = *(const uint32_t*)(a.codes + e0);
    const float ov[4] = {o4.x, o4.y, o4.z, o4.w};
    float dv[4];
    if (a.dO32) {
      const float4 g4 = *(const float4*)(a.dO32 + e0);
      dv[0] = g4.x; dv[1] = g4.y; dv[2] = g4.z; dv[3] = g4.w;
    } else {
      const uint2 d2 = *(const uint2*)(a.dO + e0);
      dv[0] = bf16_to_f32((u16)(d2.x & 0xFFFF));
      dv[1] = bf16_to_f32((u16)(d2.x >> 16));
      dv[2] = bf16_to_f32((u16)(d2.y & 0xFFFF));
      dv[3] = bf16_to_f32((u16)(d2.y >> 16));
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const double o = ov[q], g = dv[q];
      dref += g * o;
      dr += g * ((double)s * (double)f8_value((c4 >> (8 * q)) & 0xFFu, a.f) - o);
      const float y = __fdiv_rn(ov[q], s);
      const Bracket b = f8_bracket(fminf(fabsf(y), a.f.fmax), a.f);
      const double sg = signbit(y) ? -1.0 : 1.0;
      const double step = f8_step(b);
      A += g * ((double)s * sg * (double)b.mi * step - o);
      F[q] = sr_threshold(b.frac);
      w[q] = g * sg * step;
    }
  }
  // fixed-order sums over the 16 lanes of a row (xor tree 8, 4, 2, 1)
  auto rowsum = [&](double v) {
#pragma unroll
    for (int o = 8; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
  };
  dref = rowsum(dref);
  dr = rowsum(dr);
  A = rowsum(A);
  double mean = 0.0, m2 = 0.0;
  if (a.want_n) {
    const uint64_t g = (uint64_t)(e0 >> 2);
    for (int k = 1; k <= a.K; ++k) {
      const Philox4 p = philox_group(a.seed, g, (uint32_t)k, a.use);
      const uint32_t R[4] = {p.w0, p.w1, p.w2, p.w3};
      double Sk = 0.0;
#pragma unroll
      for (int q = 0; q < 4; ++q) Sk += sr_up(F[q], R[q]) ? w[q] : 0.0;
      Sk = rowsum(Sk);
      const double dl = Sk - mean;
      mean += dl / k;
      m2 += dl * (Sk - mean);
    }
  }
  if (ok && sub == 0) {
    a.D_ref[row] = (float)dref;
    a.dD_R[row] = (float)dr;
    if (a.want_n) {
      a.dD_N[row] = (float)(A + (double)s * mean);
      a.sd_N[row] = a.K > 1 ? (float)((double)s * sqrt(m2 / (a.K - 1))) : 0.0f;
    }
  }
}

// ------------------------------------------------------------------------------------
// backward, query-block-major: dQ = c dS K and G = P K; per-policy dQ estimates
//   bias_v = -c dD_v G (row-scaled), se_N = c |G| sd_N / sqrt(K).
// ------------------------------------------------------------------------------------
template <int NDO>
__global__ __launch_bounds__(256) void attn_bwd_q_kernel(AttnBwdArgs a) {
  __shared__ __attribute__((aligned(16))) u16 sQ[AT * AT], sdO[NDO][AT * AT], sK[AT * AT], sV[AT * AT], sKt[AT * AT],
      sP[3][AT * AT], sdS[3][AT * AT];
  const int qb = blockIdx.x, bh = blockIdx.y;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int q0 = qb * AT;
  const int64_t hb = (int64_t)bh * a.S * AT, rb = (int64_t)bh * a.S;
  load_tile(sQ, a.Q + hb, q0, a.S);
  if (NDO == 1) {
    load_tile(sdO[0], a.dO + hb, q0, a.S);
  } else {
    u16* const t3[3] = {sdO[0], sdO[NDO > 1 ? 1 : 0], sdO[NDO > 2 ? 2 : 0]};
    load_tile3(t3, a.dO32 + hb, q0, a.S);
  }
  float mr[4], il[4], dr[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int q = q0 + 16 * w + 4 * (lane >> 4) + r;
    const bool ok = q < a.S;
    mr[r] = ok ? a.m[rb + q] : 0.0f;
    il[r] = ok ? a.l[rb + q] : 1.0f;
    dr[r] = ok ? a.D_ref[rb + q] : 0.0f;
  }
  floatx4 aq[4], ag[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) aq[t] = ag[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int nkb = a.causal ? qb + 1 : (a.S + AT - 1) / AT;
  for (int kb = 0; kb < nkb; ++kb) {
    __syncthreads();
    load_tile(sK, a.K + hb, kb * AT, a.S);
    load_tile(sV, a.V + hb, kb * AT, a.S);
    load_tile_t(sKt, a.K + hb, kb * AT, a.S);
    __syncthreads();
    floatx4 s[4], dp[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) s[t] = dp[t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < AT; kk += 32) {
      const bf16x8 fq = frag(sQ, 16 * w, kk, lane);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const bf16x8 fv = frag(sV, 16 * t, kk, lane);
        s[t] = mfma(fq, frag(sK, 16 * t, kk, lane), s[t]);
#pragma unroll
        for (int i = 0; i < NDO; ++i) dp[t] = mfma(frag(sdO[i], 16 * w, kk, lane), fv, dp[t]);
      }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int ql = 16 * w + 4 * (lane >> 4) + r, q = q0 + ql;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int kl = 16 * t + (lane & 15), key = kb * AT + kl;
        const bool ok = key < a.S && q < a.S && (!a.causal || key <= q);
        const float p = ok ? expf(a.scale * s[t][r] - mr[r]) / il[r] : 0.0f;
        put3(sP[0], sP[1], sP[2], ql, kl, p);
        put3(sdS[0], sdS[1], sdS[2], ql, kl, p * (dp[t][r] - dr[r]));
      }
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < AT; kk += 32) {
#pragma unroll
      for (int tm = 0; tm < 3; ++tm) {
        const bf16x8 fs = frag(sdS[tm], 16 * w, kk, lane), fp = frag(sP[tm], 16 * w, kk, lane);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const bf16x8 fk = frag(sKt, 16 * t, kk, lane);
          aq[t] = mfma(fs, fk, aq[t]);
          ag[t] = mfma(fp, fk, ag[t]);
        }
      }
    }
  }
  const float c = a.scale;
  const float rk = a.ntrial > 0 ? 1.0f / sqrtf((float)a.ntrial) : 0.0f;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int q = q0 + 16 * w + 4 * (lane >> 4) + r;
    if (q >= a.S) continue;
    const float ddr = a.dD_R ? a.dD_R[rb + q] : 0.0f;
    const float ddn = a.dD_N ? a.dD_N[rb + q] : 0.0f;
    const float sdn = a.sd_N ? a.sd_N[rb + q] : 0.0f;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int64_t e = hb + (int64_t)q * AT + 16 * t + (lane & 15);
      const float dq = c * aq[t][r];
      const float g = ag[t][r];
      a.dQ_ref[e] = dq;
      for (int p = 0; p < a.n_pol; ++p) {
        const int kind = a.pol[p];
        const float bias = kind == BS_READ_U ? 0.0f : -c * (kind == BS_READ_R ? ddr : ddn) * g;
        if (a.mean[p]) a.mean[p][e] = dq + bias;
        if (a.bias[p]) a.bias[p][e] = bias;
        if (a.se[p]) a.se[p][e] = kind == BS_READ_N ? c * fabsf(g) * sdn * rk : 0.0f;
      }
    }
  }
}

// ------------------------------------------------------------------------------------
// backward, key-block-major: dV = P^T dO, dK = c dS^T Q and the bias terms
// dK_v = -c P^T (dD_v * Q) for v in {R, N}, from S^T = K Q^T so that each wave reads only
// its own key rows of the P^T / dS^T tiles.
// ------------------------------------------------------------------------------------
template <int NDO>
__global__ __launch_bounds__(256) void attn_bwd_k_kernel(AttnBwdArgs a) {
  __shared__ __attribute__((aligned(16))) u16 sK[AT * AT], sV[AT * AT], sQ[AT * AT], sQt[AT * AT], sdO[NDO][AT * AT],
      sdOt[NDO][AT * AT], sPt[3][AT * AT], sdSt[3][AT * AT];
  __shared__ float rowm[AT], rowil[AT], rowd[AT], rowdr[AT], rowdn[AT];
  const int kb = blockIdx.x, bh = blockIdx.y;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int k0 = kb * AT;
  const int64_t hb = (int64_t)bh * a.S * AT, rb = (int64_t)bh * a.S;
  load_tile(sK, a.K + hb, k0, a.S);
  load_tile(sV, a.V + hb, k0, a.S);
  floatx4 av[4], ak[4], akr[4], akn[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) av[t] = ak[t] = akr[t] = akn[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int nqb = (a.S + AT - 1) / AT;
  for (int qb = a.causal ? kb : 0; qb < nqb; ++qb) {
    const int q0 = qb * AT;
    __syncthreads();
    load_tile(sQ, a.Q + hb, q0, a.S);
    load_tile_t(sQt, a.Q + hb, q0, a.S);
    if (NDO == 1) {
      load_tile(sdO[0], a.dO + hb, q0, a.S);
      load_tile_t(sdOt[0], a.dO + hb, q0, a.S);
    } else {
      u16* const t3[3] = {sdO[0], sdO[NDO > 1 ? 1 : 0], sdO[NDO > 2 ? 2 : 0]};
      u16* const t3t[3] = {sdOt[0], sdOt[NDO > 1 ? 1 : 0], sdOt[NDO > 2 ? 2 : 0]};
      load_tile3(t3, a.dO32 + hb, q0, a.S);
      load_tile3_t(t3t, a.dO32 + hb, q0, a.S);
    }
    if (threadIdx.x < AT) {
      const int q = q0 + threadIdx.x;
      const bool ok = q < a.S;
      rowm[threadIdx.x] = ok ? a.m[rb + q] : 0.0f;
      rowil[threadIdx.x] = ok ? a.l[rb + q] : 1.0f;
      rowd[threadIdx.x] = ok ? a.D_ref[rb + q] : 0.0f;
      rowdr[threadIdx.x] = (ok && a.dD_R) ? a.dD_R[rb + q] : 0.0f;
      rowdn[threadIdx.x] = (ok && a.dD_N) ? a.dD_N[rb + q] : 0.0f;
    }
    __syncthreads();
    // S^T and dP^T for keys 16w.. of this block, all 64 queries
    floatx4 s[4], dp[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) s[t] = dp[t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < AT; kk += 32) {
      const bf16x8 fk = frag(sK, 16 * w, kk, lane), fv = frag(sV, 16 * w, kk, lane);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        s[t] = mfma(fk, frag(sQ, 16 * t, kk, lane), s[t]);
#pragma unroll
        for (int i = 0; i < NDO; ++i) dp[t] = mfma(fv, frag(sdO[i], 16 * t, kk, lane), dp[t]);
      }
    }
    float pv[4][4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int kl = 16 * w + 4 * (lane >> 4) + r, key = k0 + kl;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int ql = 16 * t + (lane & 15), q = q0 + ql;
        const bool ok = key < a.S && q < a.S && (!a.causal || key <= q);
        const float p = ok ? expf(a.scale * s[t][r] - rowm[ql]) / rowil[ql] : 0.0f;
        pv[t][r] = p;
        put3(sPt[0], sPt[1], sPt[2], kl, ql, p);
        put3(sdSt[0], sdSt[1], sdSt[2], kl, ql, p * (dp[t][r] - rowd[ql]));
      }
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < AT; kk += 32) {
#pragma unroll
      for (int tm = 0; tm < 3; ++tm) {
        const bf16x8 fp = frag(sPt[tm], 16 * w, kk, lane), fs = frag(sdSt[tm], 16 * w, kk, lane);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
#pragma unroll
          for (int i = 0; i < NDO; ++i)
            if (tm + i <= 2) av[t] = mfma(fp, frag(sdOt[i], 16 * t, kk, lane), av[t]);
          ak[t] = mfma(fs, frag(sQt, 16 * t, kk, lane), ak[t]);
        }
      }
    }
    // bias terms: P^T scaled by dD_v per query, reusing the P^T tiles of this wave's rows
    for (int v = 0; v < 2; ++v) {
      if (v == 0 ? !a.dD_R : !a.dD_N) continue;
      const float* dd = v == 0 ? rowdr : rowdn;
      __syncthreads();
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int kl = 16 * w + 4 * (lane >> 4) + r;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int ql = 16 * t + (lane & 15);
          put3(sPt[0], sPt[1], sPt[2], kl, ql, pv[t][r] * dd[ql]);
        }
      }
      __syncthreads();
#pragma unroll
      for (int kk = 0; kk < AT; kk += 32) {
#pragma unroll
        for (int tm = 0; tm < 3; ++tm) {
          const bf16x8 fp = frag(sPt[tm], 16 * w, kk, lane);
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            if (v == 0)
              akr[t] = mfma(fp, frag(sQt, 16 * t, kk, lane), akr[t]);
            else
              akn[t] = mfma(fp, frag(sQt, 16 * t, kk, lane), akn[t]);
          }
        }
      }
    }
  }
  const float c = a.scale;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int key = k0 + 16 * w + 4 * (lane >> 4) + r;
    if (key >= a.S) continue;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int64_t e = hb + (int64_t)key * AT + 16 * t + (lane & 15);
      const float dk = c * ak[t][r];
      a.dV[e] = av[t][r];
      a.dK_ref[e] = dk;
      for (int p = 0; p < a.n_pol; ++p) {
        const int kind = a.pol[p];
        const float bias = kind == BS_READ_U ? 0.0f : -c * (kind == BS_READ_R ? akr[t][r] : akn[t][r]);
        if (a.kmean[p]) a.kmean[p][e] = dk + bias;
        if (a.kbias[p]) a.kbias[p][e] = bias;
      }
    }
  }
}

// ------------------------------------------------------------------------------------
bs_status launch_attn_fwd(const AttnArgs& a, int B, int H, hipStream_t st) {
  dim3 grid((unsigned)((a.S + AT - 1) / AT), (unsigned)(B * H));
  ProfScope prof("attn_fwd", st);
  if (a.O_out)
    attn_fwd_kernel<true><<<grid, 256, 0, st>>>(a);
  else
    attn_fwd_kernel<false><<<grid, 256, 0, st>>>(a);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status launch_attn_d(const AttnDArgs& a, hipStream_t st) {
  if (a.rows <= 0) return BS_OK;
  attn_d_kernel<<<(unsigned)((a.rows + 15) / 16), 256, 0, st>>>(a);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status launch_attn_bwd(const AttnBwdArgs& a, int B, int H, hipStream_t st) {
  dim3 grid((unsigned)((a.S + AT - 1) / AT), (unsigned)(B * H));
  ProfScope prof("attn_bwd", st);
  if (a.dO32) {
    attn_bwd_k_kernel<3><<<grid, 256, 0, st>>>(a);
    attn_bwd_q_kernel<3><<<grid, 256, 0, st>>>(a);
  } else {
    attn_bwd_k_kernel<1><<<grid, 256, 0, st>>>(a);
    attn_bwd_q_kernel<1><<<grid, 256, 0, st>>>(a);
  }
  BS_CHECK_LAUNCH();
  return BS_OK;
}

}  // namespace bsp
