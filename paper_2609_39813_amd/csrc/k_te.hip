// An emulation of an FP8 attention backward with delayed scaling (App. D.2; App. E.3), dh = 64:
// dO cast to E5M2 at its delayed scale; P re-formed and stored in E4M3 at the forward's scale;
// dV = P_q^T dO_q; dP = dO_q V^T; D from the selected source; dS = P (dP - D) cast to E5M2 at its
// delayed scale; dQ = c dS_q K, dK = c dS_q^T Q; dQ, dK and dV cast to E5M2 at the gradients'
// delayed scale. Every cast rounds to nearest even after clamping |x / s| to FMAX (counted). The
// amaxes of dO, of the pre-cast dS and of the pre-cast gradients are reported for the caller's
// histories.
//
// Every product has exact bf16 operands (FP8 values and bf16 inputs), one MFMA term each, with
// the scales applied in fp32 after the accumulation. The query-major pass writes the dS and P
// codes tile by tile ([key][query], one byte each) for the key-major pass.
#include "k_attn.h"
#include "k_qmajor.h"

#define BS_TRY(x)               \
  do {                          \
    const bs_status _s = (x);   \
    if (_s != BS_OK) return _s; \
  } while (0)

namespace bsp {

namespace {

struct TeArgs {
  const u16 *Q, *K, *V, *dO;   // dO: the E5M2 incoming gradient's code values (dO_q / s_dO), bf16
  const u16 *Qt, *Kt, *dOt;    // transposed copies [BH][64][Sp]
  int S, Sp, causal, BH;
  float scale;                 // softmax scale c
  const float *m, *l;
  const float* sc;             // device [4]: s_P, s_dO, s_dS, s_g
  const float* D;              // [rows] the correction term
  uint8_t *dsq, *pq;           // tile-major codes [BH][tiles][64 key][64 query]
  float *P_out, *dS_out;       // nullable [BH][S][S]: the realized P and pre-cast dS
  uint8_t *P_codes, *dS_codes; // nullable [BH][S][S]
  float* pre;                  // nullable [3][BH][S][64]: pre-cast dQ, dK, dV
  float *dQ, *dK, *dV;
  uint32_t* amax;              // [3] fp32 bits: dO, dS, gradients
  uint32_t* counts;            // [4]: saturated rows, clamps of dO, dS and the gradients
};

constexpr float kE5M2Max = 57344.0f, kE4M3Max = 448.0f;

// RNE codes of 4 values already divided by their scale, clamped to +-FMAX first; returns the
// number of clamped values in nsat
template <int FMT>
__device__ __forceinline__ uint32_t codes4(const float (&y)[4], uint32_t& nsat) {
  const float fm = FMT == BS_E5M2 ? kE5M2Max : kE4M3Max;
  float c[4];
  nsat = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    nsat += fabsf(y[i]) > fm ? 1u : 0u;
    c[i] = __builtin_amdgcn_fmed3f(y[i], -fm, fm);
  }
  uint32_t w = FMT == BS_E5M2 ? (uint32_t)__builtin_amdgcn_cvt_pk_bf8_f32(c[0], c[1], 0, false)
                              : (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(c[0], c[1], 0, false);
  w = FMT == BS_E5M2 ? (uint32_t)__builtin_amdgcn_cvt_pk_bf8_f32(c[2], c[3], (int)w, true)
                     : (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(c[2], c[3], (int)w, true);
  return w;
}

// largest of v >= 0 over the wave, folded into *p (fp32 bits of non-negative values order as integers)
__device__ __forceinline__ void atomic_amax(uint32_t* p, float v) {
  const uint32_t m = wave_max_u32(__float_as_uint(v));
  if ((threadIdx.x & 63) == 0 && m) atomicMax(p, m);
}
__device__ __forceinline__ void atomic_count(uint32_t* p, uint32_t v) {
  v = wave_sum_u32(v);
  if ((threadIdx.x & 63) == 0 && v) atomicAdd(p, v);
}

__global__ void te_init_kernel(uint32_t* amax, uint32_t* counts) {
  if (threadIdx.x < 3) amax[threadIdx.x] = 0u;
  if (threadIdx.x < 4) counts[threadIdx.x] = 0u;
}

// dO -> its E5M2 code values (bf16, exact), 4 elements per thread
__global__ __launch_bounds__(256) void te_prep_kernel(const u16* __restrict__ dO, int64_t n, const float* sc,
                                                      u16* __restrict__ dOq, uint32_t* amax, uint32_t* counts) {
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  const float s = sc[1];
  float am = 0.0f;
  uint32_t nsat = 0;
  if (i < n) {
    const uint2 d2 = *(const uint2*)(dO + i);
    const float x[4] = {bf16_to_f32((u16)(d2.x & 0xFFFF)), bf16_to_f32((u16)(d2.x >> 16)),
                        bf16_to_f32((u16)(d2.y & 0xFFFF)), bf16_to_f32((u16)(d2.y >> 16))};
    float y[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      am = fmaxf(am, fabsf(x[r]));
      y[r] = x[r] / s;
    }
    const uint32_t w = codes4<BS_E5M2>(y, nsat);
    u16 v[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] = (u16)(__float_as_uint(f8_val<BS_E5M2>(w, r)) >> 16);  // exact in bf16
    *(uint2*)(dOq + i) = make_uint2((uint32_t)v[0] | ((uint32_t)v[1] << 16), (uint32_t)v[2] | ((uint32_t)v[3] << 16));
  }
  atomic_amax(&amax[0], am);
  atomic_count(&counts[1], nsat);
}

// D per row (4 lanes per row, 16 elements each), in fp64 from exact operands: dO_q against the
// forward's P V (P), the original O (U), the E4M3 store of O (R), a new stochastic rounding of O
// at the store's scale (N), or the repair (P where the row's largest probability, exactly
// fl32(1 / l), reaches the threshold, R elsewhere). Rows at or over the threshold are counted.
__global__ __launch_bounds__(256) void te_d_kernel(const u16* __restrict__ dOq, const float* __restrict__ OP,
                                                   const float* __restrict__ O, const uint8_t* __restrict__ Oc,
                                                   const float* Os, const float* __restrict__ l, int64_t rows,
                                                   int source, float thr, uint64_t seed, uint32_t trial, uint32_t use,
                                                   const float* sc, float* __restrict__ D, uint32_t* counts) {
  const int64_t row = (int64_t)blockIdx.x * 64 + (threadIdx.x >> 2);
  const int sub = threadIdx.x & 3;
  const bool ok = row < rows;
  const F8 f = f8_format(BS_E4M3);
  const bool sat = ok && 1.0f / l[ok ? row : 0] >= thr;
  const int src = source == BS_D_REPAIR ? (sat ? BS_D_FROM_P : BS_D_R) : source;
  double acc = 0.0;
  if (ok) {
    const int64_t e0 = row * AT + 16 * sub;
    const float so = (src == BS_D_R || src == BS_D_N) ? *Os : 1.0f;
    const double rs = 1.0 / (double)so;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t e = e0 + 4 * j;
      const uint2 d2 = *(const uint2*)(dOq + e);
      const float g[4] = {bf16_to_f32((u16)(d2.x & 0xFFFF)), bf16_to_f32((u16)(d2.x >> 16)),
                          bf16_to_f32((u16)(d2.y & 0xFFFF)), bf16_to_f32((u16)(d2.y >> 16))};
      double c[4];
      if (src == BS_D_FROM_P || src == BS_D_U) {
        const float4 o4 = *(const float4*)((src == BS_D_FROM_P ? OP : O) + e);
        c[0] = o4.x;
        c[1] = o4.y;
        c[2] = o4.z;
        c[3] = o4.w;
      } else if (src == BS_D_R) {
        const uint32_t w = *(const uint32_t*)(Oc + e);
#pragma unroll
        for (int r = 0; r < 4; ++r) c[r] = (double)so * (double)f8_value((w >> (8 * r)) & 0xFFu, f);
      } else {
        const float4 o4 = *(const float4*)(O + e);
        const float ov[4] = {o4.x, o4.y, o4.z, o4.w};
        const Philox4 p = philox_group(seed, (uint64_t)(e >> 2), trial, use);
        const uint32_t R[4] = {p.w0, p.w1, p.w2, p.w3};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float y = div_scale(ov[r], rs);
          const Bracket b = f8_bracket(fminf(fabsf(y), f.fmax), f);
          const double mag = (double)(b.mi + sr_up(b.F, R[r])) * (double)f8_step(b);
          c[r] = (signbit(y) ? -mag : mag) * (double)so;
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) acc += (double)g[r] * c[r];
    }
  }
  acc += __shfl_xor(acc, 1, 64);
  acc += __shfl_xor(acc, 2, 64);
  if (ok && sub == 0) D[row] = (float)((double)sc[1] * acc);
  atomic_count(&counts[0], (ok && sub == 0 && sat) ? 1u : 0u);
}

// query-major: dS = P (dP - D), its E5M2 codes at s_dS and P's E4M3 codes at s_P (tile-major),
// dQ = c s_dS val(dS_q) K cast at s_g
__global__ __launch_bounds__(256) void te_dq_kernel(TeArgs a) {
  __shared__ __attribute__((aligned(16))) u16 sm[2][3][AT * AT];  // K, V, K^T
  const QMajor z = qmajor_setup(a, true);
  const float sP = a.sc[0], sdO = a.sc[1], sdS = a.sc[2], sg = a.sc[3];
  const float Dq = z.qok ? a.D[z.rb + z.q] : 0.0f;
  const int nqb = (a.S + AT - 1) / AT;
  floatx4 aq[4];
#pragma unroll
  for (int n = 0; n < 4; ++n) aq[n] = floatx4{0.f, 0.f, 0.f, 0.f};
  TileRegs pf[3];
  auto fetch = [&](int k0) {
    tile_fetch(pf[0], a.K + z.hb, k0, a.S);
    tile_fetch(pf[1], a.V + z.hb, k0, a.S);
    tile_fetch_t(pf[2], a.Kt + z.tb, k0, a.Sp);
  };
  auto put = [&](int st) {
    tile_put(sm[st][0], pf[0]);
    tile_put(sm[st][1], pf[1]);
    tile_put_t(sm[st][2], pf[2]);
  };
  const int nkb = a.causal ? z.qb + 1 : nqb;
  float amds = 0.0f;
  uint32_t nsat = 0;
  fetch(0);
  put(0);
  __syncthreads();
  for (int kb = 0; kb < nkb; ++kb) {
    const int st = kb & 1, k0 = kb * AT;
    if (kb + 1 < nkb) fetch(k0 + AT);
    float p[4][4], dp[4][4];
    probs(a, z, sm[st][0], k0, p);
    dprobs(z, sm[st][1], dp);
    const int64_t tile = fld_tile(a, z.bh, z.qb, kb, nqb);
    float dv[4][4];  // the dS codes' values
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int key = k0 + 16 * t + 4 * z.g;
      float ds[4], y[4], yp[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        ds[r] = p[t][r] * (sdO * dp[t][r] - Dq);
        amds = fmaxf(amds, fabsf(ds[r]));
        y[r] = ds[r] / sdS;
        yp[r] = p[t][r] / sP;
      }
      uint32_t ns, nsp;
      const uint32_t wd = codes4<BS_E5M2>(y, ns), wp = codes4<BS_E4M3>(yp, nsp);
      nsat += ns;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        dv[t][r] = f8_val<BS_E5M2>(wd, r);
        const int64_t o = tile + (16 * t + 4 * z.g + r) * AT + 16 * z.w + z.c16;
        a.dsq[o] = (uint8_t)(wd >> (8 * r));
        a.pq[o] = (uint8_t)(wp >> (8 * r));
      }
      if (z.qok && key < a.S) {
        const uint64_t e = pelem(a, z, key);
        if (a.dS_out) *(float4*)(a.dS_out + e) = make_float4(ds[0], ds[1], ds[2], ds[3]);
        if (a.P_out) *(float4*)(a.P_out + e) = make_float4(p[t][0], p[t][1], p[t][2], p[t][3]);
        if (a.dS_codes) *(uint32_t*)(a.dS_codes + e) = wd;
        if (a.P_codes) *(uint32_t*)(a.P_codes + e) = wp;
      }
    }
    // dQ += val(dS_q) K (k index: keys 32 s2 + 16 (v >> 2) + 4 g + (v & 3); exact bf16 operands)
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      uint32_t pk[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int v = 2 * i;
        pk[i] = pk_bf16(dv[2 * s2 + (v >> 2)][v & 3], dv[2 * s2 + ((v + 1) >> 2)][(v + 1) & 3]);
      }
      const bf16x8 td = __builtin_bit_cast(bf16x8, make_uint4(pk[0], pk[1], pk[2], pk[3]));
#pragma unroll
      for (int n = 0; n < 4; ++n) aq[n] = mfma(td, frag_t(sm[st][2], 16 * n + z.c16, s2, z.g), aq[n]);
    }
    if (kb + 1 < nkb) put(st ^ 1);
    __syncthreads();
  }
  atomic_amax(&a.amax[1], amds);
  atomic_count(&a.counts[2], nsat);
  // dQ = c s_dS acc, cast at the gradients' scale
  const float cs = a.scale * sdS;
  float amg = 0.0f;
  uint32_t nsg = 0;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int qr = z.q0 + 16 * z.w + 4 * z.g + r;
    if (qr >= a.S) continue;
    float y[4], pre[4];
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      pre[n] = cs * aq[n][r];
      y[n] = pre[n] / sg;
      amg = fmaxf(amg, fabsf(pre[n]));
    }
    uint32_t ns;
    const uint32_t w = codes4<BS_E5M2>(y, ns);
    nsg += ns;
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const int64_t e = z.hb + (int64_t)qr * AT + 16 * n + z.c16;
      a.dQ[e] = f8_val<BS_E5M2>(w, n) * sg;
      if (a.pre) a.pre[e] = pre[n];
    }
  }
  atomic_amax(&a.amax[2], amg);
  atomic_count(&a.counts[3], nsg);
}

// key-major: dK = c s_dS sum_q val(dS_q) Q, dV = s_P s_dO sum_q val(P_q) val(dO_q), both cast at s_g
__global__ __launch_bounds__(256) void te_dkv_kernel(TeArgs a) {
  __shared__ __attribute__((aligned(16))) u16 sm[2][2][AT * AT];  // Q^T, dO_q^T
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane >> 4, c16 = lane & 15;
  const int bh = blockIdx.x, kb = blockIdx.y;  // under the causal mask block 0 walks the most query blocks
  const int k0 = kb * AT;
  const int64_t hb = (int64_t)bh * a.S * AT, tb = (int64_t)bh * AT * a.Sp;
  const int nqb = (a.S + AT - 1) / AT;
  const float sP = a.sc[0], sdO = a.sc[1], sdS = a.sc[2], sg = a.sc[3];
  floatx4 ak[4], av[4];
#pragma unroll
  for (int n = 0; n < 4; ++n) ak[n] = av[n] = floatx4{0.f, 0.f, 0.f, 0.f};
  TileRegs pf[2];
  auto fetch = [&](int q0) {
    tile_fetch_t(pf[0], a.Qt + tb, q0, a.Sp);
    tile_fetch_t(pf[1], a.dOt + tb, q0, a.Sp);
  };
  auto put = [&](int st) {
    tile_put_t(sm[st][0], pf[0]);
    tile_put_t(sm[st][1], pf[1]);
  };
  const int qb0 = a.causal ? kb : 0;
  fetch(qb0 * AT);
  put(0);
  __syncthreads();
  for (int qb = qb0; qb < nqb; ++qb) {
    const int st = (qb - qb0) & 1, q0 = qb * AT;
    if (qb + 1 < nqb) fetch(q0 + AT);
    const int64_t tile = fld_tile(a, bh, qb, kb, nqb) + (int64_t)(16 * w + c16) * AT;
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      // queries 32 s2 + 16 hh + 4 g + (0..3) of this lane's key, as the k index of the products
      float dsv[8], pv[8];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const uint32_t wd = *(const uint32_t*)(a.dsq + tile + 32 * s2 + 16 * hh + 4 * g);
        const uint32_t wp = *(const uint32_t*)(a.pq + tile + 32 * s2 + 16 * hh + 4 * g);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          dsv[4 * hh + r] = f8_val<BS_E5M2>(wd, r);
          pv[4 * hh + r] = f8_val<BS_E4M3>(wp, r);
        }
      }
      uint32_t pkd[4], pkp[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pkd[i] = pk_bf16(dsv[2 * i], dsv[2 * i + 1]);
        pkp[i] = pk_bf16(pv[2 * i], pv[2 * i + 1]);
      }
      const bf16x8 td = __builtin_bit_cast(bf16x8, make_uint4(pkd[0], pkd[1], pkd[2], pkd[3]));
      const bf16x8 tp = __builtin_bit_cast(bf16x8, make_uint4(pkp[0], pkp[1], pkp[2], pkp[3]));
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        ak[n] = mfma(td, frag_t(sm[st][0], 16 * n + c16, s2, g), ak[n]);
        av[n] = mfma(tp, frag_t(sm[st][1], 16 * n + c16, s2, g), av[n]);
      }
    }
    if (qb + 1 < nqb) put(st ^ 1);
    __syncthreads();
  }
  const float ck = a.scale * sdS, cv = sP * sdO;
  const int64_t numel = (int64_t)a.BH * a.S * AT;
  float amg = 0.0f;
  uint32_t nsg = 0;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int kr = k0 + 16 * w + 4 * g + r;
    if (kr >= a.S) continue;
    float yk[4], yv[4], prk[4], prv[4];
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      prk[n] = ck * ak[n][r];
      prv[n] = cv * av[n][r];
      yk[n] = prk[n] / sg;
      yv[n] = prv[n] / sg;
      amg = fmaxf(amg, fmaxf(fabsf(prk[n]), fabsf(prv[n])));
    }
    uint32_t nk, nv;
    const uint32_t wk = codes4<BS_E5M2>(yk, nk), wv = codes4<BS_E5M2>(yv, nv);
    nsg += nk + nv;
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const int64_t e = hb + (int64_t)kr * AT + 16 * n + c16;
      a.dK[e] = f8_val<BS_E5M2>(wk, n) * sg;
      a.dV[e] = f8_val<BS_E5M2>(wv, n) * sg;
      if (a.pre) {
        a.pre[numel + e] = prk[n];
        a.pre[2 * numel + e] = prv[n];
      }
    }
  }
  atomic_amax(&a.amax[2], amg);
  atomic_count(&a.counts[3], nsg);
}

struct TeWs {
  u16 *dOq, *Qt, *Kt, *Vt, *dOt;
  float *m, *l, *D, *OP;
  uint8_t *dsq, *pq;
};

TeWs carve_te(Carver& c, int64_t bh, int S, int causal, bool need_op) {
  TeWs w{};
  const int64_t Sp = round_up(S, AT), rows = bh * S;
  const int nqb = (int)(Sp / AT);
  w.dOq = c.take<u16>(rows * AT);
  for (u16** p : {&w.Qt, &w.Kt, &w.Vt, &w.dOt}) *p = c.take<u16>(bh * AT * Sp);
  for (float** p : {&w.m, &w.l, &w.D}) *p = c.take<float>(rows);
  if (need_op) w.OP = c.take<float>(rows * AT);
  const int64_t nt = bh * causal_tiles(nqb, causal) * AT * AT;
  w.dsq = c.take<uint8_t>(nt);
  w.pq = c.take<uint8_t>(nt);
  return w;
}

bool needs_op(int source) { return source == BS_D_FROM_P || source == BS_D_REPAIR; }

}  // namespace

struct TeIO {
  const void *Q, *K, *V, *dO;
  int B, H, S, dh, causal;
  float scale;
  const float* O;
  const uint8_t* O_codes;
  const float* O_scale;
  int source;
  float thr;
  const float* scales;
  uint64_t seed;
  uint32_t store_id, trial;
  float *dQ, *dK, *dV, *amax;
  uint32_t* counts;
  float *P_out, *dS_out;
  uint8_t *P_codes, *dS_codes;
  float* grad_pre;
};

size_t te_ws_size(int B, int H, int S, int dh, int causal, int source) {
  if (B < 1 || H < 1 || S < 1 || dh != AT || source < BS_D_FROM_P || source > BS_D_REPAIR) return 0;
  Carver c;
  carve_te(c, (int64_t)B * H, S, causal ? 1 : 0, needs_op(source));
  return c.used();
}

bs_status te_run(const TeIO& io, void* ws, size_t ws_bytes, hipStream_t st) {
  if (!io.Q || !io.K || !io.V || !io.dO || !io.scales || !io.dQ || !io.dK || !io.dV || !io.amax || !io.counts)
    return BS_EINVAL;
  if (io.B < 1 || io.H < 1 || io.S < 1 || !(io.scale > 0.0f)) return BS_EINVAL;
  if (io.source < BS_D_FROM_P || io.source > BS_D_REPAIR) return BS_EINVAL;
  const bool need_codes = io.source == BS_D_R || io.source == BS_D_REPAIR;
  if ((need_codes && !io.O_codes) || ((need_codes || io.source == BS_D_N) && !io.O_scale)) return BS_EINVAL;
  if ((io.source == BS_D_U || io.source == BS_D_N) && !io.O) return BS_EINVAL;
  if (io.dh != AT || io.S % 4 != 0) return BS_ESHAPE;
  if ((int64_t)io.B * io.H > 65535 || (io.S + AT - 1) / AT > 65535) return BS_ESHAPE;
  for (const void* p : {io.Q, io.K, io.V, io.dO, (const void*)io.O, (const void*)io.P_out, (const void*)io.dS_out})
    if ((uintptr_t)p & 15) return BS_EINVAL;  // 16-byte vector loads and stores
  for (const void* p : {(const void*)io.O_codes, (const void*)io.P_codes, (const void*)io.dS_codes})
    if ((uintptr_t)p & 3) return BS_EINVAL;
  const int64_t bh = (int64_t)io.B * io.H, Sp = round_up(io.S, AT), rows = bh * io.S, numel = rows * AT;
  const int causal = io.causal ? 1 : 0;
  Carver probe;
  carve_te(probe, bh, io.S, causal, needs_op(io.source));
  if (!ws || ((uintptr_t)ws & 255) || ws_bytes < probe.used()) return BS_EWORKSPACE;
  Carver c(ws, ws_bytes);
  const TeWs w = carve_te(c, bh, io.S, causal, needs_op(io.source));
  uint32_t* amax = (uint32_t*)io.amax;

  {
    ProfScope prof("te_prep", st);
    te_init_kernel<<<1, 64, 0, st>>>(amax, io.counts);
    te_prep_kernel<<<(unsigned)((numel / 4 + 255) / 256), 256, 0, st>>>((const u16*)io.dO, numel, io.scales, w.dOq,
                                                                         amax, io.counts);
    BS_CHECK_LAUNCH();
  }
  {
    const u16* src[4] = {(const u16*)io.V, (const u16*)io.Q, (const u16*)io.K, w.dOq};
    u16* dst[4] = {w.Vt, w.Qt, w.Kt, w.dOt};
    BS_TRY(launch_attn_transpose(src, dst, 4, (int)bh, io.S, (int)Sp, st));
  }
  AttnArgs fa{(const u16*)io.Q, (const u16*)io.K, (const u16*)io.V, io.S, causal, io.scale, w.m, w.l, w.OP,
              w.Vt, (int)Sp};
  BS_TRY(launch_attn_fwd(fa, io.B, io.H, st));
  {
    ProfScope prof("te_d", st);
    te_d_kernel<<<(unsigned)((rows + 63) / 64), 256, 0, st>>>(
        w.dOq, w.OP, io.O, io.O_codes, io.O_scale, w.l, rows, io.source, io.thr, io.seed, io.trial,
        io.store_id * 256u + 1u, io.scales, w.D, io.counts);
    BS_CHECK_LAUNCH();
  }
  TeArgs a{};
  a.Q = (const u16*)io.Q;
  a.K = (const u16*)io.K;
  a.V = (const u16*)io.V;
  a.dO = w.dOq;
  a.Qt = w.Qt;
  a.Kt = w.Kt;
  a.dOt = w.dOt;
  a.S = io.S;
  a.Sp = (int)Sp;
  a.causal = causal;
  a.BH = (int)bh;
  a.scale = io.scale;
  a.m = w.m;
  a.l = w.l;
  a.sc = io.scales;
  a.D = w.D;
  a.dsq = w.dsq;
  a.pq = w.pq;
  a.P_out = io.P_out;
  a.dS_out = io.dS_out;
  a.P_codes = io.P_codes;
  a.dS_codes = io.dS_codes;
  a.pre = io.grad_pre;
  a.dQ = io.dQ;
  a.dK = io.dK;
  a.dV = io.dV;
  a.amax = amax;
  a.counts = io.counts;
  const dim3 grid((unsigned)bh, (unsigned)(Sp / AT));
  {
    ProfScope prof("te_dq", st);
    te_dq_kernel<<<grid, 256, 0, st>>>(a);
    BS_CHECK_LAUNCH();
  }
  {
    ProfScope prof("te_dkv", st);
    te_dkv_kernel<<<grid, 256, 0, st>>>(a);
    BS_CHECK_LAUNCH();
  }
  return BS_OK;
}

}  // namespace bsp

using namespace bsp;

extern "C" {

size_t bs_te_attn_workspace_size(int B, int H, int S, int dh, int causal, bs_d_source source) {
  return te_ws_size(B, H, S, dh, causal, (int)source);
}

bs_status bs_te_attn_bwd(const void* Q, const void* Kt, const void* V, const void* dO, int B, int H, int S, int dh,
                         int causal, float softmax_scale, const float* O, const uint8_t* O_codes, const float* O_scale,
                         bs_d_source source, float threshold, const float* scales, uint64_t seed, uint32_t store_id,
                         uint32_t trial, float* dQ, float* dK, float* dV, float* amax, uint32_t* counts, float* P_out,
                         float* dS_out, uint8_t* P_codes, uint8_t* dS_codes, float* grad_pre, void* ws,
                         size_t ws_bytes, void* stream) {
  TeIO io{Q,      Kt,      V,       dO,          B,         H,      S,    dh,       causal, softmax_scale,
          O,      O_codes, O_scale, (int)source, threshold, scales, seed, store_id, trial,  dQ,
          dK,     dV,      amax,    counts,      P_out,     dS_out, P_codes, dS_codes, grad_pre};
  return te_run(io, ws, ws_bytes, (hipStream_t)stream);
}

}  // extern "C"
