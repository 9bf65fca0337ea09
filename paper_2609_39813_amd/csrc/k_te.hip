// An emulation of an FP8 attention backward with delayed scaling (App. D.2; App. E.3), dh = 64:
// dO cast to E5M2 at its delayed scale; P re-formed and stored in E4M3 at the forward's scale;
// dV = P_q^T dO_q; dP = dO_q V^T; D from the selected source; dS = P (dP - D) cast to E5M2 at its
// delayed scale; dQ = c dS_q K, dK = c dS_q^T Q; dQ, dK and dV cast to E5M2 at the gradients'
// delayed scale. Every cast rounds to nearest even after clamping |x / s| to FMAX (counted). The
// amaxes of dO, of the pre-cast dS and of the pre-cast gradients are reported for the caller's
// histories.
//
// Q, K and V are bf16, or the forward's E4M3 stores at scales s_Q, s_K, s_V (App. D.2: the
// forward recomputes its output from the dequantized FP8 Q, K and V); the returned gradients are
// BF16 (App. D.2) or fp32 values of code times s_g.
//
// Every product has exact bf16 operands (FP8 values and bf16 inputs), one MFMA term each, with
// the scales applied in fp32 after the accumulation (s_Q s_K on the scores, s_V on dP and P V,
// s_K on dQ, s_Q on dK). The query-major pass writes the dS and P codes tile by tile ([key][query],
// one byte each) for the key-major pass.
#include "k_attn.h"
#include "k_qmajor.h"

#include <algorithm>

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
  const float* scale_mul;      // nullable device [1]: s_Q s_K (FP8 operands)
  const float* qkv;            // nullable device [3]: s_Q, s_K, s_V (FP8 operands)
  int grad_bf16;               // returned gradients: bf16 (1) or fp32 (0)
  const float *m, *l;
  const float* sc;             // device [4]: s_P, s_dO, s_dS, s_g
  const float* D;              // [rows] the correction term
  uint8_t *dsq, *pq;           // tile-major codes [BH][tiles][64 key][64 query, in code_pos order]
  float *P_out, *dS_out;       // nullable [BH][S][S]: the realized P and pre-cast dS
  uint8_t *P_codes, *dS_codes; // nullable [BH][S][S]
  float* pre;                  // nullable [3][BH][S][64]: pre-cast dQ, dK, dV
  void *dQ, *dK, *dV;          // returned gradients, bf16 or fp32 (grad_bf16)
  uint32_t *part_dq, *part_dkv; // per-block partials (amaxes as fp32 bits, clamp counts)
};

constexpr float kE5M2Max = 57344.0f, kE4M3Max = 448.0f;
constexpr int TE_BLOCK = 256;  // threads per block of every kernel here

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

// The block's totals of N quantities written to out[0..N-1]: MAX[i] selects the largest (fp32 bits
// of non-negative values order as integers) or the sum. Every thread of the block must call it.
// (Per-block partials instead of atomics on shared counters: those serialize, and the order of
// the final reduction is fixed.)
template <int N>
__device__ __forceinline__ void block_total(const uint32_t (&v)[N], const bool (&MAX)[N], uint32_t* out) {
  __shared__ uint32_t part[N][TE_BLOCK / 64];
  const int w = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const uint32_t r = MAX[i] ? wave_max_u32(v[i]) : wave_sum_u32(v[i]);
    if ((threadIdx.x & 63) == 0) part[i][w] = r;
  }
  __syncthreads();
  if (threadIdx.x < N) {
    const int i = threadIdx.x;
    uint32_t r = part[i][0];
#pragma unroll
    for (int k = 1; k < TE_BLOCK / 64; ++k) r = MAX[i] ? max(r, part[i][k]) : r + part[i][k];
    out[i] = r;
  }
}

// Byte position of tile-local query q in a tile row of the code arrays: 16 (q >> 2 & 3) +
// 8 (q >> 5) + 4 (q >> 4 & 1) + (q & 3), so that the 8 queries 32 s2 + 16 hh + 4 g + r (s2, hh < 2,
// r < 4) a key-major lane reads for group g are the 16 bytes at 16 g.
__device__ __forceinline__ int code_pos(int q) {
  return 16 * ((q >> 2) & 3) + 8 * (q >> 5) + 4 * ((q >> 4) & 1) + (q & 3);
}

// 4 x 4 byte transpose within a quad of lanes: lane j's byte i becomes lane i's byte j (two DPP
// exchanges, with the lane j ^ 2 and then with the lane j ^ 1)
__device__ __forceinline__ uint32_t quad_transpose(uint32_t w, int j) {
  const uint32_t x = (uint32_t)__builtin_amdgcn_mov_dpp((int)w, 0x4E, 0xF, 0xF, false);  // quad_perm 2,3,0,1
  const uint32_t n = (j & 2) ? ((x >> 16) | (w & 0xFFFF0000u)) : ((w & 0x0000FFFFu) | (x << 16));
  const uint32_t y = (uint32_t)__builtin_amdgcn_mov_dpp((int)n, 0xB1, 0xF, 0xF, false);  // quad_perm 1,0,3,2
  return (j & 1) ? (((y >> 8) & 0x00FF00FFu) | (n & 0xFF00FF00u)) : ((n & 0x00FF00FFu) | ((y & 0x00FF00FFu) << 8));
}

__device__ __forceinline__ int block_linear() { return (int)(blockIdx.y * gridDim.x + blockIdx.x); }

// a returned gradient: the fp32 dequantization fl32(val(C) s_g) of its E5M2 code, in BF16 (rounded
// to nearest even) or left in fp32
__device__ __forceinline__ void put_grad(void* out, int64_t e, float v, int as_bf16) {
  if (as_bf16)
    ((u16*)out)[e] = bf16_bits(v);
  else
    ((float*)out)[e] = v;
}

// E4M3 codes of Q, K and V -> their code values as bf16 (exact), 16 per thread and step; block 0
// also writes s_Q s_K (the scores' scale multiplier)
__global__ __launch_bounds__(256) void te_qkv_kernel(const uint8_t* __restrict__ Qc, const uint8_t* __restrict__ Kc,
                                                     const uint8_t* __restrict__ Vc, int64_t n, const float* qkv,
                                                     u16* __restrict__ Qv, u16* __restrict__ Kv, u16* __restrict__ Vv,
                                                     float* qk) {
  if (blockIdx.x == 0 && threadIdx.x == 0) qk[0] = qkv[0] * qkv[1];
  const uint8_t* src[3] = {Qc, Kc, Vc};
  u16* dst[3] = {Qv, Kv, Vv};
  for (int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 16; i < n; i += (int64_t)gridDim.x * 256 * 16) {
#pragma unroll
    for (int t = 0; t < 3; ++t) {
      const uint4 c = *(const uint4*)(src[t] + i);
      const uint32_t cw[4] = {c.x, c.y, c.z, c.w};
      uint32_t o[8];
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        o[2 * h] = (__float_as_uint(f8_val<BS_E4M3>(cw[h], 0)) >> 16) | (__float_as_uint(f8_val<BS_E4M3>(cw[h], 1)) & 0xFFFF0000u);
        o[2 * h + 1] = (__float_as_uint(f8_val<BS_E4M3>(cw[h], 2)) >> 16) | (__float_as_uint(f8_val<BS_E4M3>(cw[h], 3)) & 0xFFFF0000u);
      }
      *(uint4*)(dst[t] + i) = make_uint4(o[0], o[1], o[2], o[3]);
      *(uint4*)(dst[t] + i + 8) = make_uint4(o[4], o[5], o[6], o[7]);
    }
  }
}

// Per-block partials of every kernel: [n][width] words each
struct TeParts {
  uint32_t *prep, *d, *dq, *dkv;  // widths 2 (amax dO, clamps dO), 2 (rows, amax P), 4 (amax dS, clamps
  int n_prep, n_d, n_dq, n_dkv;   // dS, amax gradients, clamps gradients), 2 (amax gradients, clamps)
};

// The call's amaxes and counts from the per-block partials: one block; every thread folds its
// share of each partial array (all nine quantities at once), then one fixed tree over the waves.
__global__ __launch_bounds__(TE_BLOCK) void te_final_kernel(TeParts q, float* amax, uint32_t* counts) {
  // quantities: 0 amax P, 1 amax dO, 2 amax dS, 3 amax gradients (max); 4 rows, 5 clamps dO,
  // 6 clamps dS, 7 clamps gradients (sum)
  uint32_t v[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int i = threadIdx.x; i < q.n_prep; i += TE_BLOCK) {
    v[1] = max(v[1], q.prep[2 * i]);
    v[5] += q.prep[2 * i + 1];
  }
  for (int i = threadIdx.x; i < q.n_d; i += TE_BLOCK) {
    v[4] += q.d[2 * i];
    v[0] = max(v[0], q.d[2 * i + 1]);
  }
  for (int i = threadIdx.x; i < q.n_dq; i += TE_BLOCK) {
    const uint4 w = *(const uint4*)(q.dq + 4 * (int64_t)i);
    v[2] = max(v[2], w.x);
    v[6] += w.y;
    v[3] = max(v[3], w.z);
    v[7] += w.w;
  }
  for (int i = threadIdx.x; i < q.n_dkv; i += TE_BLOCK) {
    v[3] = max(v[3], q.dkv[2 * i]);
    v[7] += q.dkv[2 * i + 1];
  }
  __shared__ uint32_t red[8][TE_BLOCK / 64];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const uint32_t r = k < 4 ? wave_max_u32(v[k]) : wave_sum_u32(v[k]);
    if ((threadIdx.x & 63) == 0) red[k][threadIdx.x >> 6] = r;
  }
  __syncthreads();
  if (threadIdx.x < 8) {
    const int k = threadIdx.x;
    uint32_t r = red[k][0];
    for (int w = 1; w < TE_BLOCK / 64; ++w) r = k < 4 ? max(r, red[k][w]) : r + red[k][w];
    if (k < 4)
      amax[k] = __uint_as_float(r);
    else
      counts[k - 4] = r;
  }
}

// dO -> its E5M2 code values (bf16, exact), 8 elements per thread and step (grid-stride)
__global__ __launch_bounds__(TE_BLOCK) void te_prep_kernel(const u16* __restrict__ dO, int64_t n, const float* sc,
                                                           u16* __restrict__ dOq, uint32_t* part) {
  const double rs = 1.0 / (double)sc[1];
  float am = 0.0f;
  uint32_t nsat = 0;
  for (int64_t i = ((int64_t)blockIdx.x * TE_BLOCK + threadIdx.x) * 8; i < n; i += (int64_t)gridDim.x * TE_BLOCK * 8) {
    const uint4 d4 = *(const uint4*)(dO + i);
    const uint32_t dw[4] = {d4.x, d4.y, d4.z, d4.w};
    uint32_t ow[4];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      float y[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float x = bf16_to_f32((u16)(dw[2 * h + (r >> 1)] >> (16 * (r & 1))));
        am = fmaxf(am, fabsf(x));
        y[r] = div_scale(x, rs);
      }
      uint32_t ns;
      const uint32_t w = codes4<BS_E5M2>(y, ns);
      nsat += ns;
      // the code values are exact in bf16: their fp32 bit patterns' upper halves
      ow[2 * h] = (__float_as_uint(f8_val<BS_E5M2>(w, 0)) >> 16) | (__float_as_uint(f8_val<BS_E5M2>(w, 1)) & 0xFFFF0000u);
      ow[2 * h + 1] = (__float_as_uint(f8_val<BS_E5M2>(w, 2)) >> 16) | (__float_as_uint(f8_val<BS_E5M2>(w, 3)) & 0xFFFF0000u);
    }
    *(uint4*)(dOq + i) = make_uint4(ow[0], ow[1], ow[2], ow[3]);
  }
  const uint32_t v[2] = {__float_as_uint(am), nsat};
  const bool mx[2] = {true, false};
  block_total(v, mx, part + 2 * block_linear());
}

// D per row (4 lanes per row, 16 elements each), in fp64 from exact operands: dO_q against the
// forward's P V (P), the original O (U), the E4M3 store of O (R), a new stochastic rounding of O
// at the store's scale (N), or the repair (P where the row's largest probability, exactly
// fl32(1 / l), reaches the threshold, R elsewhere). Rows at or over the threshold are counted.
__global__ __launch_bounds__(TE_BLOCK) void te_d_kernel(const u16* __restrict__ dOq, const float* __restrict__ OP,
                                                   const float* __restrict__ O, const uint8_t* __restrict__ Oc,
                                                   const float* Os, const float* __restrict__ l, int64_t rows,
                                                   int source, float thr, uint64_t seed, uint32_t trial, uint32_t use,
                                                   const float* sc, const float* qkv, float* __restrict__ D,
                                                   uint32_t* part) {
  const int64_t row = (int64_t)blockIdx.x * 64 + (threadIdx.x >> 2);
  const int sub = threadIdx.x & 3;
  const bool ok = row < rows;
  const F8 f = f8_format(BS_E4M3);
  const float pmax = ok ? 1.0f / l[row] : 0.0f;  // the row's largest probability
  const bool sat = ok && pmax >= thr;
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
  // the forward's P V was formed from V's code values: s_V applies here
  const double sv = (src == BS_D_FROM_P && qkv) ? (double)qkv[2] : 1.0;
  if (ok && sub == 0) D[row] = (float)((double)sc[1] * sv * acc);
  const uint32_t v[2] = {(ok && sub == 0 && sat) ? 1u : 0u, __float_as_uint(pmax)};
  const bool mx[2] = {false, true};
  block_total(v, mx, part + 2 * block_linear());
}

// query-major: dS = P (dP - D), its E5M2 codes at s_dS and P's E4M3 codes at s_P (tile-major),
// dQ = c s_dS val(dS_q) K cast at s_g
__global__ __launch_bounds__(TE_BLOCK) __attribute__((amdgpu_waves_per_eu(3, 8))) void te_dq_kernel(TeArgs a) {
  __shared__ __attribute__((aligned(16))) u16 sm[2][3][AT * AT];  // K, V, K^T
  const QMajor z = qmajor_setup(a, true);
  const float sdS = a.sc[2];
  const float sdO = a.qkv ? a.sc[1] * a.qkv[2] : a.sc[1];  // dP = s_dO (s_V) val(dO_q) V
  const double rP = 1.0 / (double)a.sc[0], rdS = 1.0 / (double)sdS, rg = 1.0 / (double)a.sc[3];
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
        y[r] = div_scale(ds[r], rdS);
        yp[r] = div_scale(p[t][r], rP);
      }
      uint32_t ns, nsp;
      const uint32_t wd = codes4<BS_E5M2>(y, ns), wp = codes4<BS_E4M3>(yp, nsp);
      nsat += ns;
#pragma unroll
      for (int r = 0; r < 4; ++r) dv[t][r] = f8_val<BS_E5M2>(wd, r);
      // after the quad transpose lane j (= c16 & 3) holds key 16 t + 4 g + j at the quad's 4
      // consecutive positions
      const int64_t o = tile + (16 * t + 4 * z.g + (z.c16 & 3)) * AT + code_pos(16 * z.w + (z.c16 & ~3));
      *(uint32_t*)(a.dsq + o) = quad_transpose(wd, z.c16 & 3);
      *(uint32_t*)(a.pq + o) = quad_transpose(wp, z.c16 & 3);
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
  // dQ = c (s_K) s_dS acc, cast at the gradients' scale
  const float cs = (a.qkv ? a.scale * a.qkv[1] : a.scale) * sdS;
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
      y[n] = div_scale(pre[n], rg);
      amg = fmaxf(amg, fabsf(pre[n]));
    }
    uint32_t ns;
    const uint32_t w = codes4<BS_E5M2>(y, ns);
    nsg += ns;
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const int64_t e = z.hb + (int64_t)qr * AT + 16 * n + z.c16;
      put_grad(a.dQ, e, f8_val<BS_E5M2>(w, n) * a.sc[3], a.grad_bf16);
      if (a.pre) a.pre[e] = pre[n];
    }
  }
  const uint32_t v[4] = {__float_as_uint(amds), nsat, __float_as_uint(amg), nsg};
  const bool mx[4] = {true, false, true, false};
  block_total(v, mx, a.part_dq + 4 * block_linear());
}

// key-major: dK = c s_dS sum_q val(dS_q) Q, dV = s_P s_dO sum_q val(P_q) val(dO_q), both cast at s_g
__global__ __launch_bounds__(TE_BLOCK) void te_dkv_kernel(TeArgs a) {
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
  // the lane's key's codes of one query block: bytes 16 g .. 16 g + 15 of its tile row (queries
  // 32 s2 + 16 hh + 4 g + r at byte 8 s2 + 4 hh + r), loaded one step ahead of their use
  auto load_codes = [&](int qb_, uint4& d, uint4& p) {
    const int64_t o = fld_tile(a, bh, qb_, kb, nqb) + (int64_t)(16 * w + c16) * AT + 16 * g;
    d = *(const uint4*)(a.dsq + o);
    p = *(const uint4*)(a.pq + o);
  };
  const int qb0 = a.causal ? kb : 0;
  uint4 cd, cp;
  load_codes(qb0, cd, cp);
  fetch(qb0 * AT);
  put(0);
  __syncthreads();
  for (int qb = qb0; qb < nqb; ++qb) {
    const int st = (qb - qb0) & 1, q0 = qb * AT;
    if (qb + 1 < nqb) fetch(q0 + AT);
    uint4 nd = make_uint4(0, 0, 0, 0), np = make_uint4(0, 0, 0, 0);
    if (qb + 1 < nqb) load_codes(qb + 1, nd, np);
    const uint32_t dwd[4] = {cd.x, cd.y, cd.z, cd.w}, dwp[4] = {cp.x, cp.y, cp.z, cp.w};
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      // queries 32 s2 + 16 hh + 4 g + (0..3) of this lane's key, as the k index of the products
      float dsv[8], pv[8];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const uint32_t wd = dwd[2 * s2 + hh], wp = dwp[2 * s2 + hh];
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
    cd = nd;
    cp = np;
    if (qb + 1 < nqb) put(st ^ 1);
    __syncthreads();
  }
  const float ck = (a.qkv ? a.scale * a.qkv[0] : a.scale) * sdS, cv = sP * sdO;  // dK: c (s_Q) s_dS
  const double rg = 1.0 / (double)sg;
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
      yk[n] = div_scale(prk[n], rg);
      yv[n] = div_scale(prv[n], rg);
      amg = fmaxf(amg, fmaxf(fabsf(prk[n]), fabsf(prv[n])));
    }
    uint32_t nk, nv;
    const uint32_t wk = codes4<BS_E5M2>(yk, nk), wv = codes4<BS_E5M2>(yv, nv);
    nsg += nk + nv;
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const int64_t e = hb + (int64_t)kr * AT + 16 * n + c16;
      put_grad(a.dK, e, f8_val<BS_E5M2>(wk, n) * sg, a.grad_bf16);
      put_grad(a.dV, e, f8_val<BS_E5M2>(wv, n) * sg, a.grad_bf16);
      if (a.pre) {
        a.pre[numel + e] = prk[n];
        a.pre[2 * numel + e] = prv[n];
      }
    }
  }
  const uint32_t v[2] = {__float_as_uint(amg), nsg};
  const bool mx[2] = {true, false};
  block_total(v, mx, a.part_dkv + 2 * block_linear());
}

constexpr int TE_PREP_BLOCKS = 256;  // grid-stride cast of dO: few blocks, few partials

// One step of delayed scaling for the four tensors of the call (P in E4M3; dO, dS and the
// gradients in E5M2): the step's amax enters the ring history at step % len, and the scale for
// the next step is the largest amax in the history divided by FMAX (fl32), kept unchanged when
// that largest amax is zero or not finite. Block i serves tensor i.
__global__ __launch_bounds__(TE_BLOCK) void te_scales_kernel(const float* amax, float* history, int len, int pos,
                                                             float* scales) {
  __shared__ uint32_t red[TE_BLOCK / 64];
  const int i = blockIdx.x;
  const float a = amax[i];
  float* h = history + (int64_t)i * len;
  // non-negative finite amaxes order as their bits; a NaN (or infinite) one wins the max as well
  uint32_t m = threadIdx.x == 0 ? __float_as_uint(fabsf(a)) : 0u;
  for (int j = threadIdx.x; j < len; j += TE_BLOCK)
    if (j != pos) m = max(m, __float_as_uint(fabsf(h[j])));
  m = wave_max_u32(m);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int k = 1; k < TE_BLOCK / 64; ++k) m = max(m, red[k]);
    h[pos] = a;
    const float am = __uint_as_float(m);
    const float fm = i == 0 ? kE4M3Max : kE5M2Max;
    if (am > 0.0f && am <= 3.402823466e38f) scales[i] = am / fm;
  }
}

struct TeWs {
  u16 *dOq, *Qt, *Kt, *Vt, *dOt;
  u16 *Qv, *Kv, *Vv;  // FP8 operands: the code values as bf16
  float* qk;          // FP8 operands: s_Q s_K
  float *m, *l, *D, *OP;
  uint8_t *dsq, *pq;
  TeParts parts;
};

int prep_blocks(int64_t numel) {
  return (int)std::min<int64_t>((numel / 8 + TE_BLOCK - 1) / TE_BLOCK, TE_PREP_BLOCKS);
}

TeWs carve_te(Carver& c, int64_t bh, int S, int causal, bool need_op, bool fp8_qkv) {
  TeWs w{};
  const int64_t Sp = round_up(S, AT), rows = bh * S;
  const int nqb = (int)(Sp / AT);
  w.parts.n_prep = prep_blocks(rows * AT);
  w.parts.n_d = (int)((rows + 63) / 64);
  w.parts.n_dq = w.parts.n_dkv = (int)(bh * nqb);
  w.parts.prep = c.take<uint32_t>(2 * (int64_t)w.parts.n_prep);
  w.parts.d = c.take<uint32_t>(2 * (int64_t)w.parts.n_d);
  w.parts.dq = c.take<uint32_t>(4 * (int64_t)w.parts.n_dq);
  w.parts.dkv = c.take<uint32_t>(2 * (int64_t)w.parts.n_dkv);
  w.dOq = c.take<u16>(rows * AT);
  for (u16** p : {&w.Qt, &w.Kt, &w.Vt, &w.dOt}) *p = c.take<u16>(bh * AT * Sp);
  for (float** p : {&w.m, &w.l, &w.D}) *p = c.take<float>(rows);
  if (need_op) w.OP = c.take<float>(rows * AT);
  const int64_t nt = bh * causal_tiles(nqb, causal) * AT * AT;
  w.dsq = c.take<uint8_t>(nt);
  w.pq = c.take<uint8_t>(nt);
  if (fp8_qkv) {
    for (u16** p : {&w.Qv, &w.Kv, &w.Vv}) *p = c.take<u16>(rows * AT);
    w.qk = c.take<float>(1);
  }
  return w;
}

bool needs_op(int source) { return source == BS_D_FROM_P || source == BS_D_REPAIR; }

}  // namespace

struct TeIO {
  const void *Q, *K, *V, *dO;
  int B, H, S, dh, causal;
  float scale;
  const float* qkv_scales;  // nullable: Q, K, V are E4M3 codes at these scales
  const float* O;
  const uint8_t* O_codes;
  const float* O_scale;
  int source;
  float thr;
  const float* scales;
  uint64_t seed;
  uint32_t store_id, trial;
  int grad_type;
  void *dQ, *dK, *dV;
  float* amax;
  uint32_t* counts;
  float *P_out, *dS_out;
  uint8_t *P_codes, *dS_codes;
  float* grad_pre;
};

size_t te_ws_size(int B, int H, int S, int dh, int causal, int source, int fp8_qkv) {
  if (B < 1 || H < 1 || S < 1 || dh != AT || source < BS_D_FROM_P || source > BS_D_REPAIR) return 0;
  Carver c;
  carve_te(c, (int64_t)B * H, S, causal ? 1 : 0, needs_op(source), fp8_qkv != 0);
  return c.used();
}

bs_status te_run(const TeIO& io, void* ws, size_t ws_bytes, hipStream_t st) {
  if (!io.Q || !io.K || !io.V || !io.dO || !io.scales || !io.dQ || !io.dK || !io.dV || !io.amax || !io.counts)
    return BS_EINVAL;
  if (io.B < 1 || io.H < 1 || io.S < 1 || !(io.scale > 0.0f)) return BS_EINVAL;
  if (io.source < BS_D_FROM_P || io.source > BS_D_REPAIR) return BS_EINVAL;
  if (io.grad_type != BS_F32 && io.grad_type != BS_BF16) return BS_EDTYPE;
  const bool need_codes = io.source == BS_D_R || io.source == BS_D_REPAIR;
  if ((need_codes && !io.O_codes) || ((need_codes || io.source == BS_D_N) && !io.O_scale)) return BS_EINVAL;
  if ((io.source == BS_D_U || io.source == BS_D_N) && !io.O) return BS_EINVAL;
  if (io.dh != AT || io.S % 4 != 0) return BS_ESHAPE;
  if ((int64_t)io.B * io.H > 65535 || (io.S + AT - 1) / AT > 65535) return BS_ESHAPE;
  for (const void* p : {io.Q, io.K, io.V, io.dO, (const void*)io.O, (const void*)io.P_out, (const void*)io.dS_out})
    if ((uintptr_t)p & 15) return BS_EINVAL;  // 16-byte vector loads and stores
  if ((uintptr_t)io.qkv_scales & 3) return BS_EINVAL;
  for (const void* p : {(const void*)io.O_codes, (const void*)io.P_codes, (const void*)io.dS_codes})
    if ((uintptr_t)p & 3) return BS_EINVAL;
  const int64_t bh = (int64_t)io.B * io.H, Sp = round_up(io.S, AT), rows = bh * io.S, numel = rows * AT;
  const int causal = io.causal ? 1 : 0;
  const bool fq = io.qkv_scales != nullptr;
  Carver probe;
  carve_te(probe, bh, io.S, causal, needs_op(io.source), fq);
  if (!ws || ((uintptr_t)ws & 255) || ws_bytes < probe.used()) return BS_EWORKSPACE;
  Carver c(ws, ws_bytes);
  const TeWs w = carve_te(c, bh, io.S, causal, needs_op(io.source), fq);
  // the operands: bf16 inputs, or the FP8 stores' code values (exact in bf16)
  const u16* Qo = fq ? w.Qv : (const u16*)io.Q;
  const u16* Ko = fq ? w.Kv : (const u16*)io.K;
  const u16* Vo = fq ? w.Vv : (const u16*)io.V;
  if (fq) {
    te_qkv_kernel<<<prep_blocks(numel / 2), 256, 0, st>>>((const uint8_t*)io.Q, (const uint8_t*)io.K,
                                                         (const uint8_t*)io.V, numel, io.qkv_scales, w.Qv, w.Kv,
                                                         w.Vv, w.qk);
    BS_CHECK_LAUNCH();
  }

  {
    ProfScope prof("te_prep", st);
    te_prep_kernel<<<(unsigned)w.parts.n_prep, TE_BLOCK, 0, st>>>((const u16*)io.dO, numel, io.scales, w.dOq,
                                                                  w.parts.prep);
    BS_CHECK_LAUNCH();
  }
  {
    const u16* src[4] = {Vo, Qo, Ko, w.dOq};
    u16* dst[4] = {w.Vt, w.Qt, w.Kt, w.dOt};
    BS_TRY(launch_attn_transpose(src, dst, 4, (int)bh, io.S, (int)Sp, st));
  }
  AttnArgs fa{Qo, Ko, Vo, io.S, causal, io.scale, w.m, w.l, w.OP, w.Vt, (int)Sp, fq ? w.qk : nullptr};
  BS_TRY(launch_attn_fwd(fa, io.B, io.H, st));
  {
    ProfScope prof("te_d", st);
    te_d_kernel<<<(unsigned)((rows + 63) / 64), TE_BLOCK, 0, st>>>(
        w.dOq, w.OP, io.O, io.O_codes, io.O_scale, w.l, rows, io.source, io.thr, io.seed, io.trial,
        io.store_id * 256u + 1u, io.scales, io.qkv_scales, w.D, w.parts.d);
    BS_CHECK_LAUNCH();
  }
  TeArgs a{};
  a.Q = Qo;
  a.K = Ko;
  a.V = Vo;
  a.dO = w.dOq;
  a.Qt = w.Qt;
  a.Kt = w.Kt;
  a.dOt = w.dOt;
  a.S = io.S;
  a.Sp = (int)Sp;
  a.causal = causal;
  a.BH = (int)bh;
  a.scale = io.scale;
  a.scale_mul = fq ? w.qk : nullptr;
  a.qkv = io.qkv_scales;
  a.grad_bf16 = io.grad_type == BS_BF16 ? 1 : 0;
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
  a.part_dq = w.parts.dq;
  a.part_dkv = w.parts.dkv;
  const dim3 grid((unsigned)bh, (unsigned)(Sp / AT));
  {
    ProfScope prof("te_dq", st);
    te_dq_kernel<<<grid, TE_BLOCK, 0, st>>>(a);
    BS_CHECK_LAUNCH();
  }
  {
    ProfScope prof("te_dkv", st);
    te_dkv_kernel<<<grid, TE_BLOCK, 0, st>>>(a);
    BS_CHECK_LAUNCH();
  }
  te_final_kernel<<<1, TE_BLOCK, 0, st>>>(w.parts, io.amax, io.counts);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

}  // namespace bsp

using namespace bsp;

extern "C" {

size_t bs_te_attn_workspace_size(int B, int H, int S, int dh, int causal, bs_d_source source, int fp8_qkv) {
  return te_ws_size(B, H, S, dh, causal, (int)source, fp8_qkv);
}

bs_status bs_te_delayed_scales(const float* amax, float* history, int len, int64_t step, float* scales,
                               void* stream) {
  if (!amax || !history || !scales || len < 1 || step < 0) return BS_EINVAL;
  te_scales_kernel<<<4, TE_BLOCK, 0, (hipStream_t)stream>>>(amax, history, len, (int)(step % len), scales);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status bs_te_attn_bwd(const void* Q, const void* Kt, const void* V, const float* qkv_scales, const void* dO, int B,
                         int H, int S, int dh, int causal, float softmax_scale, const float* O, const uint8_t* O_codes,
                         const float* O_scale, bs_d_source source, float threshold, const float* scales, uint64_t seed,
                         uint32_t store_id, uint32_t trial, bs_dtype grad_type, void* dQ, void* dK, void* dV,
                         float* amax, uint32_t* counts, float* P_out, float* dS_out, uint8_t* P_codes,
                         uint8_t* dS_codes, float* grad_pre, void* ws, size_t ws_bytes, void* stream) {
  TeIO io{Q,       Kt,      V,         dO,     B,        H,     S,          dh,   causal, softmax_scale,
          qkv_scales, O,    O_codes,   O_scale, (int)source, threshold, scales, seed, store_id, trial,
          (int)grad_type, dQ, dK,      dV,     amax,     counts, P_out,     dS_out, P_codes, dS_codes,
          grad_pre};
  return te_run(io, ws, ws_bytes, (hipStream_t)stream);
}

}  // extern "C"
