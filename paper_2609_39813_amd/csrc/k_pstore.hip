// The FP8 store of attention probabilities (gfx950, dh = 64) and the per-use estimates of its
// two uses: the gradient of V reads p, p_q or a new rounding a; the softmax's backward reads
// J(p), J(p_q), J(a), K(a), J2(a, b) or J2(p_q, a) (App. B.2-B.4).
//
// Every pass recomputes its 64 x 64 tiles of scores the same way, so that P is bit-identical in
// all of them: with m the row max of x = fl(c log2(e) S) (fl: rounded, never contracted into an
// FMA), p = 2^(x - m) / l. The largest probability of a row is then exactly 1 / l, and the
// store's amax is the largest 1 / l. Query-major passes (forward, row sums, dQ) hold in each lane
// one query and 16 keys: the lane's scores are an MFMA result tile of K Q^T (keys on the tile's
// rows), and the products with K and V take them as register operands (k-step order as in the
// attention backward). The key-major pass (dK, dV) reads the bias fields the dQ pass stored.
//
// Collapsed trials. With r = p_q - p, a new rounding a_k = p + e + u_k h (e = lo - p, h the grid
// step, u_k its up-decision) and a row's D = p . dp, each policy's mean over the K trials of
// Jhat dp - J(p) dp is a combination of per-row sums (Ga_k = sum u_k h dp, Ha_k = sum u_k h,
// ...) and per-element sums over trials (n = sum u_k, sum u_k Ga_k, ...): the trials never
// materialize, and the dQ / dK contractions run once per field. The row-sum pass draws each
// up-decision once (one Philox call per 4 elements, trial and use) and leaves them as bits for
// the dQ pass.
#include "k_pstore.h"
#include "k_qmajor.h"

namespace bsp {

namespace {

// residuals of one element: r = p_q - p, e = lo - p, h = step (real units), F = SR threshold
struct Resid {
  float r, e, h;
  uint32_t F;
};
__device__ __forceinline__ Resid resid(float p, float val, float s, double rs, F8 f) {
  Resid o;
  const float y = fminf(div_scale(p, rs), f.fmax);
  const Bracket b = f8_bracket(y, f);
  const float step = f8_step(b);
  o.r = fmaf(s, val, -p);
  o.e = fmaf(s, (float)b.mi * step, -p);
  o.h = s * step;
  o.F = b.F;
  return o;
}

// one output element of every policy: mean = ref + bias[field], bias = bias[field] (b[0] = 0
// for a read that is the reference's own)
template <int NF>
__device__ __forceinline__ void write_policies(const PstoreArgs& a, const int (&field)[PSTORE_MAXPOL],
                                               const PstoreOut& o, int64_t e, float ref, const float (&b)[NF]) {
#pragma unroll
  for (int i = 0; i < PSTORE_MAXPOL; ++i) {
    if (i >= a.n_pol) break;
    const int fi = field[i];
    float bi = 0.0f;
#pragma unroll
    for (int j = 1; j < NF; ++j) bi = fi == j ? b[j] : bi;
    if (o.mean[i]) o.mean[i][e] = fi ? ref + bi : ref;
    if (o.bias[i]) o.bias[i][e] = bi;
  }
}

}  // namespace

// ------------------------------------------------------------------------------------
// the store's scale: amax = max over rows of 1 / l, s = fl32(amax / FMAX)
// ------------------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void pstore_scale_kernel(const float* __restrict__ l, int64_t rows, float fmax,
                                                            bs_diag* __restrict__ diag, float* __restrict__ scale_out) {
  // the largest probability of a row is fl32(1 / l); correctly rounded reciprocals are monotone,
  // so the largest over rows is fl32(1 / min l) (rows with a bad sum are flagged, not counted)
  float mn = INFINITY;
  bool bad = false;
  auto take = [&](float v) {
    const bool ok = v > 0.0f && isfinite(v);
    bad |= !ok;
    mn = ok ? fminf(mn, v) : mn;
  };
  const int64_t n4 = ((uintptr_t)l & 15) == 0 ? rows / 4 : 0;
  for (int64_t i = threadIdx.x; i < n4; i += blockDim.x) {
    const float4 v = ((const float4*)l)[i];
    take(v.x);
    take(v.y);
    take(v.z);
    take(v.w);
  }
  for (int64_t i = 4 * n4 + threadIdx.x; i < rows; i += blockDim.x) take(l[i]);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mn = fminf(mn, __shfl_xor(mn, off, 64));
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __shared__ float red[16];
  __shared__ int anybad;
  if (threadIdx.x == 0) anybad = 0;
  __syncthreads();
  if (bad) anybad = 1;
  if (lane == 0) red[w] = mn;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int k = 1; k < (int)(blockDim.x >> 6); ++k) mn = fminf(mn, red[k]);
    const float amax = isfinite(mn) ? 1.0f / mn : 0.0f;
    diag->amax = amax;
    diag->nonfinite = anybad ? 1u : 0u;
    diag->n_saturated = 0;
    const float sc = (anybad || !(amax > 0.0f)) ? 1.0f : __fdiv_rn(amax, fmax);
    diag->scale = sc;
    if (scale_out) *scale_out = sc;
  }
}

// ------------------------------------------------------------------------------------
// forward: codes of P (RNE or SR), P_out, O = s val(C) V (val(C) exact in bf16, one MFMA term)
// ------------------------------------------------------------------------------------
template <int FMT>
__global__ __launch_bounds__(256, 2) void pstore_fwd_kernel(PstoreArgs a) {
  __shared__ __attribute__((aligned(16))) u16 sm[2][2][AT * AT];  // K, V^T
  if (a.diag->nonfinite) return;
  const QMajor z = qmajor_setup(a, false);
  const float s = a.diag->scale;
  const double rs = 1.0 / (double)s;
  const F8 f = a.f;
  const float min_normal = __uint_as_float((uint32_t)(128 - f.bias) << 23);
  floatx4 acc[4];
#pragma unroll
  for (int n = 0; n < 4; ++n) acc[n] = floatx4{0.f, 0.f, 0.f, 0.f};
  TileRegs pf[2];
  auto fetch = [&](int k0) {
    tile_fetch(pf[0], a.K + z.hb, k0, a.S);
    tile_fetch_t(pf[1], a.Vt + z.tb, k0, a.Sp);
  };
  auto put = [&](int st) {
    tile_put(sm[st][0], pf[0]);
    tile_put_t(sm[st][1], pf[1]);
  };
  const int nkb_all = (a.S + AT - 1) / AT;
  const int nkb = a.causal ? z.qb + 1 : nkb_all;
  uint32_t nsat = 0;
  fetch(0);
  put(0);
  __syncthreads();
  for (int kb = 0; kb < nkb; ++kb) {
    const int st = kb & 1, k0 = kb * AT;
    if (kb + 1 < nkb) fetch(k0 + AT);
    float p[4][4];
    probs(a, z, sm[st][0], k0, p);
    float val[4][4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int key = k0 + 16 * t + 4 * z.g;
      float y[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float yy = div_scale(p[t][r], rs);
        nsat += yy > f.fmax ? 1u : 0u;
        y[r] = fminf(yy, f.fmax);
      }
      uint32_t w;
      if (a.fwd_mode == BS_SR) {
        const Philox4 ph = philox_group(a.seed, pelem(a, z, key) >> 2, 0, a.use_fwd);
        const uint32_t R[4] = {ph.w0, ph.w1, ph.w2, ph.w3};
        w = FMT == BS_E5M2 ? (uint32_t)__builtin_amdgcn_cvt_sr_bf8_f32(y[0], (int)R[0], 0, 0)
                           : (uint32_t)__builtin_amdgcn_cvt_sr_fp8_f32(y[0], (int)R[0], 0, 0);
        w = FMT == BS_E5M2 ? (uint32_t)__builtin_amdgcn_cvt_sr_bf8_f32(y[1], (int)R[1], (int)w, 1)
                           : (uint32_t)__builtin_amdgcn_cvt_sr_fp8_f32(y[1], (int)R[1], (int)w, 1);
        w = FMT == BS_E5M2 ? (uint32_t)__builtin_amdgcn_cvt_sr_bf8_f32(y[2], (int)R[2], (int)w, 2)
                           : (uint32_t)__builtin_amdgcn_cvt_sr_fp8_f32(y[2], (int)R[2], (int)w, 2);
        w = FMT == BS_E5M2 ? (uint32_t)__builtin_amdgcn_cvt_sr_bf8_f32(y[3], (int)R[3], (int)w, 3)
                           : (uint32_t)__builtin_amdgcn_cvt_sr_fp8_f32(y[3], (int)R[3], (int)w, 3);
        // below the smallest normal magnitude the instruction does not resolve F to 32 bits
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (y[r] < min_normal && y[r] != 0.0f) {
            const Bracket b = f8_bracket(y[r], f);
            w = (w & ~(0xFFu << (8 * r))) | ((b.base + b.mi + sr_up(b.F, R[r])) << (8 * r));
          }
      } else {
        w = FMT == BS_E5M2 ? (uint32_t)__builtin_amdgcn_cvt_pk_bf8_f32(y[0], y[1], 0, false)
                           : (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(y[0], y[1], 0, false);
        w = FMT == BS_E5M2 ? (uint32_t)__builtin_amdgcn_cvt_pk_bf8_f32(y[2], y[3], (int)w, true)
                           : (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(y[2], y[3], (int)w, true);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) val[t][r] = f8_val<FMT>(w, r);
      if (z.qok && key < a.S) {
        const int64_t e = (int64_t)pelem(a, z, key);
        *(uint32_t*)(a.codes + e) = w;
        if (a.P_out) *(float4*)(a.P_out + e) = make_float4(p[t][0], p[t][1], p[t][2], p[t][3]);
      }
    }
    // O += val(C) V^T (k-step s takes keys 32 s + 16 (v >> 2) + 4 g + (v & 3))
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      uint32_t pk[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int v = 2 * i;
        pk[i] = pk_bf16(val[2 * s2 + (v >> 2)][v & 3], val[2 * s2 + ((v + 1) >> 2)][(v + 1) & 3]);
      }
      const bf16x8 tv = __builtin_bit_cast(bf16x8, make_uint4(pk[0], pk[1], pk[2], pk[3]));
#pragma unroll
      for (int n = 0; n < 4; ++n) acc[n] = mfma(tv, frag_t(sm[st][1], 16 * n + z.c16, s2, z.g), acc[n]);
    }
    if (kb + 1 < nkb) put(st ^ 1);
    __syncthreads();
  }
  // zero codes (and probabilities) above the causal diagonal
  if (z.qok) {
    for (int kb = nkb; kb < nkb_all; ++kb)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int key = kb * AT + 16 * t + 4 * z.g;
        if (key < a.S) {
          const int64_t e = (int64_t)pelem(a, z, key);
          *(uint32_t*)(a.codes + e) = 0u;
          if (a.P_out) *(float4*)(a.P_out + e) = make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
  }
  nsat = wave_sum_u32(nsat);
  if ((threadIdx.x & 63) == 0 && nsat) atomicAdd(&a.diag->n_saturated, nsat);
  // O rows 16 w + 4 g + r, columns 16 n + c16
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int qr = z.q0 + 16 * z.w + 4 * z.g + r;
    if (qr >= a.S) continue;
#pragma unroll
    for (int n = 0; n < 4; ++n) a.O[z.hb + (int64_t)qr * AT + 16 * n + z.c16] = s * acc[n][r];
  }
}

// ------------------------------------------------------------------------------------
// row sums (per query) over keys: D, DR, E, Ee, Ps1 (fp64), and per trial Ga, Ha, Gb (fp32),
// and the up-decision words. The key blocks are walked once per chunk of RC trials; the first
// walk also forms the trial-independent sums. Within a tile the trial loop is outermost: the
// 4 groups x 2 uses of Philox calls of one trial are independent, and each thread's per-trial
// partial sums live in its own LDS slots (added in key-block order, so the result is fixed).
// ------------------------------------------------------------------------------------
constexpr int RC = PSTORE_RC;
template <int FMT, int DRAW>  // DRAW: 0 no new rounding is read, 1 only a, 2 a and b
__global__ __launch_bounds__(256, 2) void pstore_rows_kernel(PstoreArgs a) {
  __shared__ __attribute__((aligned(16))) u16 sm[2][2][AT * AT];  // K, V
  __shared__ float acc[3][RC][256];                                // per thread: Ga, Ha, Gb per trial
  if (a.diag->nonfinite) return;
  const QMajor z = qmajor_setup(a, true);
  const float s = a.diag->scale;
  const double rs = 1.0 / (double)s;
  const F8 f = a.f;
  const int tid = threadIdx.x;
  const int64_t row = z.rb + z.q, rows = (int64_t)a.BH * a.S;
  double sD = 0.0, sDR = 0.0, sE = 0.0, sEe = 0.0, sP = 0.0;
  TileRegs pf[2];
  auto fetch = [&](int k0) {
    tile_fetch(pf[0], a.K + z.hb, k0, a.S);
    tile_fetch(pf[1], a.V + z.hb, k0, a.S);
  };
  auto put = [&](int st) {
    tile_put(sm[st][0], pf[0]);
    tile_put(sm[st][1], pf[1]);
  };
  auto red32 = [](float v) { v += __shfl_xor(v, 16, 64); return v + __shfl_xor(v, 32, 64); };
  const int nqb = (a.S + AT - 1) / AT;
  const int nkb = a.causal ? z.qb + 1 : nqb;
  const int64_t plane = (int64_t)a.BH * pstore_tiles(nqb, a.causal) * AT * AT;
  for (int k0t = 0; k0t < a.ntrial; k0t += RC) {
    const int jn = min(RC, a.ntrial - k0t);
    uint32_t* bits = a.ubits + (k0t / RC) * plane;
#pragma unroll
    for (int i = 0; i < 3; ++i)
#pragma unroll
      for (int j = 0; j < RC; ++j) acc[i][j][tid] = 0.0f;
    fetch(0);
    put(0);
    __syncthreads();
    for (int kb = 0; kb < nkb; ++kb) {
      const int st = kb & 1, k0 = kb * AT;
      if (kb + 1 < nkb) fetch(k0 + AT);
      float p[4][4], dp[4][4];
      probs(a, z, sm[st][0], k0, p);
      dprobs(z, sm[st][1], dp);
      float hh[4][4], hd[4][4];
      // per element: the decisions of this chunk's trials, two bits per trial shifted in from
      // the bottom (a, then b), so that trial j of jn ends at bits 2 (jn - 1 - j) + 1 (a) and
      // 2 (jn - 1 - j) (b)
      uint32_t FF[4][4], ub[4][4];
      uint64_t grp[4];
      bool need[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int key = k0 + 16 * t + 4 * z.g;
        const bool ok = z.qok && key < a.S;
        const uint32_t cw = ok ? *(const uint32_t*)(a.codes + pelem(a, z, key)) : 0u;
        uint32_t any = 0u;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const Resid x = resid(p[t][r], f8_val<FMT>(cw, r), s, rs, f);
          if (k0t == 0) {
            sD += (double)p[t][r] * dp[t][r];
            sDR += (double)x.r * dp[t][r];
            sE += (double)x.e * dp[t][r];
            sEe += (double)x.e;
            sP += (double)p[t][r];
          }
          hh[t][r] = x.h;
          hd[t][r] = x.h * dp[t][r];
          FF[t][r] = x.F;
          ub[t][r] = 0u;
          any |= x.F;
        }
        grp[t] = pelem(a, z, key) >> 2;
        // a group with no fraction (on the grid, masked, past S) never rounds up; a tile
        // with no such group in the whole wave skips the draws
        need[t] = __ballot(any != 0u) != 0ull;
      }
      if (DRAW >= 1 && (need[0] || need[1] || need[2] || need[3])) {
        for (int j = 0; j < jn; ++j) {
          const uint32_t trial = (uint32_t)(k0t + j + 1);
          float gaj = 0.0f, haj = 0.0f, gbj = 0.0f;
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const Philox4 pa = philox_group(a.seed, grp[t], trial, a.use_a);
            const uint32_t Ra[4] = {pa.w0, pa.w1, pa.w2, pa.w3};
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const uint32_t u = sr_up(FF[t][r], Ra[r]);
              ub[t][r] = ub[t][r] + ub[t][r] + u;
              const float uf = u ? 1.0f : 0.0f;
              gaj = fmaf(uf, hd[t][r], gaj);
              haj = fmaf(uf, hh[t][r], haj);
            }
            if (DRAW == 2) {
              const Philox4 pb = philox_group(a.seed, grp[t], trial, a.use_b);
              const uint32_t Rb[4] = {pb.w0, pb.w1, pb.w2, pb.w3};
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                const uint32_t u = sr_up(FF[t][r], Rb[r]);
                ub[t][r] = ub[t][r] + ub[t][r] + u;
                gbj += u ? hd[t][r] : 0.0f;
              }
            } else {
#pragma unroll
              for (int r = 0; r < 4; ++r) ub[t][r] += ub[t][r];
            }
          }
          acc[0][j][tid] += gaj;
          acc[1][j][tid] += haj;
          if (DRAW == 2) acc[2][j][tid] += gbj;
        }
      }
      // the thread's 16 decision words of this tile are contiguous (the dQ pass reads them alike)
      uint4* T = (uint4*)(bits + fld_tile(a, z.bh, z.qb, kb, nqb) + (int64_t)tid * 16);
#pragma unroll
      for (int t = 0; t < 4; ++t) T[t] = make_uint4(ub[t][0], ub[t][1], ub[t][2], ub[t][3]);
      if (kb + 1 < nkb) put(st ^ 1);
      __syncthreads();
    }
    // the four lane groups of a query column hold its four key quarters
    for (int j = 0; j < jn; ++j) {
      const float ga = red32(acc[0][j][tid]), ha = red32(acc[1][j][tid]), gb = red32(acc[2][j][tid]);
      if (z.g == 0 && z.qok) {
        const int k = k0t + j;
        a.Ga[k * rows + row] = ga;
        a.Ha[k * rows + row] = ha;
        a.Gb[k * rows + row] = gb;
      }
    }
    __syncthreads();
  }
  auto red64 = [](double v) { v += __shfl_xor(v, 16, 64); return v + __shfl_xor(v, 32, 64); };
  sD = red64(sD);
  sDR = red64(sDR);
  sE = red64(sE);
  sEe = red64(sEe);
  sP = red64(sP);
  if (z.g == 0 && z.qok) {
    a.D[row] = (float)sD;
    a.DR[row] = (float)sDR;
    a.E[row] = (float)sE;
    a.Ee[row] = (float)sEe;
    a.Ps1[row] = (float)(sP - 1.0);
  }
}

// ------------------------------------------------------------------------------------
// bias fields and dQ: per element the sums over trials, then the fields of every read; the
// fields go to memory for the key-major pass and into dQ = c sum_k field K (three bf16 terms)
// ------------------------------------------------------------------------------------
template <int FMT>
__global__ __launch_bounds__(256) void pstore_dq_kernel(PstoreArgs a) {
  __shared__ __attribute__((aligned(16))) u16 sm[2][3][AT * AT];  // K, V, K^T
  __shared__ float tv[3][AT][PSTORE_KMAX + 1];                     // Ga, Ha, Gb of the block's queries
  if (a.diag->nonfinite) return;
  const QMajor z = qmajor_setup(a, true);
  const float s = a.diag->scale;
  const double rs = 1.0 / (double)s;
  const F8 f = a.f;
  const int64_t row = z.rb + z.q, rows = (int64_t)a.BH * a.S;
  // this lane's query: row sums; the block's per-trial sums in LDS
  const float D = z.qok ? a.D[row] : 0.f, DR = z.qok ? a.DR[row] : 0.f, E = z.qok ? a.E[row] : 0.f;
  const float Ee = z.qok ? a.Ee[row] : 0.f, Ps = z.qok ? 1.0f + a.Ps1[row] : 0.f;
  const float Ps1 = z.qok ? a.Ps1[row] : 0.f;
  for (int i = threadIdx.x; i < AT * a.ntrial; i += blockDim.x) {
    const int qq = i / a.ntrial, k = i - qq * a.ntrial;
    const bool ok = z.q0 + qq < a.S;
    const int64_t rr = z.rb + z.q0 + qq;
    tv[0][qq][k] = ok ? a.Ga[k * rows + rr] : 0.f;
    tv[1][qq][k] = ok ? a.Ha[k * rows + rr] : 0.f;
    tv[2][qq][k] = ok ? a.Gb[k * rows + rr] : 0.f;
  }
  __syncthreads();
  const int ql = 16 * z.w + z.c16;
  float mGa = 0.f, mHa = 0.f, mGb = 0.f;
  for (int k = 0; k < a.ntrial; ++k) {
    mGa += tv[0][ql][k];
    mHa += tv[1][ql][k];
    mGb += tv[2][ql][k];
  }
  const float iK = 1.0f / (float)a.ntrial;
  mGa *= iK;
  mHa *= iK;
  mGb *= iK;
  const float dDa = E + mGa, dDb = E + mGb, rho = Ee + mHa;
  const int nqb = (a.S + AT - 1) / AT;
  const int nchunk = (a.ntrial + PSTORE_RC - 1) / PSTORE_RC;
  const int64_t plane = (int64_t)a.BH * pstore_tiles(nqb, a.causal) * AT * AT;
  // a chunk of jn trials fills the top 2 jn bits of its reversed word (an absent chunk: 0)
  int sh[2];
#pragma unroll
  for (int c = 0; c < 2; ++c) sh[c] = c < nchunk ? 32 - 2 * min(PSTORE_RC, a.ntrial - PSTORE_RC * c) : 0;

  floatx4 aq[PF_SOFTMAX][4];
#pragma unroll
  for (int i = 0; i < PF_SOFTMAX; ++i)
#pragma unroll
    for (int n = 0; n < 4; ++n) aq[i][n] = floatx4{0.f, 0.f, 0.f, 0.f};
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
  // one k-step's (key sub-tiles t = 2 s2, 2 s2 + 1) codes and decision words [chunk][tt], loaded
  // one k-step ahead of their use
  auto load_step = [&](int kb_, int s2_, uint32_t (&cw)[2], uint4 (&bw)[2][2]) {
    const int64_t base = fld_tile(a, z.bh, z.qb, kb_, nqb) + (int64_t)threadIdx.x * 16 + 8 * s2_;
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      const int key = kb_ * AT + 16 * (2 * s2_ + tt) + 4 * z.g;
      cw[tt] = (z.qok && key < a.S) ? *(const uint32_t*)(a.codes + pelem(a, z, key)) : 0u;
#pragma unroll
      for (int c = 0; c < 2; ++c)
        bw[c][tt] = c < nchunk ? *(const uint4*)(a.ubits + c * plane + base + 4 * tt) : make_uint4(0, 0, 0, 0);
    }
  };
  uint32_t cw_cur[2];
  uint4 bw_cur[2][2];
  load_step(0, 0, cw_cur, bw_cur);
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
    // one k-step at a time: fields, their store, their dQ terms
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      uint32_t cw_nxt[2] = {0u, 0u};
      uint4 bw_nxt[2][2] = {};
      if (s2 == 0)
        load_step(kb, 1, cw_nxt, bw_nxt);
      else if (kb + 1 < nkb)
        load_step(kb + 1, 0, cw_nxt, bw_nxt);
      float fl[PF_COUNT][2][4];
      Resid x[2][4];
      uint32_t nw[2][2][4];          // per chunk: the elements' decision words, normalized
      float na[2][4], nb[2][4];      // up-counts of a and b over the trials
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
        const int t = 2 * s2 + tt;
        const uint32_t w4[2][4] = {{bw_cur[0][tt].x, bw_cur[0][tt].y, bw_cur[0][tt].z, bw_cur[0][tt].w},
                                   {bw_cur[1][tt].x, bw_cur[1][tt].y, bw_cur[1][tt].z, bw_cur[1][tt].w}};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          x[tt][r] = resid(p[t][r], f8_val<FMT>(cw_cur[tt], r), s, rs, f);
          // chunk c's word with trial j's a at bit 2 j and b at bit 2 j + 1
#pragma unroll
          for (int c = 0; c < 2; ++c) nw[c][tt][r] = __builtin_bitreverse32(w4[c][r]) >> sh[c];
          na[tt][r] = (float)(__popc(nw[0][tt][r] & 0x55555555u) + __popc(nw[1][tt][r] & 0x55555555u));
          nb[tt][r] = (float)(__popc(nw[0][tt][r] & 0xAAAAAAAAu) + __popc(nw[1][tt][r] & 0xAAAAAAAAu));
        }
      }
      // per element: sum over trials of the up-decision times the row's per-trial sums
      float uga[2][4], uha[2][4], ugab[2][4], ugba[2][4];
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int r = 0; r < 4; ++r) uga[tt][r] = uha[tt][r] = ugab[tt][r] = ugba[tt][r] = 0.0f;
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        if (c >= nchunk) break;
        const int jn = min(PSTORE_RC, a.ntrial - PSTORE_RC * c);
#pragma unroll 2
        for (int j = 0; j < jn; ++j) {
          const int k = PSTORE_RC * c + j;
          const float gak = tv[0][ql][k], hak = tv[1][ql][k], gbk = tv[2][ql][k];
#pragma unroll
          for (int tt = 0; tt < 2; ++tt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float ua = (float)((nw[c][tt][r] >> (2 * j)) & 1u);
              const float vb = (float)((nw[c][tt][r] >> (2 * j + 1)) & 1u);
              uga[tt][r] = fmaf(ua, gak, uga[tt][r]);
              uha[tt][r] = fmaf(ua, hak, uha[tt][r]);
              ugab[tt][r] = fmaf(ua, gbk, ugab[tt][r]);
              ugba[tt][r] = fmaf(vb, gak, ugba[tt][r]);
            }
        }
      }
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
        const int t = 2 * s2 + tt;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float pp = p[t][r], d = dp[t][r], rr = x[tt][r].r, e = x[tt][r].e, h = x[tt][r].h;
          const float na_ = na[tt][r], nb_ = nb[tt][r];
          const float dpm = d - D;
          const float m1a = e + h * na_ * iK, m1b = e + h * nb_ * iK;
          const float mrDa = e * dDa + h * (E * na_ + uga[tt][r]) * iK;   // mean r_a dD_a
          const float mrRa = e * rho + h * (Ee * na_ + uha[tt][r]) * iK;  // mean r_a rho_a
          const float mrab = e * dDb + h * (E * na_ + ugab[tt][r]) * iK;  // mean r_a dD_b
          const float mrba = e * dDa + h * (E * nb_ + ugba[tt][r]) * iK;  // mean r_b dD_a
          fl[PF_REF][tt][r] = pp * dpm;
          fl[PF_R][tt][r] = rr * (dpm - DR) - pp * DR;
          fl[PF_N][tt][r] = m1a * dpm - pp * dDa - mrDa;
          fl[PF_K][tt][r] = pp * ((Ps1 + rho) * d - dDa) + (Ps * m1a + mrRa) * d - D * m1a - mrDa;
          fl[PF_J2][tt][r] = 0.5f * ((m1a + m1b) * dpm - pp * (dDa + dDb) - (mrab + mrba));
          fl[PF_Q2][tt][r] = 0.5f * ((m1a + rr) * dpm - pp * (dDa + DR) - (m1a * DR + rr * dDa));
          fl[PF_VU][tt][r] = -rr;
          fl[PF_VN][tt][r] = m1a - rr;
        }
        // store: tile (qb, kb) as [key][query]
#pragma unroll
        for (int i = 0; i < PF_COUNT; ++i) {
          float* T = a.fld[i] + tile;
#pragma unroll
          for (int r = 0; r < 4; ++r) T[(16 * t + 4 * z.g + r) * AT + 16 * z.w + z.c16] = fl[i][tt][r];
        }
      }
      // dQ terms of the softmax fields (k index: keys 32 s2 + 16 (v >> 2) + 4 g + (v & 3))
      bf16x8 fk[4];
#pragma unroll
      for (int n = 0; n < 4; ++n) fk[n] = frag_t(sm[st][2], 16 * n + z.c16, s2, z.g);
#pragma unroll
      for (int i = 0; i < PF_SOFTMAX; ++i) {
        float vd[8];
#pragma unroll
        for (int v = 0; v < 8; ++v) vd[v] = fl[i][v >> 2][v & 3];
        bf16x8 td[3];
        pack3(vd, td);
#pragma unroll
        for (int n = 0; n < 4; ++n)
#pragma unroll
          for (int j = 0; j < 3; ++j) aq[i][n] = mfma(td[j], fk[n], aq[i][n]);
      }
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
        cw_cur[tt] = cw_nxt[tt];
        bw_cur[0][tt] = bw_nxt[0][tt];
        bw_cur[1][tt] = bw_nxt[1][tt];
      }
    }
    if (kb + 1 < nkb) put(st ^ 1);
    __syncthreads();
  }
  const float c = a.scale;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int qr = z.q0 + 16 * z.w + 4 * z.g + r;
    if (qr >= a.S) continue;
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const int64_t e = z.hb + (int64_t)qr * AT + 16 * n + z.c16;
      const float ref = c * aq[PF_REF][n][r];
      float b[PF_SOFTMAX];
#pragma unroll
      for (int i = 0; i < PF_SOFTMAX; ++i) b[i] = c * aq[i][n][r];
      a.dQ_ref[e] = ref;
      write_policies(a, a.sm_field, a.dQ, e, ref, b);
    }
  }
}

// ------------------------------------------------------------------------------------
// key-major, one launch per gradient (PART 0: dK, PART 1: dV). dK = c sum_q field Q (three bf16
// terms per field); dV = s sum_q val(C) dO (one term), its biases sum_q (p - p_q) dO and
// sum_q (mean a - p_q) dO (three terms each). Lane (g, c16) of wave w owns key k0 + 16 w + c16.
// ------------------------------------------------------------------------------------
template <int FMT, int PART>
__global__ __launch_bounds__(256) void pstore_dkv_kernel(PstoreArgs a) {
  constexpr int NACC = PART == 0 ? PF_SOFTMAX : 3;
  __shared__ __attribute__((aligned(16))) u16 sm[2][AT * AT];  // Q^T (dK) or dO^T (dV)
  if (a.diag->nonfinite) return;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane >> 4, c16 = lane & 15;
  const int bh = blockIdx.x;
  const int kb = blockIdx.y;  // under the causal mask block 0 walks the most query blocks: first out
  const int k0 = kb * AT;
  const int key = k0 + 16 * w + c16;
  const int64_t hb = (int64_t)bh * a.S * AT, tb = (int64_t)bh * AT * a.Sp;
  const int nqb = (a.S + AT - 1) / AT;
  const float s = a.diag->scale;
  const u16* src = PART == 0 ? a.Qt : a.dOt;
  floatx4 acc[NACC][4];
#pragma unroll
  for (int n = 0; n < 4; ++n)
#pragma unroll
    for (int i = 0; i < NACC; ++i) acc[i][n] = floatx4{0.f, 0.f, 0.f, 0.f};
  TileRegs pf;
  const int qb0 = a.causal ? kb : 0;
  tile_fetch_t(pf, src + tb, qb0 * AT, a.Sp);
  tile_put_t(sm[0], pf);
  __syncthreads();
  for (int qb = qb0; qb < nqb; ++qb) {
    const int st = (qb - qb0) & 1, q0 = qb * AT;
    if (qb + 1 < nqb) tile_fetch_t(pf, src + tb, q0 + AT, a.Sp);
    const int64_t tile = fld_tile(a, bh, qb, kb, nqb);
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      // queries 32 s2 + 16 hh + 4 g + (0..3) of this lane's key, as the k index of the products
      bf16x8 fo[4];
#pragma unroll
      for (int n = 0; n < 4; ++n) fo[n] = frag_t(sm[st], 16 * n + c16, s2, g);
      auto fields = [&](int i, float (&v)[8]) {
        const float* T = a.fld[i] + tile + (int64_t)(16 * w + c16) * AT + 32 * s2 + 4 * g;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const float4 x = *(const float4*)(T + 16 * hh);
          v[4 * hh + 0] = x.x;
          v[4 * hh + 1] = x.y;
          v[4 * hh + 2] = x.z;
          v[4 * hh + 3] = x.w;
        }
      };
      if (PART == 0) {
        float vals[PF_SOFTMAX][8];
#pragma unroll
        for (int i = 0; i < PF_SOFTMAX; ++i) fields(i, vals[i]);
#pragma unroll
        for (int i = 0; i < PF_SOFTMAX; ++i) {
          bf16x8 td[3];
          pack3(vals[i], td);
#pragma unroll
          for (int n = 0; n < 4; ++n)
#pragma unroll
            for (int j = 0; j < 3; ++j) acc[i][n] = mfma(td[j], fo[n], acc[i][n]);
        }
      } else {
        float vu[8], vn[8], cv[8];
        fields(PF_VU, vu);
        fields(PF_VN, vn);
        // val(C) of (query, key) for the same eight queries (exact in bf16)
#pragma unroll
        for (int v = 0; v < 8; ++v) {
          const int qq = q0 + 32 * s2 + 16 * (v >> 2) + 4 * g + (v & 3);
          const bool ok = qq < a.S && key < a.S;
          const uint32_t b = ok ? a.codes[((int64_t)bh * a.S + qq) * a.S + key] : 0u;
          cv[v] = f8_val<FMT>(b, 0);
        }
        uint32_t pk[4];
#pragma unroll
        for (int i2 = 0; i2 < 4; ++i2) pk[i2] = pk_bf16(cv[2 * i2], cv[2 * i2 + 1]);
        const bf16x8 tv = __builtin_bit_cast(bf16x8, make_uint4(pk[0], pk[1], pk[2], pk[3]));
        bf16x8 tu[3], tn[3];
        pack3(vu, tu);
        pack3(vn, tn);
#pragma unroll
        for (int n = 0; n < 4; ++n) {
          acc[0][n] = mfma(tv, fo[n], acc[0][n]);
#pragma unroll
          for (int j = 0; j < 3; ++j) {
            acc[1][n] = mfma(tu[j], fo[n], acc[1][n]);
            acc[2][n] = mfma(tn[j], fo[n], acc[2][n]);
          }
        }
      }
    }
    if (qb + 1 < nqb) tile_put_t(sm[st ^ 1], pf);
    __syncthreads();
  }
  const float c = a.scale;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int kr = k0 + 16 * w + 4 * g + r;
    if (kr >= a.S) continue;
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const int64_t e = hb + (int64_t)kr * AT + 16 * n + c16;
      if (PART == 0) {
        const float ref = c * acc[PF_REF][n][r];
        float b[PF_SOFTMAX];
#pragma unroll
        for (int i = 0; i < PF_SOFTMAX; ++i) b[i] = c * acc[i][n][r];
        a.dK_ref[e] = ref;
        write_policies(a, a.sm_field, a.dK, e, ref, b);
      } else {
        const float ref = s * acc[0][n][r];
        const float b[3] = {0.0f, acc[1][n][r], acc[2][n][r]};
        a.dV_ref[e] = ref;
        write_policies(a, a.v_field, a.dV, e, ref, b);
      }
    }
  }
}

// ------------------------------------------------------------------------------------
bs_status launch_pstore_scale(const PstoreArgs& a, hipStream_t st) {
  pstore_scale_kernel<<<1, 1024, 0, st>>>(a.l, (int64_t)a.BH * a.S, a.f.fmax, a.diag, a.P_scale);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

static dim3 pstore_grid(const PstoreArgs& a) { return dim3((unsigned)a.BH, (unsigned)((a.S + AT - 1) / AT)); }

bs_status launch_pstore_fwd(const PstoreArgs& a, hipStream_t st) {
  ProfScope prof("pstore_fwd", st);
  if (a.fmt == BS_E5M2)
    pstore_fwd_kernel<BS_E5M2><<<pstore_grid(a), 256, 0, st>>>(a);
  else
    pstore_fwd_kernel<BS_E4M3><<<pstore_grid(a), 256, 0, st>>>(a);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

#define BS_PSTORE_KM(KERNEL, FMTV) KERNEL<FMTV><<<pstore_grid(a), 256, 0, st>>>(a)

template <int FMT>
static void rows_draw(const PstoreArgs& a, hipStream_t st) {
  const dim3 grid = pstore_grid(a);
  if (a.draw_b)
    pstore_rows_kernel<FMT, 2><<<grid, 256, 0, st>>>(a);
  else if (a.draw_a)
    pstore_rows_kernel<FMT, 1><<<grid, 256, 0, st>>>(a);
  else
    pstore_rows_kernel<FMT, 0><<<grid, 256, 0, st>>>(a);
}

bs_status launch_pstore_rows(const PstoreArgs& a, hipStream_t st) {
  if (a.ntrial < 1 || a.ntrial > PSTORE_KMAX) return BS_EINVAL;
  ProfScope prof("pstore_rows", st);
  if (a.fmt == BS_E5M2)
    rows_draw<BS_E5M2>(a, st);
  else
    rows_draw<BS_E4M3>(a, st);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status launch_pstore_dq(const PstoreArgs& a, hipStream_t st) {
  if (a.ntrial < 1 || a.ntrial > PSTORE_KMAX) return BS_EINVAL;
  ProfScope prof("pstore_dq", st);
  if (a.fmt == BS_E5M2)
    BS_PSTORE_KM(pstore_dq_kernel, BS_E5M2);
  else
    BS_PSTORE_KM(pstore_dq_kernel, BS_E4M3);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
#undef BS_PSTORE_KM

bs_status launch_pstore_dkv(const PstoreArgs& a, hipStream_t st) {
  ProfScope prof("pstore_dkv", st);
  if (a.fmt == BS_E5M2) {
    pstore_dkv_kernel<BS_E5M2, 0><<<pstore_grid(a), 256, 0, st>>>(a);
    pstore_dkv_kernel<BS_E5M2, 1><<<pstore_grid(a), 256, 0, st>>>(a);
  } else {
    pstore_dkv_kernel<BS_E4M3, 0><<<pstore_grid(a), 256, 0, st>>>(a);
    pstore_dkv_kernel<BS_E4M3, 1><<<pstore_grid(a), 256, 0, st>>>(a);
  }
  BS_CHECK_LAUNCH();
  return BS_OK;
}

}  // namespace bsp
