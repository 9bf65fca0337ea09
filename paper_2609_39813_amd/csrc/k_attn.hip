// Attention with an FP8 store of its output and a backward whose correction term D reads
// the original, the forward's rounding or a new rounding of that output (gfx950, dh = 64).
//
// Tile layouts and helpers: k_attn_tiles.h. fp32-valued operands (P, dS, P*dD) enter as three
// exact bf16 terms. Four waves per workgroup; wave w owns rows 16 w .. 16 w + 15 of a 64-row block.
#include "k_attn.h"
#include "k_attn_tiles.h"

namespace bsp {

// ------------------------------------------------------------------------------------
// D variants, one row per 4 lanes (16 elements per lane, four Philox calls per trial):
//   D_ref = sum dO O; dD_R = sum dO (s val(C_O) - O);
//   dD_k  = sum dO (s val(C_k) - O) for new roundings k = 1..K, = A + s S_k with
//   A = sum dO (s sign lo - O) (fp64) and S_k = sum dO sign step up_k. S_k holds no
//   trial-independent term, so it is summed in fp32 (per lane in element order, then over the
//   row's 4 lanes); its mean and sample SD over k come from fp64 sums of S_k - S_1.
// ------------------------------------------------------------------------------------
// (v_l + v_(l^1)) + (v_(l^2) + v_(l^3)) within a quad of lanes by two DPP exchanges (no LDS
// round trip): the same value in the four lanes, equal to two xor shuffles' sum
__device__ __forceinline__ float quad_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, false));  // quad_perm 1,0,3,2
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, false));  // quad_perm 2,3,0,1
  return v;
}

__global__ __launch_bounds__(256) void attn_d_kernel(AttnDArgs a) {
  constexpr int EPL = 16;
  const int64_t row = (int64_t)blockIdx.x * 64 + (threadIdx.x >> 2);
  const int sub = threadIdx.x & 3;
  const bool ok = row < a.rows;
  const int64_t e0 = row * AT + EPL * sub;
  const float s = *a.scale;
  const double rs = 1.0 / (double)s;
  double dref = 0.0, dr = 0.0, A = 0.0;
  uint32_t F[EPL];
  float w[EPL];
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
    F[q] = 0u;
    w[q] = 0.0f;
  }
  if (ok) {
#pragma unroll
    for (int j = 0; j < EPL / 4; ++j) {
      const int64_t e = e0 + 4 * j;
      const float4 o4 = *(const float4*)(a.O + e);
      const uint32_t c4 = *(const uint32_t*)(a.codes + e);
      const float ov[4] = {o4.x, o4.y, o4.z, o4.w};
      float dv[4];
      if (a.dO32) {
        const float4 g4 = *(const float4*)(a.dO32 + e);
        dv[0] = g4.x; dv[1] = g4.y; dv[2] = g4.z; dv[3] = g4.w;
      } else {
        const uint2 d2 = *(const uint2*)(a.dO + e);
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
        const float y = div_scale(ov[q], rs);
        const Bracket b = f8_bracket(fminf(fabsf(y), a.f.fmax), a.f);
        const float step = f8_step(b);
        A += g * ((double)s * (signbit(y) ? -1.0 : 1.0) * (double)b.mi * (double)step - o);
        F[4 * j + q] = b.F;
        w[4 * j + q] = (signbit(y) ? -dv[q] : dv[q]) * step;  // exact: a power-of-two scaling
      }
    }
  }
  // fixed-order sums over the row's 4 lanes
  auto rowsum = [&](auto v) {
    v += __shfl_xor(v, 1, 64);
    v += __shfl_xor(v, 2, 64);
    return v;
  };
  dref = rowsum(dref);
  dr = rowsum(dr);
  A = rowsum(A);
  double mean = 0.0, var = 0.0;
  if (a.want_n) {
#pragma unroll
    for (int q = 0; q < EPL; ++q) asm volatile("" : "+v"(F[q]), "+v"(w[q]));
    double s1 = 0.0, d1 = 0.0, d2 = 0.0;
    const uint64_t g0 = (uint64_t)(e0 >> 2);
    for (int k = 1; k <= a.K; ++k) {
      float Sk = 0.0f;
#pragma unroll
      for (int j = 0; j < EPL / 4; ++j) {
        const Philox4 p = philox_group(a.seed, g0 + j, (uint32_t)k, a.use);
        const uint32_t R[4] = {p.w0, p.w1, p.w2, p.w3};
#pragma unroll
        for (int q = 0; q < 4; ++q) Sk += sr_up(F[4 * j + q], R[q]) ? w[4 * j + q] : 0.0f;
      }
      Sk = quad_sum(Sk);
      if (a.dD_trials && ok && sub == 0) a.dD_trials[(int64_t)(k - 1) * a.rows + row] = (float)(A + (double)s * Sk);
      if (k == 1) s1 = Sk;
      const double dl = (double)Sk - s1;
      d1 += dl;
      d2 += dl * dl;
    }
    mean = s1 + d1 / a.K;
    var = a.K > 1 ? fmax(d2 - d1 * d1 / a.K, 0.0) / (a.K - 1) : 0.0;
  }
  if (ok && sub == 0) {
    a.D_ref[row] = (float)dref;
    a.dD_R[row] = (float)dr;
    if (a.want_n) {
      a.dD_N[row] = (float)(A + (double)s * mean);
      a.sd_N[row] = (float)((double)s * sqrt(var));
    }
  }
}

// ------------------------------------------------------------------------------------
// Backward. P and dS never leave registers: an MFMA result tile holds D[i][j] with j on
// lane & 15 and i = 4 (lane >> 4) + r, which is the layout of an MFMA operand whose row is j
// and whose k index runs over i. A 32-deep k step joins two such tiles: slot v of lane group
// g holds k = 16 (v >> 2) + 4 g + (v & 3) (within 32 of the step), and the other operand is
// read from a transposed tile in the same order (two 8-byte reads). Transposed tiles keep
// their 8-byte units XOR-swizzled by (row & 15), so the 16 rows of a read phase hit distinct
// banks. P and dS enter their products as three exact bf16 terms.
// ------------------------------------------------------------------------------------
// ------------------------------------------------------------------------------------
// forward: row max m, row sum l (P = exp(c S - m) / l) and optionally O = P V.
// S^T = K Q^T puts keys on the k index of the P operand of P V (register resident, three
// bf16 terms); wave w owns queries 16 w .. 16 w + 15, one per lane column.
// ------------------------------------------------------------------------------------
template <bool WRITE_O>
__global__ __launch_bounds__(256, 2) void attn_fwd_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) u16 sm[2][2][AT * AT];  // K, V^T
  // heaviest (most key blocks) first: blocks are dispatched in index order
  const int bh = blockIdx.x, qb = a.causal ? (int)gridDim.y - 1 - (int)blockIdx.y : (int)blockIdx.y;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane >> 4, c16 = lane & 15;
  const int q0 = qb * AT;
  const int64_t hb = (int64_t)bh * a.S * AT, tb = (int64_t)bh * AT * a.Sp;
  const int q = q0 + 16 * w + c16;
  const bool qok = q < a.S;
  bf16x8 fq[2];
#pragma unroll
  for (int s = 0; s < 2; ++s)
    fq[s] = __builtin_bit_cast(bf16x8, qok ? *(const uint4*)(a.Q + hb + (int64_t)q * AT + 32 * s + 8 * g)
                                           : make_uint4(0, 0, 0, 0));
  const float c2 = scores_scale(a.scale, a.scale_mul) * kLog2e;
  float m2 = -INFINITY, l = 0.0f;  // running max of c log2(e) S and sum, for query q (this lane's column)
  floatx4 acc[4];
#pragma unroll
  for (int n = 0; n < 4; ++n) acc[n] = floatx4{0.f, 0.f, 0.f, 0.f};
  TileRegs pf[2];
  auto fetch = [&](int k0) {
    tile_fetch(pf[0], a.K + hb, k0, a.S);
    tile_fetch_t(pf[1], a.Vt + tb, k0, a.Sp);
  };
  auto put = [&](int st) {
    tile_put(sm[st][0], pf[0]);
    tile_put_t(sm[st][1], pf[1]);
  };
  const int nkb = a.causal ? qb + 1 : (a.S + AT - 1) / AT;
  fetch(0);
  put(0);
  __syncthreads();
  for (int kb = 0; kb < nkb; ++kb) {
    const int st = kb & 1, k0 = kb * AT;
    if (kb + 1 < nkb) fetch(k0 + AT);
    const u16* tK = sm[st][0];
    const u16* tVt = sm[st][1];
    floatx4 sv[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) sv[t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int t = 0; t < 4; ++t) sv[t] = mfma(*(const bf16x8*)(tK + sw(16 * t + c16, 32 * s + 8 * g)), fq[s], sv[t]);
    // masks only where the block crosses S or the causal diagonal (a uniform test)
    const bool full = k0 + AT <= a.S && q0 + AT <= a.S && (!a.causal || k0 + AT - 1 <= q0);
    float x[4][4];
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) x[t][r] = c2 * sv[t][r];
    if (!full) {
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = k0 + 16 * t + 4 * g + r;
          x[t][r] = (key < a.S && qok && (!a.causal || key <= q)) ? x[t][r] : -INFINITY;
        }
    }
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) mx = fmaxf(mx, x[t][r]);
    // over the four lane groups of this query column
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float mn = fmaxf(m2, mx);
    const float alpha = (mn == -INFINITY || m2 == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(m2 - mn);
    float p[4][4], rs = 0.0f;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        // a row with no key yet has mn = -inf; its masked entries must not give 2^NaN
        p[t][r] = __builtin_amdgcn_exp2f(mn == -INFINITY ? -INFINITY : x[t][r] - mn);
        rs += p[t][r];
      }
    rs += __shfl_xor(rs, 16, 64);
    rs += __shfl_xor(rs, 32, 64);
    l = l * alpha + rs;
    m2 = mn;
    if (WRITE_O) {
      // the accumulator rows are queries 16 w + 4 g + r: their rescale factors live in the
      // lanes whose column is that query
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float ar = __shfl(alpha, 4 * g + r, 64);
#pragma unroll
        for (int n = 0; n < 4; ++n) acc[n][r] *= ar;
      }
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        float vp[8];
#pragma unroll
        for (int v = 0; v < 8; ++v) vp[v] = p[2 * s + (v >> 2)][v & 3];
        bf16x8 tp[3];
        pack3(vp, tp);
#pragma unroll
        for (int n = 0; n < 4; ++n) {
          const bf16x8 fv = frag_t(tVt, 16 * n + c16, s, g);
#pragma unroll
          for (int j = 0; j < 3; ++j) acc[n] = mfma(tp[j], fv, acc[n]);
        }
      }
    }
    if (kb + 1 < nkb) put(st ^ 1);
    __syncthreads();
  }
  const int64_t rb = (int64_t)bh * a.S;
  if (qok && g == 0) {
    a.m[rb + q] = m2;
    a.l[rb + q] = l;
  }
  if (WRITE_O) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int qr = q0 + 16 * w + 4 * g + r;
      const float lr = __shfl(l, 4 * g + r, 64);
      if (qr >= a.S) continue;
#pragma unroll
      for (int n = 0; n < 4; ++n) a.O_out[hb + (int64_t)qr * AT + 16 * n + c16] = acc[n][r] / lr;
    }
  }
}

// ------------------------------------------------------------------------------------
// key-block-major: dV = P^T dO, dK = c dS^T Q and the dK bias terms -c P^T (dD_v * Q)
// (v = R, N). S = Q K^T and dP = dO V^T are formed with queries as rows, so that their
// result tiles are the (key, query) operands of the three products.
//
// A query block's operands sit in two LDS halves: the row-major tiles (Q and the dO planes,
// read by S and dP) and the transposed ones (Q^T and the dO^T planes, read by the products).
// Both arrive by buffer loads straight into LDS (no staging registers; rows past S read as
// zero). A half is refilled for the next query block once every wave has read it: the
// row-major half after S and dP, the transposed half after the products, so each load lands
// while the other half is in use. BIAS = 0: no policy reads R or N (no bias accumulators);
// BIAS = 1 forms both bias terms (a missing dD_v reads as zero).
// ------------------------------------------------------------------------------------
// H: the incoming gradient as the two-term fp16 split of dO 2^e (NDO = 2) and V as fp16(V 2^f);
// dP comes back by 2^-e-f, and dV = P^T dO (P split at the scale 2^14, the products of the two
// splits' terms of order above 2^-22 taken) by 2^-e-14; dK = dS^T Q from the two-term split of
// dS 2^s and fp16(Q 2^q), back by 2^-s-q
template <int NDO, int BIAS, bool H>
__global__ __launch_bounds__(256, 2) void attn_bwd_k_kernel(AttnBwdArgs a) {
  static_assert(!H || (NDO == 2 && !BIAS), "fp16 operands: two terms, no dD");
  constexpr int NR = 1 + NDO;     // tiles per half
  constexpr int NL = 2 * NR;      // loads per wave and half (two 1-KB loads per tile)
  __shared__ __attribute__((aligned(1024))) u16 smR[NR][AT * AT];
  __shared__ __attribute__((aligned(1024))) u16 smT[NR][AT * AT];
  // m, 1/l, D, dD_R, dD_N per query for two query blocks, as two variables: the loop is
  // unrolled by two so each access names one of them, and loads into one are not awaited
  // before reads of the other
  constexpr int NRW = BIAS ? 2 : 1;  // row loads per wave and query block
  __shared__ float rows0[4 * NRW][AT], rows1[4 * NRW][AT];
  const int bh = blockIdx.x, kb = blockIdx.y;
  const int lane = threadIdx.x & 63, g = lane >> 4, c16 = lane & 15;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int k0 = kb * AT;
  const int64_t hb = (int64_t)bh * a.S * AT, tb = (int64_t)bh * AT * a.Sp, rb = (int64_t)bh * a.S;
  const int key = k0 + 16 * w + c16;
  const float dps = H ? a.f16_inv[0] * a.f16_inv[1] : 1.0f, avs = H ? a.f16_inv[0] * 0x1p-14f : 1.0f;
  const float dsc = H ? a.f16_inv[4] : 1.0f, dkm = H ? a.f16_inv[5] : 1.0f;
  // H: P comes out at its split's scale 2^14 (1/l scaled), and dS at its split's scale 2^s (dP's
  // multiplier and D scaled by 2^s 2^-14), so neither split multiplies per element
  const float lsc = H ? 0x1p14f : 1.0f, dpm = H ? dps * dsc * 0x1p-14f : dps, dmul = H ? dsc * 0x1p-14f : 1.0f;
  // this wave's keys as the second operand of S and dP (fixed over the loop)
  bf16x8 fk[2], fv[2];
  const u16* const Vsrc = H ? a.V16 : a.V;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int64_t e = hb + (int64_t)key * AT + 32 * s + 8 * g;
    const uint4 zk = key < a.S ? *(const uint4*)(a.K + e) : make_uint4(0, 0, 0, 0);
    const uint4 zv = key < a.S ? *(const uint4*)(Vsrc + e) : make_uint4(0, 0, 0, 0);
    fk[s] = __builtin_bit_cast(bf16x8, zk);
    fv[s] = __builtin_bit_cast(bf16x8, zv);
  }

  // resources: row-major tiles end at row S, transposed copies span their Sp columns
  __amdgpu_buffer_rsrc_t rR[NR], rT[NR];
  rR[0] = attn_rsrc(a.Q + hb, (int64_t)a.S * AT * 2);
  rT[0] = attn_rsrc((H ? a.Qt16 : a.Qt) + tb, (int64_t)AT * a.Sp * 2);
#pragma unroll
  for (int i = 0; i < NDO; ++i) {
    rR[1 + i] = attn_rsrc((NDO == 1 ? a.dO : a.dOp[i]) + hb, (int64_t)a.S * AT * 2);
    rT[1 + i] = attn_rsrc(a.dOt[i] + tb, (int64_t)AT * a.Sp * 2);
  }
  // lane l of load j (two per wave and tile) fills tile row 8 (2 w + j) + l / 8 at chunk
  // position l % 8, which holds logical chunk (l % 8) ^ (l / 8) of the row (the sw layout)
  const int lr = lane >> 3, lch = (lane & 7) ^ lr;
  const uint32_t vR = (uint32_t)(lr * AT * 2 + lch * 16), vT = (uint32_t)(lr * a.Sp * 2 + lch * 16);
  // (each resource is copied to a scalar first: the host pass rejects a 16-byte LDS load
  // whose resource is an array element)
  auto issue_R = [&](int q0) {
#pragma unroll
    for (int t = 0; t < NR; ++t) {
      const __amdgpu_buffer_rsrc_t r = rR[t];
#pragma unroll
      for (int j = 0; j < 2; ++j)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (void __attribute__((address_space(3)))*)(smR[t] + (2 * w + j) * 512),
                                                 16, vR, (uint32_t)(q0 * AT * 2 + (2 * w + j) * 1024), 0, 0);
    }
  };
  auto issue_T = [&](int q0) {
#pragma unroll
    for (int t = 0; t < NR; ++t) {
      const __amdgpu_buffer_rsrc_t r = rT[t];
#pragma unroll
      for (int j = 0; j < 2; ++j)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (void __attribute__((address_space(3)))*)(smT[t] + (2 * w + j) * 512),
                                                 16, vT, (uint32_t)(q0 * 2 + (2 * w + j) * 16 * a.Sp), 0, 0);
    }
  };
  // The per-query rows m, l, D (and dD_R, dD_N) go straight into LDS too, one dword per lane:
  // wave w loads row arrays NRW w .. NRW w + NRW - 1 of (m, l, D[, dD_R, dD_N, -, -, -]).
  // Queries past S, a missing dD_v and the padding (empty resources) read as zero; every wave
  // issues NL + NRW loads per query block.
  const float* row_src[8] = {a.m, a.l, a.D_ref, BIAS ? a.dD_R : nullptr, BIAS ? a.dD_N : nullptr,
                             nullptr, nullptr, nullptr};
  __amdgpu_buffer_rsrc_t rq[NRW];
#pragma unroll
  for (int k = 0; k < NRW; ++k) {
    const float* base = row_src[NRW * w + k];
    rq[k] = __builtin_amdgcn_make_buffer_rsrc((void*)(base ? base + rb : a.m), (short)0, base ? a.S * 4 : 0,
                                              0x00020000);
  }
  auto issue_rows = [&](float (*rows)[AT], int q0) {
#pragma unroll
    for (int k = 0; k < NRW; ++k) {
      const __amdgpu_buffer_rsrc_t r = rq[k];
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (void __attribute__((address_space(3)))*)(rows[NRW * w + k]), 4,
                                               (uint32_t)(lane * 4), (uint32_t)(q0 * 4), 0, 0);
    }
  };

  floatx4 av[4], ak[4], akr[4], akn[4];
#pragma unroll
  for (int n = 0; n < 4; ++n) av[n] = ak[n] = akr[n] = akn[n] = floatx4{0.f, 0.f, 0.f, 0.f};
  const float c2 = a.scale * kLog2e;
  const int nqb = (a.S + AT - 1) / AT, qb0 = a.causal ? kb : 0;
  issue_R(qb0 * AT);
  issue_rows(rows0, qb0 * AT);
  issue_T(qb0 * AT);
  ATTN_WAIT_VM(0);
  ATTN_LDS_BARRIER();
  // one query block; rows: its rows, nrows: the next block's
  auto step = [&](int qb, float (*rows)[AT], float (*nrows)[AT]) {
    const int q0 = qb * AT;
    const bool more = qb + 1 < nqb;
    // the rows have landed: 1/l in place (wave 1; 0 past S), read after the next barrier
    if (w == 1) {
      const float l = rows[1][lane];
      rows[1][lane] = q0 + lane < a.S ? lsc / l : 0.0f;
    }
    if (H && w == 2) rows[2][lane] *= dmul;
    // S, dP: query tiles t (rows), this wave's keys (columns)
    floatx4 sv[4], dp[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) sv[t] = dp[t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 2; ++s) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        sv[t] = mfma(*(const bf16x8*)(smR[0] + sw(16 * t + c16, 32 * s + 8 * g)), fk[s], sv[t]);
#pragma unroll
        for (int i = 0; i < NDO; ++i) {
          const bf16x8 fo = *(const bf16x8*)(smR[1 + i] + sw(16 * t + c16, 32 * s + 8 * g));
          dp[t] = H ? mfma_h(fo, fv[s], dp[t]) : mfma(fo, fv[s], dp[t]);
        }
      }
    }
    // every wave has read the row-major half: the next query block's tiles and rows go in
    // (after the last query block too: those loads read past S, as zeros, and are never used,
    // so that every wave's count of loads in flight below is fixed)
    ATTN_LDS_BARRIER();
    issue_R(q0 + AT);
    issue_rows(nrows, q0 + AT);
    // masks only where the block crosses S or the causal diagonal (a uniform test)
    const bool full = k0 + AT <= a.S && q0 + AT <= a.S && (!a.causal || k0 + AT - 1 <= q0);
    float p[4][4], ds[4][4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) p[t][r] = fmaf(c2, sv[t][r], -rows[0][16 * t + 4 * g + r]);
    if (!full) {
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int q = q0 + 16 * t + 4 * g + r;
          p[t][r] = (key < a.S && q < a.S && (!a.causal || key <= q)) ? p[t][r] : -INFINITY;  // 2^-inf = 0
        }
    }
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int ql = 16 * t + 4 * g + r;
        p[t][r] = __builtin_amdgcn_exp2f(p[t][r]) * rows[1][ql];
        ds[t][r] = p[t][r] * (dp[t][r] * dpm - rows[2][ql]);
      }
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      float vp[8], vd[8];
#pragma unroll
      for (int v = 0; v < 8; ++v) {
        vp[v] = p[2 * s + (v >> 2)][v & 3];
        vd[v] = ds[2 * s + (v >> 2)][v & 3];
      }
      bf16x8 tp[3], td[3], tr[3], tn[3];
      if constexpr (H) {
        float vs[8], ws[8];
#pragma unroll
        for (int v = 0; v < 8; ++v) {
          vs[v] = vp[v];  // P 2^14
          ws[v] = vd[v];  // dS 2^s
        }
        pack2h(vs, tp);
        pack2h(ws, td);
      } else {
        pack3t(vp, tp);
        pack3t(vd, td);
      }
      if (BIAS) {
        // bias terms: P scaled per query by dD_v
        float vr[8], vn[8];
#pragma unroll
        for (int v = 0; v < 8; ++v) {
          const int ql = 32 * s + 16 * (v >> 2) + 4 * g + (v & 3);
          vr[v] = vp[v] * rows[3][ql];
          vn[v] = vp[v] * rows[4][ql];
        }
        pack3t(vr, tr);
        pack3t(vn, tn);
      }
      if (s == 0) {
        // the transposed half of this query block has landed in every wave
        ATTN_WAIT_VM(NL + NRW);
        ATTN_LDS_BARRIER();
      }
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        const bf16x8 fq = frag_t(smT[0], 16 * n + c16, s, g);
#pragma unroll
        for (int i = 0; i < NDO; ++i) {
          const bf16x8 fo = frag_t(smT[1 + i], 16 * n + c16, s, g);
#pragma unroll
          for (int j = 0; j < (H ? 2 : 3); ++j) {
            if (H && i + j <= 1) av[n] = mfma_h(tp[j], fo, av[n]);
            if (!H && i + j <= 2) av[n] = mfma(tp[j], fo, av[n]);
          }
        }
        if constexpr (H) {
#pragma unroll
          for (int j = 0; j < 2; ++j) ak[n] = mfma_h(td[j], fq, ak[n]);
        } else {
#pragma unroll
          for (int j = 0; j < 3; ++j) ak[n] = mfma(td[j], fq, ak[n]);
        }
        if (BIAS) {
#pragma unroll
          for (int j = 0; j < 3; ++j) {
            akr[n] = mfma(tr[j], fq, akr[n]);
            akn[n] = mfma(tn[j], fq, akn[n]);
          }
        }
      }
    }
    // every wave has read the transposed half and the next row-major half has landed
    ATTN_WAIT_VM(0);
    ATTN_LDS_BARRIER();
    if (more) issue_T(q0 + AT);
  };
  for (int qb = qb0; qb < nqb; qb += 2) {
    step(qb, rows0, rows1);
    if (qb + 1 < nqb) step(qb + 1, rows1, rows0);
  }
  const float c = a.scale;
  float mx = 0.0f;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int kr = k0 + 16 * w + 4 * g + r;
    if (kr >= a.S) continue;
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const int64_t e = hb + (int64_t)kr * AT + 16 * n + c16;
      const float dk = c * (ak[n][r] * dkm);
      a.dV[e] = av[n][r] * avs;
      mx = fmaxf(mx, fmaxf(fabsf(dk), fabsf(av[n][r] * avs)));
      a.dK_ref[e] = dk;
      for (int pi = 0; pi < a.n_pol; ++pi) {
        const int kind = a.pol[pi];
        const float bias = kind == BS_READ_U ? 0.0f : -c * (kind == BS_READ_R ? akr[n][r] : akn[n][r]);
        if (a.kmean[pi]) a.kmean[pi][e] = dk + bias;
        if (a.kbias[pi]) a.kbias[pi][e] = bias;
      }
    }
  }
  if (a.amax) wave_amax_to_slot(mx, a.amax);
}

// ------------------------------------------------------------------------------------
// query-block-major: dQ = c dS K and G = P K; per-policy dQ estimates
//   bias_v = -c dD_v G (row-scaled), se_N = c |G| sd_N / sqrt(K).
// S^T = K Q^T and dP^T = V dO^T put keys on the k index of the dS / P operands.
// ------------------------------------------------------------------------------------
// The key block's tiles (K, V, K^T) arrive by buffer loads straight into LDS, two stages as two
// LDS variables (the loop is unrolled by two so that every access names one of them: loads into
// one stage are then not awaited before reads of the other); one barrier per key block.
// G: G = P K is formed (the per-policy estimates need it; without policies only dQ is). H: fp16
// operands of dO, V and dS as in the key-major pass, dP brought back by 2^-e-f, dQ = dS K (fp16(K
// 2^k)) by 2^-s-k.
template <int NDO, bool G, bool H>
__global__ __launch_bounds__(256, 2) void attn_bwd_q_kernel(AttnBwdArgs a) {
  static_assert(!H || (NDO == 2 && !G), "fp16 operands: two terms, no policies");
  __shared__ __attribute__((aligned(1024))) u16 sm0[3][AT * AT];  // K, V, K^T
  __shared__ __attribute__((aligned(1024))) u16 sm1[3][AT * AT];
  // heaviest (most key blocks) first: blocks are dispatched in index order
  const int bh = blockIdx.x, qb = a.causal ? (int)gridDim.y - 1 - (int)blockIdx.y : (int)blockIdx.y;
  const int lane = threadIdx.x & 63, g = lane >> 4, c16 = lane & 15;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int q0 = qb * AT;
  const int64_t hb = (int64_t)bh * a.S * AT, tb = (int64_t)bh * AT * a.Sp, rb = (int64_t)bh * a.S;
  const int q = q0 + 16 * w + c16;
  const bool qok = q < a.S;
  bf16x8 fq[2], fdo[NDO][2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int64_t e = hb + (int64_t)q * AT + 32 * s + 8 * g;
    fq[s] = __builtin_bit_cast(bf16x8, qok ? *(const uint4*)(a.Q + e) : make_uint4(0, 0, 0, 0));
#pragma unroll
    for (int i = 0; i < NDO; ++i) {
      const u16* src = NDO == 1 ? a.dO : a.dOp[i];
      fdo[i][s] = __builtin_bit_cast(bf16x8, qok ? *(const uint4*)(src + e) : make_uint4(0, 0, 0, 0));
    }
  }
  const float mq = qok ? a.m[rb + q] : 0.0f;
  const float c2 = a.scale * kLog2e;
  const float ilq = qok ? 1.0f / a.l[rb + q] : 0.0f;
  const float dq_ref = qok ? a.D_ref[rb + q] : 0.0f;
  const float dps = H ? a.f16_inv[0] * a.f16_inv[1] : 1.0f;
  const float dsc = H ? a.f16_inv[4] : 1.0f, dqm = H ? a.f16_inv[6] : 1.0f;
  // H: dS comes out at its split's scale 2^s (dP's multiplier and D scaled)
  const float dpm = dps * dsc, dq_s = dq_ref * dsc;

  // K and V end at row S (rows past it read as zero), K^T spans its Sp columns; lane l of load j
  // (two per wave and tile) fills tile row 8 (2 w + j) + l / 8 at chunk position l % 8, which
  // holds logical chunk (l % 8) ^ (l / 8) (the sw layout)
  const __amdgpu_buffer_rsrc_t rK = attn_rsrc(a.K + hb, (int64_t)a.S * AT * 2);
  const __amdgpu_buffer_rsrc_t rV = attn_rsrc((H ? a.V16 : a.V) + hb, (int64_t)a.S * AT * 2);
  const __amdgpu_buffer_rsrc_t rKt = attn_rsrc((H ? a.Kt16 : a.Kt) + tb, (int64_t)AT * a.Sp * 2);
  const int lr = lane >> 3, lch = (lane & 7) ^ lr;
  const uint32_t vR = (uint32_t)(lr * AT * 2 + lch * 16), vT = (uint32_t)(lr * a.Sp * 2 + lch * 16);
  auto issue = [&](u16 (*sm)[AT * AT], int k0) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const uint32_t row = (uint32_t)(2 * w + j);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rK, (void __attribute__((address_space(3)))*)(sm[0] + row * 512), 16,
                                               vR, (uint32_t)(k0 * AT * 2) + row * 1024, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rV, (void __attribute__((address_space(3)))*)(sm[1] + row * 512), 16,
                                               vR, (uint32_t)(k0 * AT * 2) + row * 1024, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rKt, (void __attribute__((address_space(3)))*)(sm[2] + row * 512), 16,
                                               vT, (uint32_t)(k0 * 2) + row * 16 * (uint32_t)a.Sp, 0, 0);
    }
  };
  floatx4 aq[4], ag[4];
#pragma unroll
  for (int n = 0; n < 4; ++n) aq[n] = ag[n] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int nkb = a.causal ? qb + 1 : (a.S + AT - 1) / AT;
  issue(sm0, 0);
  // key block kb from stage cur; the next block's tiles go into nxt, which every wave finished
  // reading in the previous step (the barrier)
  auto step = [&](int kb, u16 (*cur)[AT * AT], u16 (*nxt)[AT * AT]) {
    const int k0 = kb * AT;
    ATTN_WAIT_VM(0);  // this block's tiles (the only loads in flight)
    ATTN_LDS_BARRIER();
    if (kb + 1 < nkb) issue(nxt, k0 + AT);
    const u16* tK = cur[0];
    const u16* tV = cur[1];
    const u16* tKt = cur[2];
    floatx4 sv[4], dp[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) sv[t] = dp[t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 2; ++s) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        sv[t] = mfma(*(const bf16x8*)(tK + sw(16 * t + c16, 32 * s + 8 * g)), fq[s], sv[t]);
        const bf16x8 fvv = *(const bf16x8*)(tV + sw(16 * t + c16, 32 * s + 8 * g));
#pragma unroll
        for (int i = 0; i < NDO; ++i) dp[t] = H ? mfma_h(fvv, fdo[i][s], dp[t]) : mfma(fvv, fdo[i][s], dp[t]);
      }
    }
    // masks only where the block crosses S or the causal diagonal (a uniform test)
    const bool full = k0 + AT <= a.S && q0 + AT <= a.S && (!a.causal || k0 + AT - 1 <= q0);
    float p[4][4], ds[4][4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) p[t][r] = fmaf(c2, sv[t][r], -mq);
    if (!full) {
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int kk = k0 + 16 * t + 4 * g + r;
          p[t][r] = (kk < a.S && qok && (!a.causal || kk <= q)) ? p[t][r] : -INFINITY;  // 2^-inf = 0
        }
    }
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        p[t][r] = __builtin_amdgcn_exp2f(p[t][r]) * ilq;
        ds[t][r] = p[t][r] * (dp[t][r] * dpm - dq_s);
      }
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      float vp[8], vd[8];
#pragma unroll
      for (int v = 0; v < 8; ++v) {
        vp[v] = p[2 * s + (v >> 2)][v & 3];
        vd[v] = ds[2 * s + (v >> 2)][v & 3];
      }
      bf16x8 tp[3], td[3];
      if (G) pack3t(vp, tp);
      if constexpr (H) {
        float ws[8];
#pragma unroll
        for (int v = 0; v < 8; ++v) ws[v] = vd[v];  // dS 2^s
        pack2h(ws, td);
      } else {
        pack3t(vd, td);
      }
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        const bf16x8 fk = frag_t(tKt, 16 * n + c16, s, g);
        if constexpr (H) {
#pragma unroll
          for (int j = 0; j < 2; ++j) aq[n] = mfma_h(td[j], fk, aq[n]);
        } else {
#pragma unroll
          for (int j = 0; j < 3; ++j) {
            aq[n] = mfma(td[j], fk, aq[n]);
            if (G) ag[n] = mfma(tp[j], fk, ag[n]);
          }
        }
      }
    }
  };
  for (int kb = 0; kb < nkb; kb += 2) {
    step(kb, sm0, sm1);
    if (kb + 1 < nkb) step(kb + 1, sm1, sm0);
  }
  const float c = a.scale;
  const float rk = a.ntrial > 0 ? 1.0f / sqrtf((float)a.ntrial) : 0.0f;
  float mx = 0.0f;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int qr = q0 + 16 * w + 4 * g + r;
    if (qr >= a.S) continue;
    const float ddr = a.dD_R ? a.dD_R[rb + qr] : 0.0f;
    const float ddn = a.dD_N ? a.dD_N[rb + qr] : 0.0f;
    const float sdn = a.sd_N ? a.sd_N[rb + qr] : 0.0f;
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const int64_t e = hb + (int64_t)qr * AT + 16 * n + c16;
      const float dq = c * (aq[n][r] * dqm);
      const float gg = ag[n][r];
      a.dQ_ref[e] = dq;
      mx = fmaxf(mx, fabsf(dq));
      for (int pi = 0; G && pi < a.n_pol; ++pi) {
        const int kind = a.pol[pi];
        const float bias = kind == BS_READ_U ? 0.0f : -c * (kind == BS_READ_R ? ddr : ddn) * gg;
        if (a.mean[pi]) a.mean[pi][e] = dq + bias;
        if (a.bias[pi]) a.bias[pi][e] = bias;
        if (a.se[pi]) a.se[pi][e] = kind == BS_READ_N ? c * fabsf(gg) * sdn * rk : 0.0f;
      }
    }
  }
  if (a.amax) wave_amax_to_slot(mx, a.amax);
}

// ------------------------------------------------------------------------------------
// operand copies for the backward: X^T [BH][64][Sp] (zero past S, tiles in fragment order,
// tperm) of bf16 X [BH][S][64]; for an fp32 X, its three bf16 planes (row-major) and their
// transposes
// ------------------------------------------------------------------------------------
// H (fp32 x): the two fp16 terms (split2_f16) of x 2^e, e from the max in slots, 2^-e to inv_out;
// htok > 0: x is token-major [B][S][htok 64] (row s of head bh at ((b S + s) htok + h) 64)
template <typename X, bool H>
__global__ __launch_bounds__(256) void attn_prep_kernel(const X* __restrict__ x, int S, int Sp, int htok,
                                                        const uint32_t* __restrict__ slots, float* __restrict__ inv_out,
                                                        u16* __restrict__ xt0,
                                                        u16* __restrict__ xt1, u16* __restrict__ xt2,
                                                        u16* __restrict__ xp0, u16* __restrict__ xp1,
                                                        u16* __restrict__ xp2) {
  constexpr int NP = sizeof(X) == 4 ? (H ? 2 : 3) : 1;
  __shared__ u16 t[NP][AT][AT + 2];
  float scl = 1.0f;
  if constexpr (H) {
    const int e = f16_scale_exp(amax_of_slots(slots));
    scl = ldexpf(1.0f, e);
    if (inv_out && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) *inv_out = ldexpf(1.0f, -e);
  }
  const int r0 = blockIdx.x * AT, bh = blockIdx.y;
  const int64_t hb = (int64_t)bh * S * AT, tb = (int64_t)bh * AT * Sp;
  // source row stride and origin of this head's rows
  const int64_t xs = htok > 0 ? (int64_t)htok * AT : AT;
  const int64_t xb = htok > 0 ? ((int64_t)(bh / htok) * S * htok + bh % htok) * AT : hb;
  u16* const xp[3] = {xp0, xp1, xp2};
  u16* const xt[3] = {xt0, xt1, xt2};
  for (int e = threadIdx.x; e < AT * AT; e += 256) {
    const int r = e >> 6, c = e & 63;
    const bool ok = r0 + r < S;
    if constexpr (NP == 1) {
      t[0][r][c] = ok ? (u16)x[xb + (int64_t)(r0 + r) * xs + c] : (u16)0;
    } else {
      const float v = ok ? load_f32(x, xb + (int64_t)(r0 + r) * xs + c) : 0.0f;
      u16 h[3];
      if constexpr (H)
        split2_f16(v * scl, h[0], h[1]);
      else
        split3(v, h[0], h[1], h[2]);
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        t[p][r][c] = h[p];
        if (ok) xp[p][hb + (int64_t)(r0 + r) * AT + c] = h[p];
      }
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < AT * AT; e += 256) {
    const int c = e >> 6, r = e & 63;
#pragma unroll
    for (int p = 0; p < NP; ++p) xt[p][tb + (int64_t)c * Sp + r0 + r] = t[p][tperm(r)][c];
  }
}

// ------------------------------------------------------------------------------------
bs_status launch_attn_fwd(const AttnArgs& a, int B, int H, hipStream_t st) {
  dim3 grid((unsigned)(B * H), (unsigned)((a.S + AT - 1) / AT));
  ProfScope prof("attn_fwd", st);
  if (a.O_out)
    attn_fwd_kernel<true><<<grid, 256, 0, st>>>(a);
  else
    attn_fwd_kernel<false><<<grid, 256, 0, st>>>(a);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

// ------------------------------------------------------------------------------------
// Level-2 D use, one row per 4 lanes (16 elements per lane). Per element, with the bracket of
// y = fl32(O/s) (sign sg, lower magnitude mi step): A = s sg mi step - O (fp64, exact) and
// w = s sg step; trial k's forward rounding error is r_k = A + u_k w and a new rounding's is
// r'_k = A + u'_k w (u, u' the up-decisions; for an RNE forward u_k is the fixed RNE decision).
// With g_k = dO + beta r_k:
//   R error  rowsum(g_k r_k)  = rowsum(dO A + beta A^2) + sum u_k (dO w + beta (2 A w + w^2))
//   N error  rowsum(g_k r'_k) = rowsum(dO A + beta A^2) + sum u'_k (dO w + beta A w)
//                               + sum u_k beta A w + sum u_k u'_k beta w^2
//   T_k      = beta / 2 sum (u_k xor u'_k) w^2
// The fixed parts are summed in fp64, the trial parts in fp32 per trial (they hold no
// trial-independent term) and their mean and SD over trials from fp64 sums shifted by trial 1.
// ------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void attn_l2_kernel(AttnL2Args a) {
  constexpr int EPL = 16;
  const int64_t row = (int64_t)blockIdx.x * 64 + (threadIdx.x >> 2);
  const int sub = threadIdx.x & 3;
  const bool ok = row < a.rows;
  const int64_t e0 = row * AT + EPL * sub;
  const float s = *a.scale;
  const double rs = 1.0 / (double)s;
  const double beta = a.beta;
  // one element's bracket terms: A = s sg mi step - O (fp64, exact) and w = s sg step
  auto terms = [&](float o, double& A, double& w, Bracket& b) {
    const float y = div_scale(o, rs);
    b = f8_bracket(fminf(fabsf(y), a.f.fmax), a.f);
    const double sg = signbit(y) ? -1.0 : 1.0;
    w = (double)s * sg * (double)f8_step(b);
    A = (double)s * sg * (double)b.mi * (double)f8_step(b) - (double)o;
  };
  auto load4 = [&](int j, float (&ov)[4], float (&dv)[4]) {
    const int64_t e = e0 + 4 * j;
    const float4 o4 = *(const float4*)(a.O + e);
    const uint2 d2 = *(const uint2*)(a.dO + e);
    ov[0] = o4.x; ov[1] = o4.y; ov[2] = o4.z; ov[3] = o4.w;
    dv[0] = bf16_to_f32((u16)(d2.x & 0xFFFF));
    dv[1] = bf16_to_f32((u16)(d2.x >> 16));
    dv[2] = bf16_to_f32((u16)(d2.y & 0xFFFF));
    dv[3] = bf16_to_f32((u16)(d2.y >> 16));
  };
  // trial coefficients: R gains cR where u_k = 1; N gains cN1 where u'_k = 1, cN2 where
  // u_k = 1 and cN3 where both are; T gains cN3 / 2 where they differ
  float cR[EPL], cN1[EPL], cN2[EPL], cN3[EPL];
  uint32_t F[EPL];
  uint32_t ufix = 0u;  // bit i: RNE decision of element i
  double fixed = 0.0;
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
    cR[q] = cN1[q] = cN2[q] = cN3[q] = 0.0f;
    F[q] = 0u;
  }
  if (ok) {
#pragma unroll
    for (int j = 0; j < EPL / 4; ++j) {
      float ov[4], dv[4];
      load4(j, ov, dv);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int i = 4 * j + q;
        double A, w;
        Bracket b;
        terms(ov[q], A, w, b);
        fixed += ((double)dv[q] + beta * A) * A;
        cN1[i] = (float)((double)dv[q] * w + beta * A * w);
        cN2[i] = (float)(beta * A * w);
        cN3[i] = (float)(beta * w * w);
        cR[i] = (float)((double)dv[q] * w + beta * (2.0 * A * w + w * w));
        F[i] = b.F;
        ufix |= (a.fwd_mode == BS_RNE ? rne_up(b) : 0u) << i;
      }
    }
  }
  auto rowsum = [&](auto v) {
    v += __shfl_xor(v, 1, 64);
    v += __shfl_xor(v, 2, 64);
    return v;
  };
  // per element: up-counts of the forward's and the new roundings over the trials
  uint32_t n[EPL], np[EPL];
#pragma unroll
  for (int q = 0; q < EPL; ++q) n[q] = np[q] = 0u;
  double s1[3] = {0.0, 0.0, 0.0}, d1[3] = {0.0, 0.0, 0.0}, d2[3] = {0.0, 0.0, 0.0};
  const uint64_t g0 = (uint64_t)(e0 >> 2);
  for (int k = 1; k <= a.K; ++k) {
    float tR = 0.0f, tN = 0.0f, tT = 0.0f;
#pragma unroll
    for (int j = 0; j < EPL / 4; ++j) {
      const Philox4 pn = philox_group(a.seed, g0 + j, (uint32_t)k, a.use_n);
      const uint32_t Rn[4] = {pn.w0, pn.w1, pn.w2, pn.w3};
      uint32_t uf[4];
      if (a.fwd_mode == BS_SR) {
        const Philox4 pf = philox_group(a.seed, g0 + j, (uint32_t)k, a.use_fwd);
        const uint32_t Rf[4] = {pf.w0, pf.w1, pf.w2, pf.w3};
#pragma unroll
        for (int q = 0; q < 4; ++q) uf[q] = sr_up(F[4 * j + q], Rf[q]);
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) uf[q] = (ufix >> (4 * j + q)) & 1u;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int i = 4 * j + q;
        const uint32_t u = uf[q], up = sr_up(F[i], Rn[q]);
        n[i] += u;
        np[i] += up;
        tR += u ? cR[i] : 0.0f;
        tN += up ? cN1[i] : 0.0f;
        tN += u ? cN2[i] : 0.0f;
        tN += (u & up) ? cN3[i] : 0.0f;
        tT += (u ^ up) ? cN3[i] : 0.0f;
      }
    }
    const float t3[3] = {quad_sum(tR), quad_sum(tN), 0.5f * quad_sum(tT)};
#pragma unroll
    for (int c = 0; c < 3; ++c) {
      if (k == 1) s1[c] = t3[c];
      const double dl = (double)t3[c] - s1[c];
      d1[c] += dl;
      d2[c] += dl * dl;
    }
  }
  const double iK = 1.0 / a.K;
  double mean[3], se[3];
#pragma unroll
  for (int c = 0; c < 3; ++c) {
    mean[c] = s1[c] + d1[c] * iK;
    const double var = a.K > 1 ? fmax(d2[c] - d1[c] * d1[c] * iK, 0.0) / (a.K - 1) : 0.0;
    se[c] = sqrt(var * iK);
  }
  // means over trials per element (mean r = A + (n / K) w), the reference D and the split
  double dref = 0.0, meR = 0.0, meN = 0.0;
  if (ok) {
#pragma unroll
    for (int j = 0; j < EPL / 4; ++j) {
      float ov[4], dv[4], gm[4];
      load4(j, ov, dv);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int i = 4 * j + q;
        double A, w;
        Bracket b;
        terms(ov[q], A, w, b);
        const double mr = A + (double)n[i] * iK * w, mrp = A + (double)np[i] * iK * w;
        const double mg = (double)dv[q] + beta * mr;
        dref += mg * (double)ov[q];
        meR += mr * mg;
        meN += mrp * mg;
        gm[q] = (float)mg;
      }
      *(float4*)(a.dO_mean + e0 + 4 * j) = make_float4(gm[0], gm[1], gm[2], gm[3]);
    }
  }
  dref = rowsum(dref);
  meR = rowsum(meR);
  meN = rowsum(meN);
  fixed = rowsum(fixed);
  if (ok && sub == 0) {
    const double mR = fixed + mean[0], mN = fixed + mean[1];
    a.D_ref[row] = (float)dref;
    a.dD_R[row] = (float)mR;
    a.dD_N[row] = (float)mN;
    if (a.stat_R) {
      a.stat_R[row] = (float)mR;
      a.stat_R[a.rows + row] = (float)meR;
      a.stat_R[2 * a.rows + row] = (float)(mR - meR);
      a.stat_R[3 * a.rows + row] = (float)se[0];
    }
    if (a.stat_N) {
      a.stat_N[row] = (float)mN;
      a.stat_N[a.rows + row] = (float)meN;
      a.stat_N[2 * a.rows + row] = (float)(mN - meN);
      a.stat_N[3 * a.rows + row] = (float)se[1];
    }
    if (a.T) {
      a.T[row] = (float)mean[2];
      a.T[a.rows + row] = (float)se[2];
    }
  }
}

bs_status launch_attn_l2(const AttnL2Args& a, hipStream_t st) {
  if (a.rows <= 0) return BS_OK;
  ProfScope prof("attn_l2", st);
  attn_l2_kernel<<<(unsigned)((a.rows + 63) / 64), 256, 0, st>>>(a);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status launch_attn_d(const AttnDArgs& a, hipStream_t st) {
  if (a.rows <= 0) return BS_OK;
  ProfScope prof("attn_d", st);
  attn_d_kernel<<<(unsigned)((a.rows + 63) / 64), 256, 0, st>>>(a);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

// X^T [BH][64][Sp] of up to four bf16 X [BH][S][64] (one per grid z; columns of each tile in
// fragment order, tperm): a 64 x 64 tile through LDS with 16-byte accesses on both sides; chunk
// c of tile row r sits at c ^ ((r >> 3) & 7)
struct TransposeJobs {
  const u16* x[4];
  u16* xt[4];
};
__global__ __launch_bounds__(256) void attn_transpose_kernel(TransposeJobs jobs, int S, int Sp) {
  __shared__ __attribute__((aligned(16))) u16 t[AT * AT];
  const int r0 = blockIdx.x * AT, bh = blockIdx.y;
  const u16* __restrict__ x = jobs.x[blockIdx.z];
  u16* __restrict__ xt = jobs.xt[blockIdx.z];
  const int64_t hb = (int64_t)bh * S * AT, tb = (int64_t)bh * AT * Sp;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = (threadIdx.x >> 3) + 32 * i, c = threadIdx.x & 7;
    const uint4 v = r0 + r < S ? *(const uint4*)(x + hb + (int64_t)(r0 + r) * AT + 8 * c) : make_uint4(0, 0, 0, 0);
    *(uint4*)(t + r * AT + 8 * (c ^ ((r >> 3) & 7))) = v;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int d = (threadIdx.x >> 3) + 32 * i, m = threadIdx.x & 7;  // output row d, rows 8 m .. 8 m + 7
    u16 o[8];
#pragma unroll
    for (int v = 0; v < 8; ++v) {
      const int r = tperm(8 * m + v);
      o[v] = t[r * AT + 8 * ((d >> 3) ^ ((r >> 3) & 7)) + (d & 7)];
    }
    *(uint4*)(xt + tb + (int64_t)d * Sp + r0 + 8 * m) = *(const uint4*)o;
  }
}

bs_status launch_attn_transpose(const u16* const* X, u16* const* Xt, int n, int BH, int S, int Sp, hipStream_t st) {
  if (n < 1 || n > 4) return BS_EINVAL;
  TransposeJobs jobs{};
  for (int i = 0; i < n; ++i) {
    jobs.x[i] = X[i];
    jobs.xt[i] = Xt[i];
  }
  ProfScope prof("attn_prep", st);
  attn_transpose_kernel<<<dim3((unsigned)(Sp / AT), (unsigned)BH, (unsigned)n), 256, 0, st>>>(jobs, S, Sp);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status launch_attn_split(const float* dO32, int BH, int S, int Sp, u16* const* dOp, u16* const* dOt,
                            hipStream_t st) {
  dim3 grid((unsigned)(Sp / AT), (unsigned)BH);
  ProfScope prof("attn_prep", st);
  attn_prep_kernel<float, false><<<grid, 256, 0, st>>>(dO32, S, Sp, 0, nullptr, nullptr, dOt[0], dOt[1], dOt[2],
                                                       dOp[0], dOp[1], dOp[2]);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
__global__ void attn_f16_scales_kernel(const uint32_t* sdO, const uint32_t* sV, const uint32_t* sD, float* inv) {
  if (threadIdx.x != 0) return;
  const float bound = 64.0f * amax_of_slots(sdO) * amax_of_slots(sV) + amax_of_slots(sD);
  const int e = f16_scale_exp(bound);
  inv[4] = ldexpf(1.0f, e);
  inv[5] = ldexpf(inv[2], -e);
  inv[6] = ldexpf(inv[3], -e);
}
bs_status launch_attn_f16_scales(const uint32_t* sdO, const uint32_t* sV, const uint32_t* sD, float* f16_inv,
                                 hipStream_t st) {
  if (!sdO || !sV || !sD || !f16_inv) return BS_EINVAL;
  attn_f16_scales_kernel<<<1, 64, 0, st>>>(sdO, sV, sD, f16_inv);
  BS_CHECK_LAUNCH();
  return BS_OK;
}
bs_status launch_attn_split_f16(const float* dO32, int BH, int S, int Sp, int htok, const uint32_t* slots,
                                float* inv_out, u16* const* dOp, u16* const* dOt, hipStream_t st) {
  if (!slots || !dO32 || htok < 0 || (htok > 0 && BH % htok)) return BS_EINVAL;
  dim3 grid((unsigned)(Sp / AT), (unsigned)BH);
  ProfScope prof("attn_prep", st);
  attn_prep_kernel<float, true><<<grid, 256, 0, st>>>(dO32, S, Sp, htok, slots, inv_out, dOt[0], dOt[1], nullptr,
                                                      dOp[0], dOp[1], nullptr);
  BS_CHECK_LAUNCH();
  return BS_OK;
}

bs_status launch_attn_bwd(const AttnBwdArgs& a, int B, int H, hipStream_t st) {
  dim3 grid((unsigned)(B * H), (unsigned)((a.S + AT - 1) / AT));
  ProfScope prof("attn_bwd", st);
  if (a.V16) {
    if (a.dD_R || a.dD_N || a.n_pol > 0 || !a.f16_inv || !a.Qt16 || !a.Kt16 || !a.dOp[0] || !a.dOp[1] || !a.dOt[0] ||
        !a.dOt[1])
      return BS_EINVAL;
    attn_bwd_k_kernel<2, 0, true><<<grid, 256, 0, st>>>(a);
    if (!a.k_only) attn_bwd_q_kernel<2, false, true><<<grid, 256, 0, st>>>(a);
  } else if (a.dO32) {
    if (a.dD_R || a.dD_N)
      attn_bwd_k_kernel<3, 1, false><<<grid, 256, 0, st>>>(a);
    else
      attn_bwd_k_kernel<3, 0, false><<<grid, 256, 0, st>>>(a);
    if (!a.k_only && a.n_pol > 0)
      attn_bwd_q_kernel<3, true, false><<<grid, 256, 0, st>>>(a);
    else if (!a.k_only)
      attn_bwd_q_kernel<3, false, false><<<grid, 256, 0, st>>>(a);
  } else {
    if (a.dD_R || a.dD_N)
      attn_bwd_k_kernel<1, 1, false><<<grid, 256, 0, st>>>(a);
    else
      attn_bwd_k_kernel<1, 0, false><<<grid, 256, 0, st>>>(a);
    if (!a.k_only && a.n_pol > 0)
      attn_bwd_q_kernel<1, true, false><<<grid, 256, 0, st>>>(a);
    else if (!a.k_only)
      attn_bwd_q_kernel<1, false, false><<<grid, 256, 0, st>>>(a);
  }
  BS_CHECK_LAUNCH();
  return BS_OK;
}

}  // namespace bsp
