// The decoder layer's "every use at once" check (layer_allu.h). With letter L read at every use,
// the backward's incoming gradients move away from the reference's at the uses the backward
// reaches after u2's normalization-input use; each move is formed from residual operands:
//   dh     = dOut + (u2's normalization-input backward reading z_x)         move: dh_d
//   dWo    = O_W^T dh_L          = ref + (O_W - O_q)^T dh_L + O_q^T dh_d
//   dO     = dh_L Wo^T           move: dh_d Wo^T
//   D      = rowsum(dO_L O_D)    move: rowsum(dO_d O_D) + rowsum(dO (O_D - O))
//   dQ, dK, dV: the attention backward is linear in (dO, D): its move is the backward of the moves
//   dWqkv  = u1_W^T dQKV_L       = ref + (u1_W - u1_q)^T dQKV_L + u1_q^T dQKV_d
//   du1    = dQKV_L Wqkv^T       move: dQKV_d Wqkv^T
//   dgain1, dx: gain and normalization-input uses of u1 (k_allu.h)
// The uses the backward reaches first (a's weight use, u2's gain and weight uses) see the
// reference incoming gradient whatever the letter, with the per-use check's draws: their
// estimates are the per-use ones. N draws every use's own new rounding per trial; its K trials
// are reduced by shifted fp64 sums (mean and se over trials, App. C.4).
#include "layer_allu.h"

#include <algorithm>

#include "k_allu.h"
#include "k_attn.h"
#include "k_layer.h"
#include "k_norm.h"

#define BS_TRY(x)               \
  do {                          \
    const bs_status _s = (x);   \
    if (_s != BS_OK) return _s; \
  } while (0)

namespace bsp {

namespace {

constexpr int DH = 64;
constexpr float kAttnScale = 0.125f;  // 1 / sqrt(64)
enum { G_DX = 0, G_DGAIN1, G_DWQKV, G_DWO, G_DGAIN2, G_DWG, G_DWU, G_DWD, NGRAD };
constexpr int NCOMP = 4;  // gradients formed here per trial: dx, dgain1, dWqkv, dWo
constexpr int NB = 16;    // N trials per update of the shifted sums (one read-modify-write per NB)
constexpr int KCH = 16;   // N trials per chunk of the batched weight-use contractions (a multiple of NB)
// maxima (slot arrays) of the scaled fp16 operands: per call dh, dQKV, Wo, Wqkv, V, Q, K; per pass
// the moves dh_d, dQKV_d, dO_d, D_d
enum { AM_DH, AM_DQKV, AM_WO, AM_WQKV, AM_V, AM_Q, AM_K, AM_DHD, AM_DQKVD, AM_DOD, AM_DDD, AM_N };
// their 2^-e: the splits of dh_d, dQKV_d, Wo, Wqkv, dh, dQKV, the U residuals of O and u1; then
// the attention backward's seven in its order (dO_d, V, Q, K, dS's 2^s, 2^-s-q, 2^-s-k)
enum {
  IV_DHD, IV_DQKVD, IV_WO, IV_WQKV, IV_DH, IV_DQKV, IV_RO, IV_RU,
  IV_DOD, IV_V, IV_Q, IV_K, IV_DS, IV_DKM, IV_DQM, IV_N
};

struct AlluWs {
  float *m, *l;
  u16 *Vt, *Qt, *Kt, *valT_u1, *valT_O;
  u16 *pA[2], *rows3[3], *tB[3], *dOp[3], *dOt[3];
  u16 *tH[2], *tQ[2];    // dh, dQKV as scaled two-term fp16 splits, transposed
  u16 *pAn[2], *pWn[2];  // a chunk of N trials' difference and value planes at O's and u1's weight uses
  float *dWo_n, *dWqkv_n;  // the chunk's weight-use moves [KCH][d][d], [KCH][d][3d]
  // the chunk's moves dh_d and dQKV_d as transposed two-term fp16 planes [KCH][2][d or 3d][Tp]
  // and their 2^-e: the weight uses' products with them run once per chunk, batched
  u16 *tBo, *tBq;
  float *invo, *invq;
  float *dh_d, *dO_dt, *dD, *dQ_d, *dK_d, *dV_d, *du1_d;
  u16 *Wo16, *Wqkv16, *V16;  // the weights and V as scaled fp16 (the moves' contractions)
  u16 *Q16, *K16, *Qt16, *Kt16;  // Q, K as scaled fp16 and their transposed copies
  double* gpart;
  float* delta[NCOMP];      // the passes' moves: dx, dgain1 [min(K, NB)][n] (N's trial k in row
                            // (k - 1) % NB); dWqkv, dWo [1][n] (U, R; N's are in the chunk buffers)
  float* bias[3][NCOMP];    // per letter
  float* se_n[NCOMP];       // N's se
  float *d1[NCOMP];
  double *S1[NCOMP], *S2[NCOMP];
  float *wg[3], *wu[3], *ref_g, *ref_u, *nan_buf;
  float* part;
  int64_t part_cap;
  double* sumsq_part;
  uint32_t* amax[AM_N];  // slot arrays (AMAX_SLOTS) of max |.|
  float* inv;            // [IV_N]
};

AlluWs carve_allu(Carver& c, int B, int S, int d, int H, int F, int K) {
  AlluWs w{};
  const int64_t kc = std::max(1, std::min(K, KCH));
  const int64_t T = (int64_t)B * S, Td = T * d, Tp = round_up(T > 0 ? T : 1, 64), bh = (int64_t)B * H;
  const int64_t Sp = round_up(S, 64), d3 = 3 * (int64_t)d, F2 = 2 * (int64_t)F;
  const int64_t nc[NCOMP] = {Td, d, (int64_t)d * d3, (int64_t)d * d};
  w.m = c.take<float>(bh * S);
  w.l = c.take<float>(bh * S);
  for (u16** p : {&w.Vt, &w.Qt, &w.Kt}) *p = c.take<u16>(bh * DH * Sp);
  w.valT_u1 = c.take<u16>(d * Tp);
  w.valT_O = c.take<u16>(d * Tp);
  for (int i = 0; i < 3; ++i) {
    if (i < 2) w.pA[i] = c.take<u16>(d * Tp);
    w.rows3[i] = c.take<u16>(T * std::max(F2, d3));
    w.tB[i] = c.take<u16>(d3 * Tp);
    w.dOp[i] = c.take<u16>(Td);
    w.dOt[i] = c.take<u16>(bh * DH * Sp);
  }
  for (float** p : {&w.dh_d, &w.dO_dt, &w.du1_d}) *p = c.take<float>(Td);
  w.dQ_d = c.take<float>(3 * Td);  // dQ, dK, dV of the move, one block (one max over the three)
  w.dK_d = w.dQ_d ? w.dQ_d + Td : nullptr;
  w.dV_d = w.dQ_d ? w.dQ_d + 2 * Td : nullptr;
  w.dD = c.take<float>(bh * S);
  w.Wo16 = c.take<u16>((int64_t)d * d);
  w.Wqkv16 = c.take<u16>((int64_t)d * d3);
  w.V16 = c.take<u16>(bh * S * DH);
  w.Q16 = c.take<u16>(bh * S * DH);
  w.K16 = c.take<u16>(bh * S * DH);
  w.Qt16 = c.take<u16>(bh * DH * Sp);
  w.Kt16 = c.take<u16>(bh * DH * Sp);
  for (int i = 0; i < 2; ++i) {
    w.tH[i] = c.take<u16>(d * Tp);
    w.tQ[i] = c.take<u16>(d3 * Tp);
    w.pAn[i] = c.take<u16>(kc * d * Tp);
    w.pWn[i] = c.take<u16>(kc * d * Tp);
  }
  w.dWo_n = c.take<float>(kc * d * d);
  w.dWqkv_n = c.take<float>(kc * d * d3);
  w.tBo = c.take<u16>(kc * 2 * d * Tp);
  w.tBq = c.take<u16>(kc * 2 * d3 * Tp);
  w.invo = c.take<float>(kc);
  w.invq = c.take<float>(kc);
  w.gpart = c.take<double>(3 * ((T + 15) / 16) * (int64_t)d);
  for (int i = 0; i < NCOMP; ++i) {
    w.delta[i] = c.take<float>((i < 2 ? std::max(1, std::min(K, NB)) : 1) * nc[i]);
    for (int l = 0; l < 3; ++l) w.bias[l][i] = c.take<float>(nc[i]);
    w.se_n[i] = c.take<float>(nc[i]);
    w.d1[i] = c.take<float>(nc[i]);
    w.S1[i] = c.take<double>(nc[i]);
    w.S2[i] = c.take<double>(nc[i]);
  }
  for (int l = 0; l < 3; ++l) {
    w.wg[l] = c.take<float>((int64_t)d * F);
    w.wu[l] = c.take<float>((int64_t)d * F);
  }
  w.ref_g = c.take<float>((int64_t)d * F);
  w.ref_u = c.take<float>((int64_t)d * F);
  w.nan_buf = c.take<float>(std::max<int64_t>({Td, (int64_t)d * F2, (int64_t)d * d3}));
  w.part_cap = 8 * (int64_t)d * d3;  // split-K partials of the few-tile weight contractions
  w.part = c.take<float>(w.part_cap);
  w.sumsq_part = c.take<double>(sumsq_part_size());
  {
    uint32_t* a = c.take<uint32_t>(AM_N * AMAX_SLOTS * AMAX_STRIDE);
    for (int i = 0; i < AM_N; ++i) w.amax[i] = a ? a + i * AMAX_SLOTS * AMAX_STRIDE : nullptr;
  }
  w.inv = c.take<float>(IV_N);
  return w;
}

// C = alpha * (sum of the products A_i B_j of the given term lists) for NT operands
struct Gemm {
  GemmArgs g{};
  Gemm(int M, int N, int K, int64_t lda, int64_t ldb, float* C, int64_t ldc, const float* alpha_dev) {
    g.M = M;
    g.N = N;
    g.K = K;
    g.lda = lda;
    g.ldb = ldb;
    g.ldc = ldc;
    g.alpha = 1.0f;
    g.alpha_dev = alpha_dev;
    g.C = C;
  }
  Gemm& add(const u16* const* A, int nA, const u16* const* B, int nB, int maxsum = 2) {
    ok = ok && gemm_add_products(g, A, nA, B, nB, maxsum);
    return *this;
  }
  bs_status run(float* part, int64_t cap, hipStream_t st) {
    if (!ok) return BS_EINVAL;
    g.part = part;
    g.part_cap = cap;
    return launch_gemm(g, st);
  }
  bool ok = true;
};

bs_status copy_f32(float* dst, const float* src, int64_t n, hipStream_t st) {
  if (!dst || n <= 0) return BS_OK;
  return hipMemcpyAsync(dst, src, sizeof(float) * n, hipMemcpyDeviceToDevice, st) == hipSuccess ? BS_OK : BS_EHIP;
}

}  // namespace

size_t allu_ws_size(int B, int S, int d, int H, int F, int K) {
  Carver c;
  carve_allu(c, B, S, d, H, F, K);
  return c.used();
}

bs_status allu_run(const AlluIO& io, void* ws, size_t ws_bytes, hipStream_t st) {
  const int B = io.B, S = io.S, d = io.d, H = io.H, F = io.F, K = io.K;
  const int64_t T = (int64_t)B * S, Td = T * d, Tp = round_up(T > 0 ? T : 1, 64), bh = (int64_t)B * H;
  const int64_t Sp = round_up(S, 64), rows_h = bh * S, d3 = 3 * (int64_t)d, F2 = 2 * (int64_t)F;
  const int64_t nc[NCOMP] = {Td, d, (int64_t)d * d3, (int64_t)d * d};
  Carver probe;
  carve_allu(probe, B, S, d, H, F, K);
  if (ws_bytes < probe.used()) return BS_EWORKSPACE;
  Carver c(ws, ws_bytes);
  const AlluWs w = carve_allu(c, B, S, d, H, F, K);
  const F8 f = f8_format(io.fmt);
  const float *s_u1 = io.scales + 0, *s_O = io.scales + 1, *s_u2 = io.scales + 2;

  // ---- fixed: the stores' inputs and inverse rms, du at u1 and u2, the attention rows ----
  if (!io.u1 || !io.u2 || !io.r1 || !io.r2 || !io.du1 || !io.du2) return BS_EINVAL;
  {
    const u16* src[3] = {io.V, io.Q, io.Kk};
    u16* dst[3] = {w.Vt, w.Qt, w.Kt};
    BS_TRY(launch_attn_transpose(src, dst, 3, (int)bh, S, (int)Sp, st));
    AttnArgs fa{io.Q, io.Kk, io.V, S, 1, kAttnScale, w.m, w.l, nullptr, w.Vt, (int)Sp};
    BS_TRY(launch_attn_fwd(fa, B, H, st));
  }
  NormPlaneArgs pa{};
  pa.f = f;
  pa.T = T;
  pa.d = d;
  pa.ldo = Tp;
  pa.K = 1;
  pa.nterms = 1;
  auto planes_of = [&](int mode, const float* u, const uint8_t* codes, const float* scale, u16* const* out,
                       int nterms) {
    pa.u = u;
    pa.codes = codes;
    pa.scale = scale;
    pa.nterms = nterms;
    for (int i = 0; i < 3; ++i) pa.out[i] = i < nterms ? out[i] : nullptr;
    return launch_norm_planes(mode, pa, st);
  };
  // the R and N weight uses contract fp16 operands: FP8 values (exact in fp16) against the scaled
  // two-term fp16 split of the incoming gradient and its move
  pa.f16 = 1;
  BS_TRY(planes_of(NP_VAL, io.u1, io.c_u1, s_u1, &w.valT_u1, 1));
  BS_TRY(planes_of(NP_VAL, io.Otok, io.c_Otok, s_O, &w.valT_O, 1));
  pa.f16 = 0;
  BS_TRY(launch_fill2d((float*)w.amax[0], AM_N * AMAX_SLOTS, 1, AMAX_STRIDE, 0.0f, st));
  BS_TRY(launch_amax_f32(io.dh, Td, w.amax[AM_DH], st));
  BS_TRY(launch_amax_f32(io.dqkv, 3 * Td, w.amax[AM_DQKV], st));
  BS_TRY(launch_amax_bf16(io.Wo, (int64_t)d * d, w.amax[AM_WO], st));
  BS_TRY(launch_amax_bf16(io.Wqkv, (int64_t)d * d3, w.amax[AM_WQKV], st));
  BS_TRY(launch_amax_bf16(io.V, bh * S * DH, w.amax[AM_V], st));
  BS_TRY(launch_scale_f16(io.Wo, (int64_t)d * d, w.amax[AM_WO], w.Wo16, w.inv + IV_WO, st));
  BS_TRY(launch_scale_f16(io.Wqkv, (int64_t)d * d3, w.amax[AM_WQKV], w.Wqkv16, w.inv + IV_WQKV, st));
  BS_TRY(launch_scale_f16(io.V, bh * S * DH, w.amax[AM_V], w.V16, w.inv + IV_V, st));
  BS_TRY(launch_amax_bf16(io.Q, bh * S * DH, w.amax[AM_Q], st));
  BS_TRY(launch_amax_bf16(io.Kk, bh * S * DH, w.amax[AM_K], st));
  BS_TRY(launch_scale_f16(io.Q, bh * S * DH, w.amax[AM_Q], w.Q16, w.inv + IV_Q, st));
  BS_TRY(launch_scale_f16(io.Kk, bh * S * DH, w.amax[AM_K], w.K16, w.inv + IV_K, st));
  {
    const u16* src[2] = {w.Q16, w.K16};
    u16* dst[2] = {w.Qt16, w.Kt16};
    BS_TRY(launch_attn_transpose(src, dst, 2, (int)bh, S, (int)Sp, st));
  }
  // dh and dQKV as scaled two-term fp16 splits: under N a weight use's move is
  // W_k^T g_d + (W_k - W_q)^T g (g the reference incoming gradient, g_d its move, W_k the trial's
  // new rounding, W_q the forward's), and the second products of a chunk of trials are one
  // contraction against these
  {
    MoveSrc mh{};
    mh.rows = io.dh;
    mh.ldi = d;
    BS_TRY(launch_split_move(mh, nullptr, 0, T, d, F16Scale{w.amax[AM_DH], nullptr, w.inv + IV_DH}, w.tH, nullptr, Tp,
                             nullptr, 0, st));
    MoveSrc mg{};
    mg.rows = io.dqkv;
    mg.ldi = d3;
    BS_TRY(launch_split_move(mg, nullptr, 0, T, d3, F16Scale{w.amax[AM_DQKV], nullptr, w.inv + IV_DQKV}, w.tQ, nullptr,
                             Tp, nullptr, 0, st));
  }

  // ---- one pass per letter (K per-trial passes for N) ----
  for (int l = 0; l < 3; ++l) {
    const int ntr = l == LETTER_N ? K : 1;
    for (int k = 1; k <= ntr; ++k) {
      const auto rd = [&](const float* x, const uint8_t* codes, const float* scale, uint32_t use) {
        return StoreRead{x, codes, scale, f, l, io.seed, (uint32_t)k, use};
      };
      const int slot = l == LETTER_N ? (k - 1) % NB : 0;
      const int kk = (k - 1) % KCH;  // N: the trial's index in its chunk
      if (l == LETTER_N && kk == 0) {
        // the chunk's new roundings at O's and u1's weight uses (difference and value planes), and
        // their differences' products with the reference incoming gradients, the chunk in one
        // contraction each
        const int nbk = std::min(KCH, K - k + 1);
        TrialPlaneArgs to{io.Otok, io.c_Otok, s_O, f, T, d, Tp, io.seed, 1 * 256 + 2, k, nbk, w.pAn[0]};
        to.f16 = 1;
        to.outW = w.pWn[0];
        BS_TRY(launch_trial_planes(to, st));
        TrialPlaneArgs tu{io.u1, io.c_u1, s_u1, f, T, d, Tp, io.seed, 0 * 256 + 2, k, nbk, w.pAn[1]};
        tu.f16 = 1;
        tu.outW = w.pWn[1];
        BS_TRY(launch_trial_planes(tu, st));
        Gemm go(nbk * d, d, (int)Tp, Tp, Tp, w.dWo_n, d, s_O);
        go.g.f16 = 1;
        go.g.alpha_dev2 = w.inv + IV_DH;
        BS_TRY(go.add(&w.pAn[0], 1, w.tH, 2).run(w.part, w.part_cap, st));
        Gemm gg(nbk * d, (int)d3, (int)Tp, Tp, Tp, w.dWqkv_n, d3, s_u1);
        gg.g.f16 = 1;
        gg.g.alpha_dev2 = w.inv + IV_DQKV;
        BS_TRY(gg.add(&w.pAn[1], 1, w.tQ, 2).run(w.part, w.part_cap, st));
      }
      float* dl[NCOMP];
      for (int i = 0; i < NCOMP; ++i) dl[i] = w.delta[i] + slot * nc[i];
      if (l == LETTER_N) {
        dl[2] = w.dWqkv_n + kk * nc[2];
        dl[3] = w.dWo_n + kk * nc[3];
      }
      float* dWo = dl[3];
      float* dWqkv = dl[2];
      // R: the value planes the weight uses read with the moves (the forward's roundings)
      const u16* valO = w.valT_O;
      const u16* valU = w.valT_u1;
      // u2's normalization-input use: the move of dh (and its max |.|)
      if (l != LETTER_U) {
        BS_TRY(launch_fill2d((float*)w.amax[AM_DHD], (AM_N - AM_DHD) * AMAX_SLOTS, 1, AMAX_STRIDE, 0.0f, st));
        AlluDxArgs<float> ax{io.h, io.r2, io.gain2, rd(io.u2, io.c_u2, s_u2, 2 * 256 + 3), io.du2, nullptr,
                             nullptr, T, d, w.dh_d};
        ax.amax = w.amax[AM_DHD];
        BS_TRY(launch_allu_dx(ax, st));
      }
      const F16Scale sc_o{w.amax[AM_DHD], nullptr, w.inv + IV_DHD};
      const F16Scale sc_q{w.amax[AM_DQKVD], nullptr, w.inv + IV_DQKVD};
      // O's weight use (Wo)
      if (l == LETTER_U) {
        // (u - s val)^T dh: the residual's scaled fp16 split against dh's
        pa.f16 = 1;
        pa.inv_out = w.inv + IV_RO;
        BS_TRY(planes_of(NP_RESU, io.Otok, io.c_Otok, s_O, w.pA, 2));
        Gemm gr(d, d, (int)Tp, Tp, Tp, dWo, d, w.inv + IV_RO);
        gr.g.f16 = 1;
        gr.g.alpha_dev2 = w.inv + IV_DH;
        BS_TRY(gr.add(w.pA, 2, w.tH, 2, 1).run(w.part, w.part_cap, st));
      } else {
        // dh_d's transposed planes (the weight use) and row planes (the move of dO), one read; the
        // weight use's move: val^T dh_d (N: added to the chunk's difference product)
        // (N: into the chunk's planes, the weight use's product batched at the chunk's end)
        MoveSrc mo{};
        mo.rows = w.dh_d;
        mo.ldi = d;
        F16Scale so = sc_o;
        u16* to[2] = {w.tB[0], w.tB[1]};
        if (l == LETTER_N) {
          to[0] = w.tBo + (int64_t)kk * 2 * d * Tp;
          to[1] = to[0] + d * Tp;
          so.inv_out = w.invo + kk;
        }
        BS_TRY(launch_split_move(mo, nullptr, 0, T, d, so, to, nullptr, Tp, w.rows3, d, st));
        if (l != LETTER_N) {
          Gemm gw(d, d, (int)Tp, Tp, Tp, dWo, d, s_O);
          gw.g.f16 = 1;
          gw.g.alpha_dev2 = so.inv_out;
          BS_TRY(gw.add(&valO, 1, to, 2).run(w.part, w.part_cap, st));
        }
        // the move of dO (token-major: the D use and the attention operands read it so)
        Gemm gm((int)T, d, d, d, d, w.dO_dt, d, w.inv + IV_WO);
        gm.g.f16 = 1;
        gm.g.alpha_dev2 = so.inv_out;
        gm.g.amax = w.amax[AM_DOD];
        BS_TRY(gm.add(w.rows3, 2, &w.Wo16, 1).run(nullptr, 0, st));
      }
      // the D use: U reads the original and dO does not move: no move downstream of it
      if (l == LETTER_U) {
        pa.inv_out = w.inv + IV_RU;
        BS_TRY(planes_of(NP_RESU, io.u1, io.c_u1, s_u1, w.pA, 2));
        pa.f16 = 0;
        pa.inv_out = nullptr;
        Gemm gr(d, (int)d3, (int)Tp, Tp, Tp, dWqkv, d3, w.inv + IV_RU);
        gr.g.f16 = 1;
        gr.g.alpha_dev2 = w.inv + IV_DQKV;
        BS_TRY(gr.add(w.pA, 2, w.tQ, 2, 1).run(w.part, w.part_cap, st));
        BS_TRY(launch_fill(dl[0], Td, 0.0f, st));
        BS_TRY(launch_fill(dl[1], d, 0.0f, st));
      } else {
        AlluDArgs ad{rd(io.O, io.c_O, s_O, 1 * 256 + 1), io.dOh, w.dO_dt, rows_h, w.dD};
        ad.amax = w.amax[AM_DDD];
        ad.ddo_heads = H;
        ad.ddo_S = S;
        BS_TRY(launch_allu_d(ad, st));
        // dO_d as the scaled two-term fp16 split (V as scaled fp16) for the attention backward
        BS_TRY(launch_attn_split_f16(w.dO_dt, (int)bh, S, (int)Sp, H, w.amax[AM_DOD], w.inv + IV_DOD, w.dOp, w.dOt,
                                     st));
        BS_TRY(launch_attn_f16_scales(w.amax[AM_DOD], w.amax[AM_V], w.amax[AM_DDD], w.inv + IV_DOD, st));
        AttnBwdArgs ba{};
        ba.Qt = w.Qt;
        ba.Kt = w.Kt;
        for (int i = 0; i < 3; ++i) {
          ba.dOp[i] = w.dOp[i];
          ba.dOt[i] = w.dOt[i];
        }
        ba.Sp = (int)Sp;
        ba.Q = io.Q;
        ba.K = io.Kk;
        ba.V = io.V;
        ba.dO32 = nullptr;  // the fp16 planes carry dO_d
        ba.V16 = w.V16;
        ba.Qt16 = w.Qt16;
        ba.Kt16 = w.Kt16;
        ba.f16_inv = w.inv + IV_DOD;
        ba.amax = w.amax[AM_DQKVD];  // the max of dQKV_d, for its split
        ba.m = w.m;
        ba.l = w.l;
        ba.D_ref = w.dD;
        ba.S = S;
        ba.causal = 1;
        ba.ntrial = 1;
        ba.scale = kAttnScale;
        ba.dQ_ref = w.dQ_d;
        ba.dK_ref = w.dK_d;
        ba.dV = w.dV_d;
        ba.n_pol = 0;
        BS_TRY(launch_attn_bwd(ba, B, H, st));
        // u1's weight use (Wqkv): the move of dQKV read head-major ([T][3d] token-major view), and
        // its row planes (the move of du1)
        MoveSrc mq{};
        mq.heads[0] = w.dQ_d;
        mq.heads[1] = w.dK_d;
        mq.heads[2] = w.dV_d;
        mq.S = S;
        mq.H = H;
        mq.d = d;
        F16Scale sq = sc_q;
        u16* tq[2] = {w.tB[0], w.tB[1]};
        if (l == LETTER_N) {
          tq[0] = w.tBq + (int64_t)kk * 2 * d3 * Tp;
          tq[1] = tq[0] + d3 * Tp;
          sq.inv_out = w.invq + kk;
        }
        BS_TRY(launch_split_move(mq, nullptr, 0, T, d3, sq, tq, nullptr, Tp, w.rows3, d3, st));
        if (l != LETTER_N) {
          Gemm gq(d, (int)d3, (int)Tp, Tp, Tp, dWqkv, d3, s_u1);
          gq.g.f16 = 1;
          gq.g.alpha_dev2 = sq.inv_out;
          BS_TRY(gq.add(&valU, 1, tq, 2).run(w.part, w.part_cap, st));
        }
        // the move of du1, then u1's gain and normalization-input uses
        Gemm gu((int)T, d, (int)d3, d3, d3, w.du1_d, d, w.inv + IV_WQKV);
        gu.g.f16 = 1;
        gu.g.alpha_dev2 = sq.inv_out;
        BS_TRY(gu.add(w.rows3, 2, &w.Wqkv16, 1).run(nullptr, 0, st));
        // (one pass over u1's operands for both uses)
        AlluDxArgs<u16> ax{io.x, io.r1, io.gain1, rd(io.u1, io.c_u1, s_u1, 0 * 256 + 3), io.du1, w.du1_d, w.dh_d,
                           T, d, dl[0]};
        const AlluGainDxArgs<u16> agx{ax, rd(io.u1, io.c_u1, s_u1, 0 * 256 + 1), w.gpart};
        BS_TRY(launch_allu_gain_dx(agx, st));
        BS_TRY(launch_gain_final(w.gpart, (T + 15) / 16, d, dl[1], nullptr, nullptr, st));
      }
      // the chunk's last trial: its weight uses' products val_k^T g_d,k, one batched contraction
      // each, added to the chunk's difference products
      if (l == LETTER_N && (kk == KCH - 1 || k == ntr)) {
        const int nbk = kk + 1;
        Gemm gw(d, d, (int)Tp, Tp, Tp, w.dWo_n, d, s_O);
        gw.g.f16 = 1;
        gw.g.accumulate = 1;
        gw.g.batch = nbk;
        gw.g.sA = d * Tp;
        gw.g.sB = 2 * d * Tp;
        gw.g.sC = (int64_t)d * d;
        gw.g.alpha_dev2 = w.invo;
        gw.g.s_alpha2 = 1;
        const u16* tbo[2] = {w.tBo, w.tBo + d * Tp};
        BS_TRY(gw.add(&w.pWn[0], 1, tbo, 2).run(nullptr, 0, st));
        Gemm gq(d, (int)d3, (int)Tp, Tp, Tp, w.dWqkv_n, d3, s_u1);
        gq.g.f16 = 1;
        gq.g.accumulate = 1;
        gq.g.batch = nbk;
        gq.g.sA = d * Tp;
        gq.g.sB = 2 * d3 * Tp;
        gq.g.sC = (int64_t)d * d3;
        gq.g.alpha_dev2 = w.invq;
        gq.g.s_alpha2 = 1;
        const u16* tbq[2] = {w.tBq, w.tBq + d3 * Tp};
        BS_TRY(gq.add(&w.pWn[1], 1, tbq, 2).run(nullptr, 0, st));
      }
      // this pass's moves: the letter's bias (U, R), or N's trials k - slot .. k, in order, once
      // NB of them (or the last) are in
      for (int i = 0; i < NCOMP; ++i) {
        if (l == LETTER_N) {
          if (slot == NB - 1 || k == ntr)
            BS_TRY(launch_trial_accum(dl[i] - (int64_t)slot * nc[i], slot + 1, k - slot, nc[i], w.d1[i], w.S1[i],
                                      w.S2[i], st));
        } else {
          BS_TRY(copy_f32(w.bias[l][i], dl[i], nc[i], st));
        }
      }
    }
  }
  for (int i = 0; i < NCOMP; ++i) {
    BS_TRY(launch_trial_mean(w.d1[i], w.S1[i], K, nc[i], w.bias[LETTER_N][i], st));
    BS_TRY(launch_trial_se(w.S1[i], w.S2[i], K, nc[i], w.se_n[i], st));
  }

  // ---- every gradient's bias and se per letter, and the table ----
  const int64_t dF = (int64_t)d * F, Fd = (int64_t)F * d;
  BS_TRY(launch_split_cols(io.ref[G_DWG], w.ref_g, w.ref_u, d, F, st));
  for (int l = 0; l < 3; ++l)
    BS_TRY(launch_split_cols(io.wgu_bias + (int64_t)l * d * F2, w.wg[l], w.wu[l], d, F, st));
  BS_TRY(launch_fill(w.nan_buf, std::max<int64_t>({Td, (int64_t)d * F2, (int64_t)d * d3}), __builtin_nanf(""),
                     st));
  const int64_t n_of[NGRAD] = {Td, d, (int64_t)d * d3, (int64_t)d * d, d, dF, dF, Fd};
  const float* ref_of[NGRAD] = {io.ref[G_DX], io.ref[G_DGAIN1], io.ref[G_DWQKV], io.ref[G_DWO], io.ref[G_DGAIN2],
                                w.ref_g, w.ref_u, io.ref[G_DWD]};
  SumsqBatch batch{};
  const float* const kZero = (const float*)1;
  const float* const kNaN = (const float*)2;
  for (int gi = 0; gi < NGRAD; ++gi)
    for (int l = 0; l < 3; ++l) {
      const float* bias = nullptr;
      const float* se = l == LETTER_N ? kNaN : kZero;
      switch (gi) {
        case G_DX: bias = w.bias[l][0]; break;
        case G_DGAIN1: bias = w.bias[l][1]; break;
        case G_DWQKV: bias = w.bias[l][2]; break;
        case G_DWO: bias = w.bias[l][3]; break;
        case G_DGAIN2: bias = io.g2_bias + (int64_t)l * d; break;
        case G_DWG: bias = w.wg[l]; break;
        case G_DWU: bias = w.wu[l]; break;
        default: bias = io.wd_bias + (int64_t)l * Fd; break;
      }
      if (l == LETTER_N) {
        if (gi <= G_DWO) se = w.se_n[gi];
        if (gi == G_DGAIN2) se = io.g2_se + (int64_t)l * d;
      }
      BS_TRY(copy_f32(io.bias[l][gi], bias, n_of[gi], st));
      if (io.se[l][gi]) {
        if (se == kZero)
          BS_TRY(launch_fill(io.se[l][gi], n_of[gi], 0.0f, st));
        else
          BS_TRY(copy_f32(io.se[l][gi], se == kNaN ? w.nan_buf : se, n_of[gi], st));
      }
      if (io.table) {
        double* out = io.table + ((int64_t)gi * 3 + l) * 3;
        batch.job[batch.count++] = SumsqJob{bias, n_of[gi], out};
        batch.job[batch.count++] = SumsqJob{ref_of[gi], n_of[gi], out + 1};
        if (se == kZero)
          batch.job[batch.count++] = SumsqJob{nullptr, 1, out + 2};
        else if (se == kNaN)
          batch.job[batch.count++] = SumsqJob{nullptr, 0, out + 2};
        else
          batch.job[batch.count++] = SumsqJob{se, n_of[gi], out + 2};
      }
    }
  if (io.table) BS_TRY(launch_sumsq_batch(batch, w.sumsq_part, st));
  return BS_OK;
}

}  // namespace bsp
