// C-ABI entry point of the decoder layer: forward (or the caller's realized forward), the
// straight-through reference backward, and the per-use check of each of the four stores.
#include "attn_run.h"
#include "bsp_kernels.h"
#include "k_layer.h"
#include "k_norm.h"
#include "layer_allu.h"
#include "norm_run.h"

using namespace bsp;

#define BS_TRY(x)               \
  do {                          \
    const bs_status _s = (x);   \
    if (_s != BS_OK) return _s; \
  } while (0)

namespace {

// ------------------------------------------------------------------------------------
// Weight use of a stored tensor X [T, k] (Sec. 4.1): dW = X_read^T dY [k, n] under U (the
// original), R (the forward's rounding: no bias) and N (mean of K new roundings at the store's
// scale, trials 1..K, use id `use`, token-major element order). The biases are contractions of
// residual operands with dY: U adds (X - s val(C))^T dY, N adds (s/K)(n_up - K h)^T dY. With
// se_n set, N's se over trials by the per-trial path: trial k's residual s(val(C_k) - val(C))
// in its own contraction (trials stacked along the output rows), shifted fp64 sums over trials.
// ------------------------------------------------------------------------------------
struct WeightUseIO {
  const float* Xs;       // [T][k] fp32 store input
  const uint8_t* codes;  // [T][k] forward codes
  const float* scale;    // device s
  int fmt;
  const void* dY;        // [T][n], dtype gt
  bs_dtype gt;
  int64_t T, k, n;
  int K;
  uint64_t seed;
  uint32_t use;
  float* dW_ref;         // [k][n]
  float* bias;           // [3][k][n] for U, R, N
  float* se_n = nullptr; // [k][n] nullable: N's se (the per-trial path)
  const float* amax_x = nullptr;  // device max |X| (the store's amax; bounds the U residual)
};

// trials per per-trial contraction (stacked along the output rows)
inline int wu_trial_batch(int K) { return K < 8 ? K : 8; }

struct WeightUseWs {
  u16 *dyT[3], *valT, *res[3], *counts;
  float *bias_u, *bias_n, *gpart;
  int64_t gpart_cap;
  u16* tplanes;  // per-trial residual planes [BT][k][Tp]
  float *tdelta, *td1;
  double *tS1, *tS2;
  uint32_t* am;  // dY's max (slot array) for its fp16 split
  float* inv;    // 2^-e of dY's split and of the U residual's
};

// an fp32 incoming gradient enters as a scaled two-term fp16 split against exact fp16 operands
// (FP8 values, the U residual's split, the N residual) when K <= 256
inline bool wu_f16(bs_dtype gt, int K) { return gt == BS_F32 && K <= 256; }

WeightUseWs carve_wu(Carver& c, int64_t T, int64_t k, int64_t n, int K = 1, bool se = false) {
  WeightUseWs w{};
  const int64_t Tp = round_up(T > 0 ? T : 1, 64);
  for (int i = 0; i < 3; ++i) w.dyT[i] = c.take<u16>(n * Tp);
  w.valT = c.take<u16>(k * Tp);
  for (int i = 0; i < 3; ++i) w.res[i] = c.take<u16>(k * Tp);
  w.counts = c.take<u16>(T * k);
  w.bias_u = c.take<float>(k * n);
  w.bias_n = c.take<float>(k * n);
  w.gpart_cap = 16 * k * n;  // split-K partials: the long-T contraction has few output tiles
  w.gpart = c.take<float>(w.gpart_cap);
  if (se) {
    const int bt = wu_trial_batch(K);
    w.tplanes = c.take<u16>(bt * k * Tp);
    w.tdelta = c.take<float>(bt * k * n);
    w.td1 = c.take<float>(k * n);
    w.tS1 = c.take<double>(k * n);
    w.tS2 = c.take<double>(k * n);
  }
  w.am = c.take<uint32_t>(AMAX_SLOTS * AMAX_STRIDE);
  w.inv = c.take<float>(2);
  return w;
}

bs_status weight_use_run(const WeightUseIO& io, void* ws, size_t ws_bytes, hipStream_t st) {
  const bool se = io.se_n != nullptr;
  Carver probe;
  carve_wu(probe, io.T, io.k, io.n, io.K, se);
  if (ws_bytes < probe.used()) return BS_EWORKSPACE;
  Carver c(ws, ws_bytes);
  const WeightUseWs w = carve_wu(c, io.T, io.k, io.n, io.K, se);
  const int64_t Tp = round_up(io.T > 0 ? io.T : 1, 64);
  const bool h16 = wu_f16(io.gt, io.K);
  const int nt = h16 ? 2 : (io.gt == BS_F32 ? 3 : 1);
  if (h16) {
    BS_TRY(launch_fill2d((float*)w.am, AMAX_SLOTS, 1, AMAX_STRIDE, 0.0f, st));
    BS_TRY(launch_amax_f32((const float*)io.dY, io.T * io.n, w.am, st));
    MoveSrc ms{};
    ms.rows = (const float*)io.dY;
    ms.ldi = io.n;
    BS_TRY(launch_split_move(ms, nullptr, 0, io.T, io.n, F16Scale{w.am, nullptr, w.inv + 0}, w.dyT, nullptr, Tp,
                             nullptr, 0, st));
  } else {
    BS_TRY(launch_planes(io.dY, io.gt, io.T, io.n, io.n, true, w.dyT, nt, Tp, 1.0f, st));
  }
  NormPlaneArgs pa{};
  pa.u = io.Xs;
  pa.codes = io.codes;
  pa.scale = io.scale;
  pa.K = io.K;
  pa.f = f8_format(io.fmt);
  pa.T = io.T;
  pa.d = io.k;
  pa.ldo = Tp;
  pa.f16 = h16;
  pa.amax_u = io.amax_x;
  pa.inv_out = h16 ? w.inv + 1 : nullptr;
  // the N residual (up-count difference times a step) exact in fp16; E5M2's steps scaled by 2^-8
  pa.resn_scale = io.fmt == BS_E5M2 ? 0x1p-8f : 1.0f;
  auto gemm = [&](u16* const* A, int nA, float* C, float alpha, const float* alpha_dev) -> bs_status {
    GemmArgs g{};
    g.M = (int)io.k;
    g.N = (int)io.n;
    g.K = (int)Tp;
    g.lda = Tp;
    g.ldb = Tp;
    g.ldc = io.n;
    g.alpha = alpha;
    g.alpha_dev = alpha_dev;
    g.C = C;
    g.part = w.gpart;
    g.part_cap = w.gpart_cap;
    if (h16) {
      g.f16 = 1;
      g.alpha_dev2 = w.inv + 0;
    }
    if (!gemm_add_products(g, A, nA, w.dyT, nt, h16 && nA == 2 ? 1 : 2)) return BS_EINVAL;
    return launch_gemm(g, st);
  };
  // reference: s val(C)^T dY
  pa.out[0] = w.valT;
  pa.nterms = 1;
  BS_TRY(launch_norm_planes(NP_VAL, pa, st));
  BS_TRY(gemm(&w.valT, 1, io.dW_ref, 1.0f, io.scale));
  // U: residual X - s val(C) in three exact bf16 terms (or its scaled two-term fp16 split)
  for (int i = 0; i < 3; ++i) pa.out[i] = w.res[i];
  pa.nterms = h16 ? 2 : 3;
  BS_TRY(launch_norm_planes(NP_RESU, pa, st));
  BS_TRY(gemm(w.res, pa.nterms, w.bias_u, 1.0f, h16 ? w.inv + 1 : nullptr));
  // N: up counts over the K new roundings, residual (n_up - K h) step
  const FreshArgs<float> fa{io.Xs, io.T, io.k, pa.f, io.scale, io.seed, io.use, io.K, w.counts, nullptr, nullptr,
                            nullptr};
  BS_TRY(launch_fresh_count_t(fa, FC_COUNT, st));
  pa.counts = w.counts;
  pa.out[2] = nullptr;
  pa.nterms = io.K > 256 ? 2 : 1;
  BS_TRY(launch_norm_planes(NP_RESN, pa, st));
  BS_TRY(gemm(w.res, pa.nterms, w.bias_n, 1.0f / (float)io.K / (h16 ? pa.resn_scale : 1.0f), io.scale));
  const int64_t kn = io.k * io.n;
  const float* b[3] = {w.bias_u, nullptr, w.bias_n};
  for (int l = 0; l < 3; ++l)
    BS_TRY(launch_combine(io.dW_ref, b[l], nullptr, kn, nullptr, io.bias + l * kn, nullptr, st));
  if (se) {
    const int bt = wu_trial_batch(io.K);
    for (int k0 = 1; k0 <= io.K; k0 += bt) {
      const int nb = io.K - k0 + 1 < bt ? io.K - k0 + 1 : bt;
      TrialPlaneArgs ta{io.Xs, io.codes, io.scale, pa.f, io.T, io.k, Tp, io.seed, io.use, k0, nb, w.tplanes};
      ta.f16 = h16;
      BS_TRY(launch_trial_planes(ta, st));
      GemmArgs g{};
      g.M = (int)(nb * io.k);
      g.N = (int)io.n;
      g.K = (int)Tp;
      g.lda = Tp;
      g.ldb = Tp;
      g.ldc = io.n;
      g.alpha = 1.0f;
      g.alpha_dev = io.scale;
      g.C = w.tdelta;
      g.part = w.gpart;
      g.part_cap = w.gpart_cap;
      if (h16) {
        g.f16 = 1;
        g.alpha_dev2 = w.inv + 0;
      }
      const u16* A0 = w.tplanes;
      if (!gemm_add_products(g, &A0, 1, w.dyT, nt)) return BS_EINVAL;
      BS_TRY(launch_gemm(g, st));
      BS_TRY(launch_trial_accum(w.tdelta, nb, k0, kn, w.td1, w.tS1, w.tS2, st));
    }
    BS_TRY(launch_trial_se(w.tS1, w.tS2, io.K, kn, io.se_n, st));
  }
  return BS_OK;
}

// ------------------------------------------------------------------------------------
// workspace of the layer
// ------------------------------------------------------------------------------------
constexpr int DH = 64;
constexpr int NPOL = 4;  // U/U, R/R, N/N, and U with the R reading at the normalization input

struct NormEst {
  float *g_bias, *g_se, *w_bias, *x_bias;  // [NPOL][d], [NPOL][d], [NPOL][d*n], [NPOL][T*d]
  float* w_se = nullptr;                   // [NPOL][d*n] (the per-use se option)
};

struct LayerWs {
  float *qkv, *O, *Otok, *h, *gh, *a, *da, *dgh, *dxn2, *dh, *dOtok, *dOh, *dQ, *dK, *dV, *dqkv, *dxn1, *dWgu;
  float *dWqkv, *dWo, *dWd, *dgain1, *dgain2, *dx, *scales;
  u16 *Q, *K, *V, *Wgu, *WoT, *Oval;
  uint8_t *c_u1, *c_O, *c_Otok, *c_u2, *c_a;
  NormEst e1, e2;
  float *q_bias, *q_se, *k_bias, *wo_bias, *wd_bias;
  float *k_se = nullptr, *wo_se = nullptr, *wd_se = nullptr;  // the per-use se option
  double* part;
  bs_diag* diag;
  void* sub;
  size_t sub_bytes;
  void* allu;  // the every-use-at-once check (nullptr when not asked for)
  size_t allu_bytes;
  float *n_u1, *n_u2, *n_du1, *n_du2, *n_r1, *n_r2;  // every use at once: u, du, rstd of u1 and u2
};

size_t sub_ws_size(int B, int S, int d, int H, int F, int K, bool se) {
  const int64_t T = (int64_t)B * S;
  size_t m = norm_ws_size(T, d, 3 * (int64_t)d, K);
  m = std::max(m, norm_ws_size(T, d, 2 * (int64_t)F, K));
  m = std::max(m, attn_ws_size(B, H, S, DH, K, se));
  Carver c1, c2, c3;
  carve_wu(c1, T, d, d, K, se);
  carve_wu(c2, T, F, d, K, se);
  for (int i = 0; i < 3; ++i) c3.take<u16>(T * d);
  return std::max(m, std::max(c1.used(), std::max(c2.used(), c3.used())));
}

NormEst carve_est(Carver& c, int64_t T, int64_t d, int64_t n) {
  NormEst e{};
  e.g_bias = c.take<float>(NPOL * d);
  e.g_se = c.take<float>(NPOL * d);
  e.w_bias = c.take<float>(NPOL * d * n);
  e.x_bias = c.take<float>(NPOL * T * d);
  return e;
}

LayerWs carve_layer(Carver& c, int B, int S, int d, int H, int F, int K, bool all_uses, bool se) {
  LayerWs w{};
  const int64_t T = (int64_t)B * S, Td = T * d, TF = T * (int64_t)F;
  w.qkv = c.take<float>(3 * Td);
  w.O = c.take<float>(Td);
  w.Otok = c.take<float>(Td);
  w.h = c.take<float>(Td);
  w.gh = c.take<float>(2 * TF);
  w.a = c.take<float>(TF);
  w.da = c.take<float>(TF);
  w.dgh = c.take<float>(2 * TF);
  w.dxn2 = c.take<float>(Td);
  w.dh = c.take<float>(Td);
  w.dOtok = c.take<float>(Td);
  w.dOh = c.take<float>(Td);
  w.dQ = c.take<float>(Td);
  w.dK = c.take<float>(Td);
  w.dV = c.take<float>(Td);
  w.dqkv = c.take<float>(3 * Td);
  w.dxn1 = c.take<float>(Td);
  w.dWgu = c.take<float>((int64_t)d * 2 * F);
  w.dWqkv = c.take<float>((int64_t)d * 3 * d);
  w.dWo = c.take<float>((int64_t)d * d);
  w.dWd = c.take<float>((int64_t)F * d);
  w.dgain1 = c.take<float>(d);
  w.dgain2 = c.take<float>(d);
  w.dx = c.take<float>(Td);
  w.scales = c.take<float>(4);
  w.Q = c.take<u16>(Td);
  w.K = c.take<u16>(Td);
  w.V = c.take<u16>(Td);
  w.Wgu = c.take<u16>((int64_t)d * 2 * F);
  w.WoT = c.take<u16>((int64_t)d * d);
  w.Oval = c.take<u16>(Td);
  w.c_u1 = c.take<uint8_t>(Td);
  w.c_O = c.take<uint8_t>(Td);
  w.c_Otok = c.take<uint8_t>(Td);
  w.c_u2 = c.take<uint8_t>(Td);
  w.c_a = c.take<uint8_t>(TF);
  w.e1 = carve_est(c, T, d, 3 * (int64_t)d);
  w.e2 = carve_est(c, T, d, 2 * (int64_t)F);
  w.q_bias = c.take<float>(3 * Td);
  w.q_se = c.take<float>(3 * Td);
  w.k_bias = c.take<float>(3 * Td);
  w.wo_bias = c.take<float>(3 * (int64_t)d * d);
  w.wd_bias = c.take<float>(3 * (int64_t)F * d);
  if (se) {  // the per-use se under N of the weight uses and of dK
    w.e1.w_se = c.take<float>(NPOL * (int64_t)d * 3 * d);
    w.e2.w_se = c.take<float>(NPOL * (int64_t)d * 2 * F);
    w.k_se = c.take<float>(3 * Td);
    w.wo_se = c.take<float>((int64_t)d * d);
    w.wd_se = c.take<float>((int64_t)F * d);
  }
  w.part = c.take<double>(sumsq_part_size());
  w.diag = c.take<bs_diag>(4);
  w.sub_bytes = sub_ws_size(B, S, d, H, F, K, se);
  w.sub = c.take<char>(w.sub_bytes);
  if (all_uses) {
    w.allu_bytes = allu_ws_size(B, S, d, H, F, K);
    w.allu = c.take<char>(w.allu_bytes);
    // the normalization operands the per-use runs hand to the every-use check
    for (float** q : {&w.n_u1, &w.n_u2, &w.n_du1, &w.n_du2}) *q = c.take<float>(Td);
    for (float** q : {&w.n_r1, &w.n_r2}) *q = c.take<float>(T);
  }
  return w;
}

bool layer_shape_ok(int B, int S, int d, int H, int F) {
  if (B < 1 || S < 1 || H < 1 || d != DH * H || d > 8192 || F < 8 || (F & 7)) return false;
  const int64_t T = (int64_t)B * S;
  return T <= 0x7FFFFFFF / 4 && T * (int64_t)F <= ((int64_t)1 << 40) && (int64_t)B * H <= 65535;
}

}  // namespace

extern "C" {

size_t bs_decoder_layer_workspace_size(int B, int S, int d, int H, int F, int K, int options) {
  if (!layer_shape_ok(B, S, d, H, F) || K < 1 || K > 4096) return 0;
  Carver c;
  carve_layer(c, B, S, d, H, F, K, (options & BS_LAYER_ALL_USES) != 0, (options & BS_LAYER_PER_USE_SE) != 0);
  return c.used();
}

bs_status bs_decoder_layer_policy(const void* x, const bs_layer_weights* wt, const void* dOut, int B, int S, int d,
                                  int H, int F, float eps, bs_fp8 fmt, bs_round fwd_mode, int K, uint64_t seed,
                                  const bs_layer_forward* fixed, bs_layer_grads grads, bs_layer_stores stores,
                                  double* table, const bs_layer_all* all, int per_use_se, bs_diag* diags, void* ws,
                                  size_t ws_bytes, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  const bool se = per_use_se != 0;
  const int options = (all ? BS_LAYER_ALL_USES : 0) | (se ? BS_LAYER_PER_USE_SE : 0);
  if (!x || !wt || !dOut || !table || !wt->gain1 || !wt->Wqkv || !wt->Wo || !wt->gain2 || !wt->Wg || !wt->Wu ||
      !wt->Wd)
    return BS_EINVAL;
  if (K < 1 || K > 4096 || !(eps >= 0.0f)) return BS_EINVAL;
  if ((fmt != BS_E4M3 && fmt != BS_E5M2) || (fwd_mode != BS_RNE && fwd_mode != BS_SR)) return BS_EINVAL;
  if (!layer_shape_ok(B, S, d, H, F)) return BS_ESHAPE;
  if (fixed && (!fixed->Q || !fixed->K || !fixed->V || !fixed->O || !fixed->h || !fixed->gh || !fixed->a))
    return BS_EINVAL;
  if (!ws || ((uintptr_t)ws & 255) || ws_bytes < bs_decoder_layer_workspace_size(B, S, d, H, F, K, options))
    return BS_EWORKSPACE;
  Carver c(ws, ws_bytes);
  const LayerWs w = carve_layer(c, B, S, d, H, F, K, all != nullptr, se);
  const int64_t T = (int64_t)B * S, Td = T * d, TF = T * (int64_t)F;
  const int64_t d3d = (int64_t)d * 3 * d, d2F = (int64_t)d * 2 * F, dd = (int64_t)d * d, Fd = (int64_t)F * d;
  bs_diag* dg = diags ? diags : w.diag;
  float* scales = stores.scales ? stores.scales : w.scales;
  uint8_t* c_u1 = stores.u1 ? stores.u1 : w.c_u1;
  uint8_t* c_O = stores.O ? stores.O : w.c_O;
  uint8_t* c_u2 = stores.u2 ? stores.u2 : w.c_u2;
  uint8_t* c_a = stores.a ? stores.a : w.c_a;
  float* dWqkv = grads.dWqkv ? grads.dWqkv : w.dWqkv;
  float* dWo = grads.dWo ? grads.dWo : w.dWo;
  float* dWd = grads.dWd ? grads.dWd : w.dWd;
  float* dgain1 = grads.dgain1 ? grads.dgain1 : w.dgain1;
  float* dgain2 = grads.dgain2 ? grads.dgain2 : w.dgain2;
  const bs_norm_policy npol[NPOL] = {{BS_READ_U, BS_READ_U, BS_READ_U, 0},
                                     {BS_READ_R, BS_READ_R, BS_READ_U, 0},
                                     {BS_READ_N, BS_READ_N, BS_READ_U, 0},
                                     {BS_READ_U, BS_READ_U, BS_READ_R, 0}};
  const bs_read apol[3] = {BS_READ_U, BS_READ_R, BS_READ_N};
  const float c_attn = 0.125f;  // 1/sqrt(64)
  const bs_est none{};

  // ---------------- forward: the four stores ----------------
  // store u1 (and QKV when the forward is computed here)
  const NormIO f1{x, BS_BF16, wt->gain1, wt->Wqkv, BS_BF16, nullptr, BS_F32, T, d, 3 * (int64_t)d, eps, fmt, fwd_mode,
                  nullptr, 0, K, seed, 0, fixed ? nullptr : w.qkv, c_u1, scales + 0, nullptr, nullptr, nullptr,
                  none, none, none, dg + 0};
  BS_TRY(norm_run(f1, w.sub, w.sub_bytes, st));
  const void *Q = w.Q, *Kk = w.K, *V = w.V;
  if (fixed) {
    Q = fixed->Q;
    Kk = fixed->K;
    V = fixed->V;
  } else {
    BS_TRY(launch_qkv_heads(w.qkv, B, S, H, DH, w.Q, w.K, w.V, st));
  }
  // store O (head-major), its token-major copies for the weight use
  const float* O = fixed ? fixed->O : w.O;
  const AttnIO fa{Q, Kk, V, nullptr, nullptr, B, H, S, DH, 1, c_attn, fixed ? fixed->O : nullptr, fmt, fwd_mode,
                  nullptr, 0, K, seed, 1, fixed ? nullptr : w.O, c_O, scales + 1, nullptr, nullptr, nullptr, nullptr,
                  none, none, dg + 1};
  BS_TRY(attn_run(fa, w.sub, w.sub_bytes, st));
  BS_TRY(launch_heads_tokens_u8(c_O, w.c_Otok, B, S, H, DH, st));
  BS_TRY(launch_heads_tokens_f32(O, w.Otok, B, S, H, DH, true, st));
  const float* h = fixed ? fixed->h : w.h;
  if (!fixed) {  // h = x + s_O val(C_O) Wo
    BS_TRY(launch_bf16_to_f32((const u16*)x, w.h, Td, st));
    BS_TRY(launch_val_rows(w.c_Otok, Td, fmt, w.Oval, st));
    BS_TRY(launch_planes(wt->Wo, BS_BF16, d, d, d, true, &w.WoT, 1, d, 1.0f, st));
    GemmArgs g{};
    g.A[0] = w.Oval;
    g.B[0] = w.WoT;
    g.nseg = 1;
    g.M = (int)T;
    g.N = d;
    g.K = d;
    g.lda = d;
    g.ldb = d;
    g.ldc = d;
    g.alpha = 1.0f;
    g.alpha_dev = scales + 1;
    g.accumulate = 1;
    g.C = w.h;
    BS_TRY(launch_gemm(g, st));
  }
  // store u2 (and [g | hh])
  BS_TRY(launch_concat_cols((const u16*)wt->Wg, (const u16*)wt->Wu, w.Wgu, d, F, F, st));
  const NormIO f2{h, BS_F32, wt->gain2, w.Wgu, BS_BF16, nullptr, BS_F32, T, d, 2 * (int64_t)F, eps, fmt, fwd_mode,
                  nullptr, 0, K, seed, 2, fixed ? nullptr : w.gh, c_u2, scales + 2, nullptr, nullptr, nullptr,
                  none, none, none, dg + 2};
  BS_TRY(norm_run(f2, w.sub, w.sub_bytes, st));
  const float* gh = fixed ? fixed->gh : w.gh;
  const float* a = fixed ? fixed->a : w.a;
  if (!fixed) BS_TRY(launch_swiglu_fwd(w.gh, w.a, T, F, st));
  // store a
  BS_TRY(launch_store(a, BS_F32, TF, fmt, fwd_mode, seed, 0, 3 * 256, nullptr, c_a, scales + 3, dg + 3, st, false));

  // ---------------- reference backward, each use checked where its gradient arrives ----------------
  // store a, weight use of Wd (incoming gradient dOut)
  const WeightUseIO wa{a, c_a, scales + 3, fmt, dOut, BS_BF16, T, F, d, K, seed, 3 * 256 + 2, dWd, w.wd_bias,
                       w.wd_se};
  BS_TRY(weight_use_run(wa, w.sub, w.sub_bytes, st));
  {  // da = dOut Wd^T
    GemmArgs g{};
    g.A[0] = (const u16*)dOut;
    g.B[0] = (const u16*)wt->Wd;
    g.nseg = 1;
    g.M = (int)T;
    g.N = F;
    g.K = d;
    g.lda = d;
    g.ldb = d;
    g.ldc = F;
    g.alpha = 1.0f;
    g.C = w.da;
    BS_TRY(launch_gemm(g, st));
  }
  BS_TRY(launch_swiglu_bwd(w.da, gh, w.dgh, T, F, st));
  // store u2: gain, weight ([Wg | Wu]) and normalization-input uses (incoming gradient [dg | dhh])
  NormIO b2{h, BS_F32, wt->gain2, w.Wgu, BS_BF16, w.dgh, BS_F32, T, d, 2 * (int64_t)F, eps, fmt, fwd_mode,
            npol, NPOL, K, seed, 2, nullptr, c_u2, scales + 2, dgain2, w.dWgu, w.dxn2,
            bs_est{nullptr, w.e2.g_bias, w.e2.g_se}, bs_est{nullptr, w.e2.w_bias, w.e2.w_se},
            bs_est{nullptr, w.e2.x_bias, nullptr}, dg + 2};
  if (all) {
    b2.u_out = w.n_u2;
    b2.rstd_out = w.n_r2;
    b2.du_out = w.n_du2;
  }
  BS_TRY(norm_run(b2, w.sub, w.sub_bytes, st));
  BS_TRY(launch_add(dOut, BS_BF16, w.dxn2, w.dh, Td, st));
  // store O, weight use of Wo (incoming gradient dh)
  WeightUseIO wo{w.Otok, w.c_Otok, scales + 1, fmt, w.dh, BS_F32, T, d, d, K, seed, 1 * 256 + 2, dWo,
                 w.wo_bias, w.wo_se};
  wo.amax_x = &dg[1].amax;  // the store of O's max |O|
  BS_TRY(weight_use_run(wo, w.sub, w.sub_bytes, st));
  {  // dO (token-major) = dh Wo^T with dh in three exact bf16 terms
    Carver cs(w.sub, w.sub_bytes);
    u16* dh3[3] = {cs.take<u16>(Td), cs.take<u16>(Td), cs.take<u16>(Td)};
    BS_TRY(launch_planes(w.dh, BS_F32, T, d, d, false, dh3, 3, d, 1.0f, st));
    const u16* Wop = (const u16*)wt->Wo;
    GemmArgs g{};
    g.M = (int)T;
    g.N = d;
    g.K = d;
    g.lda = d;
    g.ldb = d;
    g.ldc = d;
    g.alpha = 1.0f;
    g.C = w.dOtok;
    gemm_add_products(g, dh3, 3, &Wop, 1);
    BS_TRY(launch_gemm(g, st));
  }
  // store O, D use: the attention backward with the fp32 incoming gradient
  BS_TRY(launch_heads_tokens_f32(w.dOtok, w.dOh, B, S, H, DH, false, st));
  const AttnIO ba{Q, Kk, V, nullptr, w.dOh, B, H, S, DH, 1, c_attn, O, fmt, fwd_mode, apol, 3, K, seed, 1, nullptr,
                  c_O, scales + 1, w.dQ, w.dK, w.dV, nullptr, bs_est{nullptr, w.q_bias, w.q_se},
                  bs_est{nullptr, w.k_bias, w.k_se}, dg + 1};
  BS_TRY(attn_run(ba, w.sub, w.sub_bytes, st));
  BS_TRY(launch_dqkv_tokens(w.dQ, w.dK, w.dV, w.dqkv, B, S, H, DH, st));
  // store u1: gain, weight (Wqkv) and normalization-input uses (incoming gradient dQKV)
  NormIO b1{x, BS_BF16, wt->gain1, wt->Wqkv, BS_BF16, w.dqkv, BS_F32, T, d, 3 * (int64_t)d, eps, fmt, fwd_mode,
            npol, NPOL, K, seed, 0, nullptr, c_u1, scales + 0, dgain1, dWqkv, w.dxn1,
            bs_est{nullptr, w.e1.g_bias, w.e1.g_se}, bs_est{nullptr, w.e1.w_bias, w.e1.w_se},
            bs_est{nullptr, w.e1.x_bias, nullptr}, dg + 0};
  if (all) {
    b1.u_out = w.n_u1;
    b1.rstd_out = w.n_r1;
    b1.du_out = w.n_du1;
  }
  BS_TRY(norm_run(b1, w.sub, w.sub_bytes, st));
  float* dx = grads.dx ? grads.dx : w.dx;
  if (grads.dx || all) BS_TRY(launch_add(w.dh, BS_F32, w.dxn1, dx, Td, st));
  if (grads.dWg || grads.dWu) BS_TRY(launch_split_cols(w.dWgu, grads.dWg, grads.dWu, d, F, st));

  // ---------------- table: sums of squares (fp64, fixed order), one batch ----------------
  // se argument: a device array, or kZero (the letter has no spread) / kNaN (no estimate here)
  const float* const kZero = (const float*)1;
  const float* const kNaN = (const float*)2;
  SumsqBatch batch{};
  auto put = [&](const float* x, int64_t n, double* out) { batch.job[batch.count++] = SumsqJob{x, n, out}; };
  auto row = [&](int r, int l, const float* bias, const float* ref, const float* se, int64_t n) {
    double* out = table + ((int64_t)r * 3 + l) * 3;
    if (!bias) {
      for (int q = 0; q < 3; ++q) put(nullptr, 0, out + q);
      return;
    }
    put(bias, n, out + 0);
    put(ref, n, out + 1);
    if (se == kZero)
      put(nullptr, 1, out + 2);
    else if (se == kNaN)
      put(nullptr, 0, out + 2);
    else
      put(se, n, out + 2);
  };
  for (int l = 0; l < 3; ++l) {  // npol[l] reads letter l at the gain and weight uses
    // N's se at the weight uses and of dK: the per-use se option (kNaN without it)
    auto nse = [&](float* arr, int64_t off) -> const float* { return l != 2 ? kZero : (se ? arr + off : kNaN); };
    row(0, l, w.e1.g_bias + l * d, dgain1, l == 2 ? w.e1.g_se + l * d : kZero, d);
    row(1, l, w.e1.w_bias + l * d3d, dWqkv, nse(w.e1.w_se, l * d3d), d3d);
    row(2, l, l == 2 ? nullptr : w.e1.x_bias + (l == 0 ? 0 : 3) * Td, w.dxn1, kZero, Td);
    row(3, l, w.q_bias + l * Td, w.dQ, l == 2 ? w.q_se + l * Td : kZero, Td);
    row(4, l, w.k_bias + l * Td, w.dK, nse(w.k_se, l * Td), Td);
    row(5, l, w.wo_bias + l * dd, dWo, nse(w.wo_se, 0), dd);
    row(6, l, w.e2.g_bias + l * d, dgain2, l == 2 ? w.e2.g_se + l * d : kZero, d);
    row(7, l, w.e2.w_bias + l * d2F, w.dWgu, nse(w.e2.w_se, l * d2F), d2F);
    row(8, l, l == 2 ? nullptr : w.e2.x_bias + (l == 0 ? 0 : 3) * Td, w.dxn2, kZero, Td);
    row(9, l, w.wd_bias + l * Fd, dWd, nse(w.wd_se, 0), Fd);
  }
  BS_TRY(launch_sumsq_batch(batch, w.part, st));

  // ---------------- every letter at every use together ----------------
  if (all) {
    AlluIO ai{};
    ai.B = B;
    ai.S = S;
    ai.d = d;
    ai.H = H;
    ai.F = F;
    ai.K = K;
    ai.eps = eps;
    ai.fmt = fmt;
    ai.seed = seed;
    ai.x = (const u16*)x;
    ai.gain1 = wt->gain1;
    ai.gain2 = wt->gain2;
    ai.Wqkv = (const u16*)wt->Wqkv;
    ai.Wo = (const u16*)wt->Wo;
    ai.Wgu = w.Wgu;
    ai.Q = (const u16*)Q;
    ai.Kk = (const u16*)Kk;
    ai.V = (const u16*)V;
    ai.O = O;
    ai.Otok = w.Otok;
    ai.h = h;
    ai.a = a;
    ai.c_u1 = c_u1;
    ai.c_O = c_O;
    ai.c_Otok = w.c_Otok;
    ai.c_u2 = c_u2;
    ai.c_a = c_a;
    ai.scales = scales;
    ai.dgh = w.dgh;
    ai.dh = w.dh;
    ai.dOh = w.dOh;
    ai.dqkv = w.dqkv;
    ai.u1 = w.n_u1;
    ai.u2 = w.n_u2;
    ai.r1 = w.n_r1;
    ai.r2 = w.n_r2;
    ai.du1 = w.n_du1;
    ai.du2 = w.n_du2;
    const float* refs[8] = {dx, dgain1, dWqkv, dWo, dgain2, w.dWgu, nullptr, dWd};
    for (int i = 0; i < 8; ++i) ai.ref[i] = refs[i];
    ai.wd_bias = w.wd_bias;
    ai.wgu_bias = w.e2.w_bias;
    ai.g2_bias = w.e2.g_bias;
    ai.g2_se = w.e2.g_se;
    for (int l = 0; l < 3; ++l) {
      const bs_layer_grads& b = all->bias[l];
      const bs_layer_grads& e = all->se[l];
      float* bp[8] = {b.dx, b.dgain1, b.dWqkv, b.dWo, b.dgain2, b.dWg, b.dWu, b.dWd};
      float* ep[8] = {e.dx, e.dgain1, e.dWqkv, e.dWo, e.dgain2, e.dWg, e.dWu, e.dWd};
      for (int i = 0; i < 8; ++i) {
        ai.bias[l][i] = bp[i];
        ai.se[l][i] = ep[i];
      }
    }
    ai.table = all->table;
    BS_TRY(allu_run(ai, w.allu, w.allu_bytes, st));
  }
  return BS_OK;
}

}  // extern "C"
