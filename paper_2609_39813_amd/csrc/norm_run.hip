// The normalization-store runner: RMSNorm -> FP8 store -> Linear and the per-use estimates
// of the store's gain, weight and normalization-input uses.
#include <algorithm>

#include "bsp_kernels.h"
#include "k_norm.h"
#include "norm_run.h"

#define BS_TRY(x)               \
  do {                          \
    const bs_status _s = (x);   \
    if (_s != BS_OK) return _s; \
  } while (0)

namespace bsp {
namespace {

// trials per per-trial contraction (stacked along the output rows)
inline int trial_batch(int K) { return K < 8 ? K : 8; }

struct NormPlan {
  bool gain_n = false, gain_r = false, weight_u = false, want_dxr = false;
  bool weight_n[2] = {false, false};  // use +1 (shared), use +2 (per use)
  bool weight_se[2] = {false, false}; // se of the weight use under N: per-trial contractions
  bool gain_se = false;
};

struct NormWs {
  float *u, *rstd, *du, *bias_rg, *bias_ng, *se_g, *bias_u, *bias_n[2], *dx_r;
  u16 *dyT[3], *uvalT, *resU[3], *resN[2], *uval_rows, *wT[3], *dy_rows[3], *w_rows[3];
  u16 *counts_g, *counts_w;
  float* partial;
  double *gain_part, *trial_sums;
  float* gpart;  // split-K partials of the contractions
  int64_t gpart_cap;
  u16* tplanes;   // per-trial residual planes [BT][d][Tp]
  float *tdelta, *td1, *se_w[2];
  double *tS1, *tS2;
  // fp16 operands (an fp32 incoming gradient, bf16 W, K <= 256): W as scaled fp16, the maxima of
  // dY and W (slot arrays) and the multipliers 2^-e of dY, W and the U residual
  u16* W16;
  uint32_t* am[2];
  float* inv;
};

// the weight and normalization-input contractions take scaled two-term fp16 splits of an fp32
// incoming gradient against exact fp16 operands (FP8 values, residuals, the scaled weights)
inline bool use_f16(bs_dtype wt, bs_dtype gt, int K) { return gt == BS_F32 && wt == BS_BF16 && K <= 256; }

NormWs carve_norm(Carver& c, int64_t T, int64_t d, int64_t n, int K, bs_dtype wt, bs_dtype gt, const NormPlan& p,
                  bool want_y) {
  NormWs w{};
  const int64_t Tp = round_up(T > 0 ? T : 1, 64);
  const int nt = gt == BS_F32 ? 3 : 1, ntw = wt == BS_F32 ? 3 : 1;
  w.u = c.take<float>(T * d);
  w.rstd = c.take<float>(T > 0 ? T : 1);
  w.du = c.take<float>(T * d);
  for (int i = 0; i < nt; ++i) w.dyT[i] = c.take<u16>(n * Tp);
  w.uvalT = c.take<u16>(d * Tp);
  if (gt == BS_F32)
    for (int i = 0; i < 3; ++i) w.dy_rows[i] = c.take<u16>(T * n);
  if (wt == BS_F32)
    for (int i = 0; i < 3; ++i) w.w_rows[i] = c.take<u16>(d * n);
  if (want_y) {
    w.uval_rows = c.take<u16>(T * d);
    for (int i = 0; i < ntw; ++i) w.wT[i] = c.take<u16>(n * d);
  }
  w.bias_rg = c.take<float>(d);
  w.bias_ng = c.take<float>(d);
  w.se_g = c.take<float>(d);
  w.gain_part = c.take<double>(3 * ((T + GAIN_RT - 1) / GAIN_RT) * d + 1);
  if (p.weight_u) {
    for (int i = 0; i < 3; ++i) w.resU[i] = c.take<u16>(d * Tp);
    w.bias_u = c.take<float>(d * n);
  }
  if (p.weight_n[0] || p.weight_n[1]) {
    const int ntN = K > 256 ? 2 : 1;
    for (int i = 0; i < ntN; ++i) w.resN[i] = c.take<u16>(d * Tp);
    for (int i = 0; i < 2; ++i)
      if (p.weight_n[i]) w.bias_n[i] = c.take<float>(d * n);
  }
  if (p.gain_n || p.weight_n[0]) w.counts_g = c.take<u16>(T * d);
  if (p.weight_n[1]) w.counts_w = c.take<u16>(T * d);
  if (p.gain_se) {
    w.partial = c.take<float>((int64_t)K * ((T + 31) / 32) * d + 1);
    w.trial_sums = c.take<double>((int64_t)K * d);
  }
  if (p.want_dxr) w.dx_r = c.take<float>(T * d);
  if (p.weight_se[0] || p.weight_se[1]) {
    const int bt = trial_batch(K);
    w.tplanes = c.take<u16>((int64_t)bt * d * Tp);
    w.tdelta = c.take<float>((int64_t)bt * d * n);
    w.td1 = c.take<float>(d * n);
    w.tS1 = c.take<double>(d * n);
    w.tS2 = c.take<double>(d * n);
    for (int i = 0; i < 2; ++i)
      if (p.weight_se[i]) w.se_w[i] = c.take<float>(d * n);
  }
  if (use_f16(wt, gt, K)) {
    w.W16 = c.take<u16>(d * n);
    uint32_t* a = c.take<uint32_t>(2 * AMAX_SLOTS * AMAX_STRIDE);
    for (int i = 0; i < 2; ++i) w.am[i] = a ? a + i * AMAX_SLOTS * AMAX_STRIDE : nullptr;
    w.inv = c.take<float>(3);
  }
  // split-K partials for the contractions with few output tiles (du: T x d; weight use: d x n)
  w.gpart_cap = 4 * d * std::max<int64_t>(std::max<int64_t>(T, n), 64);
  w.gpart = c.take<float>(w.gpart_cap);
  return w;
}

NormPlan plan_norm(const bs_norm_policy* pol, int n_pol, bool want_gain_se, bool want_weight_se) {
  NormPlan p;
  for (int i = 0; i < n_pol; ++i) {
    if (pol[i].gain_use == BS_READ_N) p.gain_n = true;
    if (pol[i].gain_use == BS_READ_R) p.gain_r = true;
    if (pol[i].weight_use == BS_READ_U) p.weight_u = true;
    if (pol[i].weight_use == BS_READ_N) p.weight_n[pol[i].fresh_shared ? 0 : 1] = true;
    if (pol[i].norm_input_use == BS_READ_R) p.want_dxr = true;
    if (pol[i].weight_use == BS_READ_N && want_weight_se) p.weight_se[pol[i].fresh_shared ? 0 : 1] = true;
  }
  p.gain_se = want_gain_se && p.gain_n;
  return p;
}

}  // namespace


size_t norm_ws_size(int64_t T, int64_t d, int64_t n, int K) {
  // sized for the most demanding policy set, over the operand types (fp32 everywhere, or the
  // fp16 path's bf16 W with an fp32 incoming gradient)
  NormPlan p;
  p.gain_n = p.gain_r = p.weight_u = p.want_dxr = p.gain_se = true;
  p.weight_n[0] = p.weight_n[1] = true;
  p.weight_se[0] = p.weight_se[1] = true;
  Carver c, c16;
  carve_norm(c, T, d, n, K, BS_F32, BS_F32, p, true);
  carve_norm(c16, T, d, n, K, BS_BF16, BS_F32, p, true);
  return std::max(c.used(), c16.used());
}

bs_status norm_run(const NormIO& io, void* ws, size_t ws_bytes, hipStream_t st) {
  const void *X = io.X, *W = io.W, *dY = io.dY;
  const float* gain = io.gain;
  const bs_dtype xt = io.xt, wt = io.wt, gt = io.gt;
  const int64_t T = io.T, d = io.d, n = io.n;
  const float eps = io.eps;
  const int fmt = io.fmt, fwd_mode = io.fwd_mode, n_pol = io.n_pol, K = io.K;
  const bs_norm_policy* pol = io.pol;
  const uint64_t seed = io.seed;
  const uint32_t store_id = io.store_id;
  float *Y = io.Y, *u_scale = io.u_scale, *dgain_ref = io.dgain_ref, *dW_ref = io.dW_ref, *dX_ref = io.dX_ref;
  uint8_t* u_codes = io.u_codes;
  const bs_est dgain = io.dgain, dW = io.dW, dX = io.dX;
  bs_diag* diag = io.diag;
  const bool fwd_only = dY == nullptr;
  if (!gain || !W || !u_scale || !diag || (!fwd_only && (!dgain_ref || !dW_ref || !pol))) return BS_EINVAL;
  if (T < 0 || (T > 0 && (!X || !u_codes || (!fwd_only && !dX_ref)))) return BS_EINVAL;
  for (bs_dtype t : {xt, wt, gt})
    if (t != BS_F32 && t != BS_BF16) return BS_EDTYPE;
  if ((fmt != BS_E4M3 && fmt != BS_E5M2) || (fwd_mode != BS_RNE && fwd_mode != BS_SR)) return BS_EINVAL;
  if ((!fwd_only && (n_pol < 1 || n_pol > 16)) || K < 1 || K > 4096 || !(eps >= 0.0f)) return BS_EINVAL;
  if (d < 8 || d > 8192 || (d & 7) || n < 8 || (n & 7) || T > 0x7FFFFFFF || n > 0x7FFFFFFF) return BS_ESHAPE;
  for (int i = 0; i < (fwd_only ? 0 : n_pol); ++i) {
    if (pol[i].gain_use < BS_READ_U || pol[i].gain_use > BS_READ_N || pol[i].weight_use < BS_READ_U ||
        pol[i].weight_use > BS_READ_N)
      return BS_EINVAL;
    if (pol[i].norm_input_use != BS_READ_U && pol[i].norm_input_use != BS_READ_R) return BS_EINVAL;
  }
  const NormPlan p = fwd_only ? NormPlan{} : plan_norm(pol, n_pol, dgain.se != nullptr, dW.se != nullptr);
  Carver probe;
  carve_norm(probe, T, d, n, K, wt, gt, p, Y != nullptr);
  if (!ws || ((uintptr_t)ws & 255) || ws_bytes < probe.used()) return BS_EWORKSPACE;
  Carver c(ws, ws_bytes);
  NormWs w = carve_norm(c, T, d, n, K, wt, gt, p, Y != nullptr);
  if (io.rstd_out) w.rstd = io.rstd_out;
  if (io.du_out) w.du = io.du_out;

  const int64_t Tp = round_up(T > 0 ? T : 1, 64);
  const int nt = gt == BS_F32 ? 3 : 1, ntw = wt == BS_F32 ? 3 : 1;
  const F8 f = f8_format(fmt);
  const uint32_t base = store_id * 256u;
  const uint32_t use_g = base + 1, use_w[2] = {base + 1, base + 2};

  // forward: fixed-order RMSNorm with fused amax, then the store
  BS_TRY(launch_init_diag(diag, st));
  BS_TRY(launch_rmsnorm_fwd(X, xt, gain, T, d, eps, io.u_out ? io.u_out : w.u, w.rstd, diag, st));
  if (io.u_out) w.u = io.u_out;
  BS_TRY(launch_store(w.u, BS_F32, T * d, fmt, fwd_mode, seed, 0, base, nullptr, u_codes, u_scale, diag, st, true));

  // Linear forward Y = s val(C_u) W  (A = val rows [T, d], B = W^T [n, d])
  if (Y) {
    BS_TRY(launch_val_rows(u_codes, T * d, fmt, w.uval_rows, st));
    BS_TRY(launch_planes(W, wt, d, n, n, true, w.wT, ntw, d, 1.0f, st));
    GemmArgs g{};
    g.M = (int)T;
    g.N = (int)n;
    g.K = (int)d;
    g.lda = d;
    g.ldb = d;
    g.ldc = n;
    g.alpha = 1.0f;
    g.alpha_dev = u_scale;
    g.C = Y;
    gemm_add_products(g, &w.uval_rows, 1, w.wT, ntw);
    BS_TRY(launch_gemm(g, st));
  }
  if (fwd_only) return BS_OK;

  const bool h16 = use_f16(wt, gt, K);
  const bool du16 = h16 && n % 64 == 0;  // du's fp16 contraction runs on the pipelined kernel (K % 64)
  const int ntd = h16 ? 2 : nt;  // terms of the incoming gradient's planes
  if (h16) {
    // dY's scaled two-term fp16 split in both layouts from one read, W as scaled fp16
    BS_TRY(launch_fill2d((float*)w.am[0], 2 * AMAX_SLOTS, 1, AMAX_STRIDE, 0.0f, st));
    BS_TRY(launch_amax_f32((const float*)dY, T * n, w.am[0], st));
    BS_TRY(launch_amax_bf16((const u16*)W, d * n, w.am[1], st));
    BS_TRY(launch_scale_f16((const u16*)W, d * n, w.am[1], w.W16, w.inv + 1, st));
    MoveSrc ms{};
    ms.rows = (const float*)dY;
    ms.ldi = n;
    BS_TRY(launch_split_move(ms, nullptr, 0, T, n, F16Scale{w.am[0], nullptr, w.inv + 0}, w.dyT, nullptr, Tp,
                             du16 ? w.dy_rows : nullptr, n, st));
  }
  // du = dY W^T  (A = dY [T, n], B = W [d, n], both n-contiguous)
  if (du16) {
    GemmArgs g{};
    g.M = (int)T;
    g.N = (int)d;
    g.K = (int)n;
    g.lda = n;
    g.ldb = n;
    g.ldc = d;
    g.alpha = 1.0f;
    g.alpha_dev = w.inv + 1;
    g.alpha_dev2 = w.inv + 0;
    g.f16 = 1;
    g.C = w.du;
    g.part = w.gpart;
    g.part_cap = w.gpart_cap;
    const u16* B0 = w.W16;
    gemm_add_products(g, w.dy_rows, 2, &B0, 1);
    BS_TRY(launch_gemm(g, st));
  } else {
    GemmArgs g{};
    g.M = (int)T;
    g.N = (int)d;
    g.K = (int)n;
    g.lda = n;
    g.ldb = n;
    g.ldc = d;
    g.alpha = 1.0f;
    g.C = w.du;
    g.part = w.gpart;
    g.part_cap = w.gpart_cap;
    u16* A0 = (u16*)dY;
    u16* B0 = (u16*)W;
    u16* const* Aops = &A0;
    u16* const* Bops = &B0;
    if (gt == BS_F32) {
      BS_TRY(launch_planes(dY, gt, T, n, n, false, w.dy_rows, 3, n, 1.0f, st));
      Aops = w.dy_rows;
    }
    if (wt == BS_F32) {
      BS_TRY(launch_planes(W, wt, d, n, n, false, w.w_rows, 3, n, 1.0f, st));
      Bops = w.w_rows;
    }
    gemm_add_products(g, Aops, gt == BS_F32 ? 3 : 1, Bops, wt == BS_F32 ? 3 : 1);
    BS_TRY(launch_gemm(g, st));
  }

  // weight-use operands in the contraction layout [*, Tp]
  if (!h16) BS_TRY(launch_planes(dY, gt, T, n, n, true, w.dyT, nt, Tp, 1.0f, st));
  NormPlaneArgs pa{};
  pa.u = w.u;
  pa.codes = u_codes;
  pa.scale = u_scale;
  pa.K = K;
  pa.f = f;
  pa.T = T;
  pa.d = d;
  pa.ldo = Tp;
  pa.out[0] = w.uvalT;
  pa.nterms = 1;
  pa.f16 = h16;
  pa.amax_u = &diag->amax;
  pa.inv_out = h16 ? w.inv + 2 : nullptr;
  // the N residual is an up-count difference (|.| <= K <= 256) times a step: exact in fp16 for
  // E4M3 (steps 2^-9 .. 2^5); E5M2's steps 2^-16 .. 2^13 take the scale 2^-8 (2^-24 .. 2^13)
  pa.resn_scale = fmt == BS_E5M2 ? 0x1p-8f : 1.0f;
  BS_TRY(launch_norm_planes(NP_VAL, pa, st));

  auto weight_gemm = [&](u16* const* A, int nA, float* C, float alpha, const float* alpha_dev) -> bs_status {
    GemmArgs g{};
    g.M = (int)d;
    g.N = (int)n;
    g.K = (int)Tp;
    g.lda = Tp;
    g.ldb = Tp;
    g.ldc = n;
    g.alpha = alpha;
    g.alpha_dev = alpha_dev;
    g.C = C;
    g.part = w.gpart;
    g.part_cap = w.gpart_cap;
    if (h16) {
      g.f16 = 1;
      g.alpha_dev2 = w.inv + 0;
    }
    if (!gemm_add_products(g, A, nA, w.dyT, ntd, h16 && nA == 2 ? 1 : 2)) return BS_EINVAL;
    return launch_gemm(g, st);
  };
  // reference: dW = s val(C_u)^T dY
  BS_TRY(weight_gemm(&w.uvalT, 1, dW_ref, 1.0f, u_scale));

  // new roundings: up counts over K trials (gain use: use +1; weight use: +1 shared / +2)
  if (p.gain_n || p.weight_n[0])
    BS_TRY(launch_fresh_count(w.u, T, d, fmt, u_scale, seed, use_g, K, w.counts_g, w.du,
                              p.gain_se ? w.partial : nullptr, st));
  if (p.weight_n[1]) BS_TRY(launch_fresh_count(w.u, T, d, fmt, u_scale, seed, use_w[1], K, w.counts_w, nullptr,
                                               nullptr, st));

  // gain use: reference and the R / N biases (fp64 column sums)
  if (xt == BS_F32) {
    GainArgs<float> ga{(const float*)X, w.rstd, gain, w.u, w.du, u_codes, p.gain_n ? w.counts_g : nullptr, u_scale, K,
                       p.gain_r ? 1 : 0, f, T, d, w.gain_part};
    BS_TRY(launch_gain_t(ga, dgain_ref, w.bias_rg, w.bias_ng, st));
  } else {
    GainArgs<u16> ga{(const u16*)X, w.rstd, gain, w.u, w.du, u_codes, p.gain_n ? w.counts_g : nullptr, u_scale, K,
                     p.gain_r ? 1 : 0, f, T, d, w.gain_part};
    BS_TRY(launch_gain_t(ga, dgain_ref, w.bias_rg, w.bias_ng, st));
  }
  if (p.gain_se) BS_TRY(launch_gain_se(w.partial, K, T, d, u_scale, gain, w.trial_sums, w.se_g, st));

  // weight use: U bias = (u - s val)^T dY; N bias = (s / K) (sum of up counts residual)^T dY
  if (p.weight_u) {
    pa.out[0] = w.resU[0];
    pa.out[1] = w.resU[1];
    pa.out[2] = h16 ? nullptr : w.resU[2];
    pa.nterms = h16 ? 2 : 3;
    BS_TRY(launch_norm_planes(NP_RESU, pa, st));
    BS_TRY(weight_gemm(w.resU, pa.nterms, w.bias_u, 1.0f, h16 ? w.inv + 2 : nullptr));
  }
  for (int i = 0; i < 2; ++i) {
    if (!p.weight_n[i]) continue;
    pa.counts = i == 0 ? w.counts_g : w.counts_w;
    pa.out[0] = w.resN[0];
    pa.out[1] = w.resN[1];
    pa.out[2] = nullptr;
    pa.nterms = K > 256 ? 2 : 1;
    BS_TRY(launch_norm_planes(NP_RESN, pa, st));
    BS_TRY(weight_gemm(w.resN, pa.nterms, w.bias_n[i], 1.0f / (float)K / (h16 ? pa.resn_scale : 1.0f), u_scale));
  }

  // se of the weight use under N: per-trial contractions (trials stacked along the rows of
  // the output), shifted fp64 sums over trials, sample SD / sqrt(K)
  for (int i = 0; i < 2; ++i) {
    if (!p.weight_se[i]) continue;
    const int bt = trial_batch(K);
    for (int k0 = 1; k0 <= K; k0 += bt) {
      const int nb = K - k0 + 1 < bt ? K - k0 + 1 : bt;
      TrialPlaneArgs ta{w.u, u_codes, u_scale, f, T, d, Tp, seed, use_w[i], k0, nb, w.tplanes};
      ta.f16 = h16;
      BS_TRY(launch_trial_planes(ta, st));
      GemmArgs g{};
      g.M = (int)(nb * d);
      g.N = (int)n;
      g.K = (int)Tp;
      g.lda = Tp;
      g.ldb = Tp;
      g.ldc = n;
      g.alpha = 1.0f;
      g.alpha_dev = u_scale;
      g.C = w.tdelta;
      if (h16) {
        g.f16 = 1;
        g.alpha_dev2 = w.inv + 0;
      }
      const u16* A0 = w.tplanes;
      if (!gemm_add_products(g, &A0, 1, w.dyT, ntd)) return BS_EINVAL;
      BS_TRY(launch_gemm(g, st));
      BS_TRY(launch_trial_accum(w.tdelta, nb, k0, d * n, w.td1, w.tS1, w.tS2, st));
    }
    BS_TRY(launch_trial_se(w.tS1, w.tS2, K, d * n, w.se_w[i], st));
  }

  // norm-input use
  if (xt == BS_F32) {
    DxArgs<float> da{(const float*)X, w.rstd, gain, w.du, u_codes, u_scale, f, T, d, dX_ref, w.dx_r};
    BS_TRY(launch_dx_t(da, st));
  } else {
    DxArgs<u16> da{(const u16*)X, w.rstd, gain, w.du, u_codes, u_scale, f, T, d, dX_ref, w.dx_r};
    BS_TRY(launch_dx_t(da, st));
  }

  // per-policy estimates: one pass per gradient over its reference
  if (!fwd_only) {
    CombineMulti cg{}, cw{}, cx{};
    cg.ref = dgain_ref;
    cw.ref = dW_ref;
    cx.ref = dX_ref;
    for (CombineMulti* c : {&cg, &cw, &cx}) c->n_pol = n_pol;
    cg.mean = dgain.mean;
    cg.bias_out = dgain.bias;
    cg.se_out = dgain.se;
    cw.mean = dW.mean;
    cw.bias_out = dW.bias;
    cw.se_out = dW.se;
    cx.mean = dX.mean;
    cx.bias_out = dX.bias;
    cx.se_out = dX.se;
    for (int i = 0; i < n_pol; ++i) {
      const bs_norm_policy& q = pol[i];
      const int fs = q.fresh_shared ? 0 : 1;
      cg.bias[i] = q.gain_use == BS_READ_R ? w.bias_rg : (q.gain_use == BS_READ_N ? w.bias_ng : nullptr);
      cg.se[i] = (q.gain_use == BS_READ_N && p.gain_se) ? w.se_g : nullptr;
      cw.bias[i] = q.weight_use == BS_READ_U ? w.bias_u : (q.weight_use == BS_READ_N ? w.bias_n[fs] : nullptr);
      cw.se[i] = (q.weight_use == BS_READ_N && p.weight_se[fs]) ? w.se_w[fs] : nullptr;
      cx.alt[i] = q.norm_input_use == BS_READ_R ? w.dx_r : nullptr;
    }
    BS_TRY(launch_combine_multi(cg, d, st));
    BS_TRY(launch_combine_multi(cw, d * n, st));
    BS_TRY(launch_combine_multi(cx, T * d, st));
  }
  return BS_OK;
}


}  // namespace bsp
