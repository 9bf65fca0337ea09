// C-ABI entry point of the Linear backward whose incoming gradient is rounded to FP8.
#include "bsp_kernels.h"
#include "k_combine.h"
#include "k_linear.h"
#include "k_norm.h"

using namespace bsp;

#define BS_TRY(x)               \
  do {                          \
    const bs_status _s = (x);   \
    if (_s != BS_OK) return _s; \
  } while (0)

namespace {
struct LinWs {
  u16 *xT, *dyT, *e1r[3], *e1c[3], *e2c[3], *wT[3], *pa[3], *pbT[3], *tc[3];
  float *tdx, *tdw, *d1x, *d1w[2];
  double *S1x, *S2x, *S1w[2], *S2w[2];
  u16 *cnt1, *cnt2;
  float *AW, *XB, *bx[2], *bw[2];
  double *part1, *part2, *fixpart, *fixed;
  float* scale_tmp;
};
LinWs carve_lin(Carver& c, int64_t M, int64_t k, int64_t n, bool any_shared, bool any_per_use, bool coupling,
                bool want_se) {
  LinWs w{};
  const int64_t Mp = round_up(M > 0 ? M : 1, 64);
  w.xT = c.take<u16>(k * Mp);
  w.dyT = c.take<u16>(n * Mp);
  for (int i = 0; i < 3; ++i) w.e1r[i] = c.take<u16>(M * n);
  if (any_shared)
    for (int i = 0; i < 3; ++i) w.e1c[i] = c.take<u16>(n * Mp);
  if (any_per_use)
    for (int i = 0; i < 3; ++i) w.e2c[i] = c.take<u16>(n * Mp);
  w.cnt1 = c.take<u16>(M * n);
  if (any_per_use) w.cnt2 = c.take<u16>(M * n);
  for (int i = 0; i < 2; ++i) {
    w.bx[i] = c.take<float>(M * k);
    w.bw[i] = c.take<float>(k * n);
  }
  if (coupling) {
    for (int i = 0; i < 3; ++i) w.wT[i] = c.take<u16>(n * k);
    for (int i = 0; i < 3; ++i) w.pa[i] = c.take<u16>(M * k);
    for (int i = 0; i < 3; ++i) w.pbT[i] = c.take<u16>(n * k);
    w.AW = c.take<float>(M * n);
    w.XB = c.take<float>(M * n);
  }
  if (want_se) {  // the per-trial path: one trial's residual planes, moves and shifted sums
    for (int i = 0; i < 3; ++i) w.tc[i] = c.take<u16>(n * Mp);
    w.tdx = c.take<float>(M * k);
    w.tdw = c.take<float>(k * n);
    w.d1x = c.take<float>(M * k);
    w.S1x = c.take<double>(M * k);
    w.S2x = c.take<double>(M * k);
    for (int i = 0; i < 2; ++i) {
      w.d1w[i] = c.take<float>(k * n);
      w.S1w[i] = c.take<double>(k * n);
      w.S2w[i] = c.take<double>(k * n);
    }
  }
  return w;
}
}  // namespace

extern "C" {

size_t bs_linear_bwd_workspace_size(int64_t M, int64_t k, int64_t n, int n_pol, int K, int want_se) {
  (void)n_pol;
  if (M < 0 || k < 0 || n < 0 || K < 1) return 0;
  Carver c;
  carve_lin(c, M, k, n, true, true, true, want_se != 0);
  const int64_t nblk = fresh_count_blocks(M, n);
  c.take<double>((int64_t)K * 2 * nblk);
  c.take<double>((int64_t)K * 2 * nblk);
  c.take<double>(2 * 1024 + 2);
  return c.used();
}

bs_status bs_linear_bwd_policy(const void* X, const void* W, const void* dY, bs_dtype dt, int64_t M, int64_t k,
                               int64_t n, bs_fp8 fmt, const int* sharing, int n_pol, int K, uint64_t seed,
                               uint32_t store_id, float* dX_ref, float* dW_ref, bs_est dX, bs_est dW,
                               const float* probeA, const float* probeB, double* coupling, float* dY_scale,
                               bs_diag* diag, void* ws, size_t ws_bytes, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  if (!W || !dW_ref || !dY_scale || !diag || !sharing) return BS_EINVAL;
  if (M < 0 || (M > 0 && (!X || !dY || !dX_ref))) return BS_EINVAL;
  if (dt != BS_BF16) return BS_EDTYPE;
  if ((fmt != BS_E4M3 && fmt != BS_E5M2) || n_pol < 1 || n_pol > 2 * 2 || K < 1 || K > 4096) return BS_EINVAL;
  if (k < 8 || (k & 7) || n < 8 || (n & 7) || M > 0x7FFFFFFF || k > 0x7FFFFFFF || n > 0x7FFFFFFF) return BS_ESHAPE;
  const bool want_se = dX.se || dW.se;
  const bool coupling_on = coupling != nullptr;
  if (coupling_on != (probeA != nullptr) || coupling_on != (probeB != nullptr)) return BS_EINVAL;
  bool any_shared = false, any_per_use = false;
  for (int i = 0; i < n_pol; ++i) {
    if (sharing[i] != 0 && sharing[i] != 1) return BS_EINVAL;
    any_shared |= sharing[i] == 0;
    any_per_use |= sharing[i] == 1;
  }
  const int64_t nblk = fresh_count_blocks(M, n);
  auto carve_all = [&](Carver& c, LinWs& w) {
    w = carve_lin(c, M, k, n, any_shared, any_per_use, coupling_on, want_se);
    if (coupling_on) {
      w.part1 = c.take<double>((int64_t)K * 2 * nblk);
      if (any_per_use) w.part2 = c.take<double>((int64_t)K * 2 * nblk);
      w.fixpart = c.take<double>(2 * 1024);
      w.fixed = c.take<double>(2);
    }
  };
  Carver probe;
  LinWs w;
  carve_all(probe, w);
  if (!ws || ((uintptr_t)ws & 255) || ws_bytes < probe.used()) return BS_EWORKSPACE;
  Carver c(ws, ws_bytes);
  carve_all(c, w);

  const int64_t Mp = round_up(M > 0 ? M : 1, 64);
  const uint32_t base = store_id * 256u;
  const F8 f = f8_format(fmt);

  // per-tensor scale of dY: s = amax(dY) / FMAX (the store's first steps; no forward codes)
  BS_TRY(launch_store(dY, BS_BF16, M * n, fmt, BS_RNE, seed, 0, base, nullptr, nullptr, dY_scale, diag, st, false));

  auto gemm = [&](int Mg, int Ng, int Kg, int64_t lda, int64_t ldb, u16* const* A, int nA, u16* const* B, int nB,
                  float* C, float alpha) -> bs_status {
    GemmArgs g{};
    g.M = Mg;
    g.N = Ng;
    g.K = Kg;
    g.lda = lda;
    g.ldb = ldb;
    g.ldc = Ng;
    g.alpha = alpha;
    g.C = C;
    if (!gemm_add_products(g, A, nA, B, nB)) return BS_EINVAL;
    return launch_gemm(g, st);
  };
  u16* dYp = (u16*)dY;
  u16* Wp = (u16*)W;
  u16* Xp = (u16*)X;
  // references with the unrounded dY: dX = dY W^T, dW = X^T dY
  BS_TRY(gemm((int)M, (int)k, (int)n, n, n, &dYp, 1, &Wp, 1, dX_ref, 1.0f));
  BS_TRY(launch_planes(X, BS_BF16, M, k, k, true, &w.xT, 1, Mp, 1.0f, st));
  BS_TRY(launch_planes(dY, BS_BF16, M, n, n, true, &w.dyT, 1, Mp, 1.0f, st));
  BS_TRY(gemm((int)k, (int)n, (int)Mp, Mp, Mp, &w.xT, 1, &w.dyT, 1, dW_ref, 1.0f));

  // coupling weights AW = A W and XB = X B
  if (coupling_on) {
    BS_TRY(launch_planes(W, BS_BF16, k, n, n, true, w.wT, 1, k, 1.0f, st));
    BS_TRY(launch_planes(probeA, BS_F32, M, k, k, false, w.pa, 3, k, 1.0f, st));
    BS_TRY(gemm((int)M, (int)n, (int)k, k, k, w.pa, 3, w.wT, 1, w.AW, 1.0f));
    BS_TRY(launch_planes(probeB, BS_F32, k, n, n, true, w.pbT, 3, k, 1.0f, st));
    BS_TRY(gemm((int)M, (int)n, (int)k, k, k, &Xp, 1, w.pbT, 3, w.XB, 1.0f));
    BS_TRY(launch_kappa_fixed((const u16*)dY, dY_scale, fmt, M, n, w.AW, w.XB, w.fixpart, w.fixed, st));
  }

  // new roundings of dY: use +1 (dX, and dW when shared), use +2 (dW per use)
  FreshArgs<u16> fa{(const u16*)dY, M, n, f, dY_scale, seed, base + 1, K, w.cnt1, nullptr, nullptr, nullptr};
  if (coupling_on) {
    fa.w1 = w.AW;
    fa.w2 = w.XB;
    fa.partial = w.part1;
    BS_TRY(launch_fresh_count_t(fa, FC_BLOCKSUM, st));
  } else {
    BS_TRY(launch_fresh_count_t(fa, FC_COUNT, st));
  }
  if (any_per_use) {
    FreshArgs<u16> fb{(const u16*)dY, M, n, f, dY_scale, seed, base + 2, K, w.cnt2, nullptr, nullptr, nullptr};
    if (coupling_on) {
      fb.w1 = w.XB;
      fb.partial = w.part2;
      BS_TRY(launch_fresh_count_t(fb, FC_BLOCKSUM, st));
    } else {
      BS_TRY(launch_fresh_count_t(fb, FC_COUNT, st));
    }
  }

  // residual planes E_u = mean of use u's roundings - dY, and the bias contractions
  ResidArgs ra{(const u16*)dY, w.cnt1, dY_scale, K, f, M, n, {w.e1r[0], w.e1r[1], w.e1r[2]},
               {any_shared ? w.e1c[0] : nullptr, w.e1c[1], w.e1c[2]}, Mp};
  BS_TRY(launch_resid_planes(ra, st));
  BS_TRY(gemm((int)M, (int)k, (int)n, n, n, w.e1r, 3, &Wp, 1, w.bx[0], 1.0f));
  if (any_shared) BS_TRY(gemm((int)k, (int)n, (int)Mp, Mp, Mp, &w.xT, 1, w.e1c, 3, w.bw[0], 1.0f));
  if (any_per_use) {
    ResidArgs rb{(const u16*)dY, w.cnt2, dY_scale, K, f, M, n, {nullptr, nullptr, nullptr},
                 {w.e2c[0], w.e2c[1], w.e2c[2]}, Mp};
    BS_TRY(launch_resid_planes(rb, st));
    BS_TRY(gemm((int)k, (int)n, (int)Mp, Mp, Mp, &w.xT, 1, w.e2c, 3, w.bw[1], 1.0f));
  }

  // per-policy estimates and coupling
  const int64_t mk = M * k, kn = k * n;
  {
    CombineMulti cx{}, cw{};
    cx.ref = dX_ref;
    cw.ref = dW_ref;
    cx.n_pol = cw.n_pol = n_pol;
    cx.mean = dX.mean;
    cx.bias_out = dX.bias;
    cw.mean = dW.mean;
    cw.bias_out = dW.bias;
    for (int i = 0; i < n_pol; ++i) {
      cx.bias[i] = w.bx[0];
      cw.bias[i] = w.bw[sharing[i]];
    }
    BS_TRY(launch_combine_multi(cx, mk, st));
    BS_TRY(launch_combine_multi(cw, kn, st));
  }
  // se over trials (App. C.4), the per-trial path: trial k's residual fresh_k - dY moves dX and dW
  // by contractions of its planes; shifted fp64 sums over trials. dX reads use +1 under both
  // sharings, dW use +1 (shared) or +2 (per use).
  if (want_se && M > 0) {
    for (int kk = 1; kk <= K; ++kk) {
      for (int u = 0; u < 2; ++u) {
        if (u == 1 && !any_per_use) continue;
        FreshArgs<u16> ft{(const u16*)dY, M, n, f, dY_scale, seed, base + 1 + u, 1, u == 0 ? w.cnt1 : w.cnt2,
                          nullptr, nullptr, nullptr};
        ft.trial0 = kk;
        BS_TRY(launch_fresh_count_t(ft, FC_COUNT, st));
        const bool need_w = u == 1 || any_shared;
        ResidArgs rt{(const u16*)dY, u == 0 ? w.cnt1 : w.cnt2, dY_scale, 1, f, M, n,
                     {u == 0 ? w.e1r[0] : nullptr, w.e1r[1], w.e1r[2]},
                     {need_w ? w.tc[0] : nullptr, w.tc[1], w.tc[2]}, Mp};
        BS_TRY(launch_resid_planes(rt, st));
        if (u == 0 && dX.se) {
          BS_TRY(gemm((int)M, (int)k, (int)n, n, n, w.e1r, 3, &Wp, 1, w.tdx, 1.0f));
          BS_TRY(launch_trial_accum(w.tdx, 1, kk, mk, w.d1x, w.S1x, w.S2x, st));
        }
        if (need_w && dW.se) {
          BS_TRY(gemm((int)k, (int)n, (int)Mp, Mp, Mp, &w.xT, 1, w.tc, 3, w.tdw, 1.0f));
          BS_TRY(launch_trial_accum(w.tdw, 1, kk, kn, w.d1w[u], w.S1w[u], w.S2w[u], st));
        }
      }
    }
    for (int i = 0; i < n_pol; ++i) {
      if (dX.se) BS_TRY(launch_trial_se(w.S1x, w.S2x, K, mk, dX.se + i * mk, st));
      if (dW.se) BS_TRY(launch_trial_se(w.S1w[sharing[i]], w.S2w[sharing[i]], K, kn, dW.se + i * kn, st));
    }
  } else if (want_se) {
    for (int i = 0; i < n_pol; ++i)
      if (dW.se) BS_TRY(launch_fill2d(dW.se + i * kn, 1, kn, kn, 0.0f, st));
  }

  for (int i = 0; i < n_pol; ++i) {
    const int sh = sharing[i];
    if (coupling_on) {
      if (sh == 0)
        BS_TRY(launch_kappa_final(w.fixed, w.part1, 0, w.part1, 1, nblk, K, dY_scale, coupling + i, st));
      else
        BS_TRY(launch_kappa_final(w.fixed, w.part1, 0, w.part2, 0, nblk, K, dY_scale, coupling + i, st));
    }
  }
  return BS_OK;
}

}  // extern "C"
