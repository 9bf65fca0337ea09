// The attention runner: forward (row max / row sum, and O when not handed in), the FP8 store of
// O, the D variants of every policy, and the two-pass multi-D backward.
#include "attn_run.h"
#include "k_attn.h"
#include "k_norm.h"

#define BS_TRY(x)               \
  do {                          \
    const bs_status _s = (x);   \
    if (_s != BS_OK) return _s; \
  } while (0)

namespace bsp {

namespace {
struct AttnWs {
  float *m, *l, *O, *D_ref, *dD_R, *dD_N, *sd_N;
  u16 *Vt, *Qt, *Kt, *dOp[3], *dOt[3];
  float *dO_mean, *stat;   // level 2: mean incoming gradient; split of R and N [2][4][rows]
  uint8_t* codes;          // level 2: the trial-0 store when the caller takes none
  float *dD_tr, *tdk, *d1, *sek, *dK_s, *dV_s;  // dK's se: per-trial dD, one trial's dK move, shift, scratch
  double *S1, *S2;
};
AttnWs carve_attn(Carver& c, int64_t rows, int64_t numel, bool need_o, bool need_dref, int64_t bh = 0, int64_t Sp = 0,
                  int ndo = 0, bool level2 = false, int K = 0) {
  AttnWs w{};
  if (K > 0) {
    w.dD_tr = c.take<float>((int64_t)K * rows);
    for (float** p : {&w.tdk, &w.d1, &w.sek, &w.dK_s, &w.dV_s}) *p = c.take<float>(numel);
    w.S1 = c.take<double>(numel);
    w.S2 = c.take<double>(numel);
  }
  if (level2) {
    w.dO_mean = c.take<float>(numel);
    w.stat = c.take<float>(8 * rows);
    w.codes = c.take<uint8_t>(numel);
  }
  w.Vt = c.take<u16>(bh * 64 * Sp);
  if (ndo > 0) {  // operand copies for the backward
    w.Qt = c.take<u16>(bh * 64 * Sp);
    w.Kt = c.take<u16>(bh * 64 * Sp);
    for (int i = 0; i < ndo; ++i) w.dOt[i] = c.take<u16>(bh * 64 * Sp);
    if (ndo == 3)
      for (int i = 0; i < 3; ++i) w.dOp[i] = c.take<u16>(numel);
  }
  w.m = c.take<float>(rows);
  w.l = c.take<float>(rows);
  if (need_o) w.O = c.take<float>(numel);
  if (need_dref) w.D_ref = c.take<float>(rows);
  w.dD_R = c.take<float>(rows);
  w.dD_N = c.take<float>(rows);
  w.sd_N = c.take<float>(rows);
  return w;
}
}  // namespace

size_t attn_ws_size(int B, int H, int S, int dh, int K, bool dk_se) {
  if (B < 0 || H < 0 || S < 0 || dh < 0 || K < 1) return 0;
  Carver c;
  const int64_t rows = (int64_t)B * H * S;
  carve_attn(c, rows, rows * dh, true, true, (int64_t)B * H, (S + 63) / 64 * 64, 3, true, dk_se ? K : 0);
  return c.used();
}

bs_status attn_run(const AttnIO& io, void* ws, size_t ws_bytes, hipStream_t st) {
  const bool fwd_only = !io.dO && !io.dO32;
  const bool l2 = io.level2 != 0;
  if (l2 && (!io.dO || io.dO32 || !(io.beta == io.beta))) return BS_EINVAL;
  if (!io.Q || !io.Kt || !io.V || (!io.O_codes && !l2) || !io.O_scale || !io.diag) return BS_EINVAL;
  if (!fwd_only && (!io.dQ_ref || !io.dK_ref || !io.dV || !io.pol)) return BS_EINVAL;
  if (io.B < 1 || io.H < 1 || io.S < 1 || io.K < 1 || io.K > 4096) return BS_EINVAL;
  if (!fwd_only && (io.n_pol < 1 || io.n_pol > ATTN_MAX_POL)) return BS_EINVAL;
  if (!(io.scale > 0.0f) || (io.fmt != BS_E4M3 && io.fmt != BS_E5M2) ||
      (io.fwd_mode != BS_RNE && io.fwd_mode != BS_SR))
    return BS_EINVAL;
  if (io.dh != 64) return BS_ESHAPE;
  for (const void* p : {io.Q, io.Kt, io.V, io.dO, (const void*)io.dO32, (const void*)io.O})
    if ((uintptr_t)p & 15) return BS_EINVAL;  // 16-byte vector loads
  if ((int64_t)io.B * io.H > 65535 || (io.S + 63) / 64 > 65535) return BS_ESHAPE;
  if (l2 && (io.dK.se || io.dQ.se)) return BS_EUNSUPPORTED;
  bool want_r = false, want_n = false;
  for (int i = 0; i < (fwd_only ? 0 : io.n_pol); ++i) {
    if (io.pol[i] < BS_READ_U || io.pol[i] > BS_READ_N) return BS_EINVAL;
    want_r |= io.pol[i] == BS_READ_R;
    want_n |= io.pol[i] == BS_READ_N;
  }
  const int64_t rows = (int64_t)io.B * io.H * io.S, numel = rows * io.dh;
  const bool need_o = !io.O && !io.O_out;
  const int64_t bh = (int64_t)io.B * io.H, Sp = (io.S + 63) / 64 * 64;
  const int ndo = fwd_only ? 0 : ((io.dO32 || l2) ? 3 : 1);
  const int dk_trials = (!fwd_only && io.dK.se && want_n) ? io.K : 0;
  Carver probe;
  carve_attn(probe, rows, numel, need_o, !io.D_ref, bh, Sp, ndo, l2, dk_trials);
  if (!ws || ((uintptr_t)ws & 255) || ws_bytes < probe.used()) return BS_EWORKSPACE;
  Carver c(ws, ws_bytes);
  AttnWs w = carve_attn(c, rows, numel, need_o, !io.D_ref, bh, Sp, ndo, l2, dk_trials);
  float* dref = io.D_ref ? io.D_ref : w.D_ref;
  uint8_t* O_codes = io.O_codes ? io.O_codes : w.codes;
  // level 2: the mean incoming gradient replaces dO in the backward (fp32, three bf16 planes)
  const float* dO32 = l2 ? (io.dO_mean ? io.dO_mean : w.dO_mean) : io.dO32;

  // forward: m, l (and O when the caller does not hand it in)
  {  // transposed operand copies: V^T for the forward; Q^T, K^T (and dO^T) for the backward
    const u16* src[4] = {(const u16*)io.V, (const u16*)io.Q, (const u16*)io.Kt, (const u16*)io.dO};
    u16* dst[4] = {w.Vt, w.Qt, w.Kt, w.dOt[0]};
    const int n = fwd_only ? 1 : (dO32 ? 3 : 4);
    BS_TRY(launch_attn_transpose(src, dst, n, (int)bh, io.S, (int)Sp, st));
  }
  AttnArgs fa{(const u16*)io.Q, (const u16*)io.Kt, (const u16*)io.V, io.S, io.causal, io.scale, w.m, w.l, nullptr,
              w.Vt, (int)Sp};
  const float* Oorig = io.O;
  if (!io.O) {
    fa.O_out = io.O_out ? io.O_out : w.O;
    Oorig = fa.O_out;
  }
  BS_TRY(launch_attn_fwd(fa, io.B, io.H, st));
  if (io.O && io.O_out) {
    if (hipMemcpyAsync(io.O_out, io.O, sizeof(float) * numel, hipMemcpyDeviceToDevice, st) != hipSuccess)
      return BS_EHIP;
  }

  // the store of O (trial 0, use store_id*256)
  const uint32_t base = io.store_id * 256u;
  BS_TRY(launch_store(Oorig, BS_F32, numel, io.fmt, io.fwd_mode, io.seed, 0, base, nullptr, O_codes, io.O_scale,
                      io.diag, st, false));
  if (fwd_only) return BS_OK;

  // D variants
  if (l2) {
    AttnL2Args la{Oorig, (const u16*)io.dO, io.O_scale, rows, f8_format(io.fmt), io.fwd_mode, io.seed, base,
                  base + 1, io.K, io.beta, (float*)dO32, dref, w.dD_R, w.dD_N, w.stat, w.stat + 4 * rows,
                  io.T};
    BS_TRY(launch_attn_l2(la, st));
    for (int i = 0; i < (io.d_use ? io.n_pol : 0); ++i) {
      float* dst = io.d_use + (int64_t)i * 4 * rows;
      if (io.pol[i] == BS_READ_U)  // U reads the original: its error is zero in every trial
        BS_TRY(launch_combine(w.stat, nullptr, nullptr, 4 * rows, nullptr, dst, nullptr, st));
      else
        BS_TRY(launch_combine(w.stat + (io.pol[i] == BS_READ_R ? 0 : 4 * rows), nullptr, nullptr, 4 * rows, dst,
                              nullptr, nullptr, st));
    }
  } else {
    AttnDArgs da{Oorig, (const u16*)io.dO, io.dO32, O_codes, io.O_scale, rows, f8_format(io.fmt), io.seed, base + 1,
                 io.K, want_n ? 1 : 0, dref, w.dD_R, w.dD_N, w.sd_N};
    da.dD_trials = dk_trials ? w.dD_tr : nullptr;
    BS_TRY(launch_attn_d(da, st));
  }

  if (dO32) BS_TRY(launch_attn_split(dO32, (int)bh, io.S, (int)Sp, w.dOp, w.dOt, st));
  AttnBwdArgs ba{};
  ba.Qt = w.Qt;
  ba.Kt = w.Kt;
  for (int i = 0; i < 3; ++i) {
    ba.dOp[i] = w.dOp[i];
    ba.dOt[i] = w.dOt[i];
  }
  ba.Sp = (int)Sp;
  ba.Q = (const u16*)io.Q;
  ba.K = (const u16*)io.Kt;
  ba.V = (const u16*)io.V;
  ba.dO = (const u16*)io.dO;
  ba.dO32 = dO32;
  ba.m = w.m;
  ba.l = w.l;
  ba.D_ref = dref;
  ba.dD_R = want_r ? w.dD_R : nullptr;
  ba.dD_N = want_n ? w.dD_N : nullptr;
  ba.sd_N = (want_n && !l2) ? w.sd_N : nullptr;
  ba.S = io.S;
  ba.causal = io.causal;
  ba.ntrial = io.K;
  ba.scale = io.scale;
  ba.dQ_ref = io.dQ_ref;
  ba.dK_ref = io.dK_ref;
  ba.dV = io.dV;
  ba.n_pol = io.n_pol;
  for (int i = 0; i < io.n_pol; ++i) {
    ba.pol[i] = io.pol[i];
    ba.mean[i] = io.dQ.mean ? io.dQ.mean + i * numel : nullptr;
    ba.bias[i] = io.dQ.bias ? io.dQ.bias + i * numel : nullptr;
    ba.se[i] = io.dQ.se ? io.dQ.se + i * numel : nullptr;
    ba.kmean[i] = io.dK.mean ? io.dK.mean + i * numel : nullptr;
    ba.kbias[i] = io.dK.bias ? io.dK.bias + i * numel : nullptr;
  }
  BS_TRY(launch_attn_bwd(ba, io.B, io.H, st));

  // se of dK over trials under N (App. C.4), the per-trial path: trial k's move of dK is the
  // key-major pass's R-bias term with dD_k in place of dD_R (-c (P dD_k)^T Q); shifted fp64 sums
  if (io.dK.se) {
    if (dk_trials) {
      AttnBwdArgs bt = ba;
      bt.k_only = 1;
      bt.dK_ref = w.dK_s;
      bt.dV = w.dV_s;
      bt.dD_N = nullptr;
      bt.sd_N = nullptr;
      bt.n_pol = 1;
      bt.pol[0] = BS_READ_R;
      bt.kmean[0] = nullptr;
      bt.kbias[0] = w.tdk;
      bt.mean[0] = bt.bias[0] = bt.se[0] = nullptr;
      for (int k = 1; k <= io.K; ++k) {
        bt.dD_R = w.dD_tr + (int64_t)(k - 1) * rows;
        BS_TRY(launch_attn_bwd(bt, io.B, io.H, st));
        BS_TRY(launch_trial_accum(w.tdk, 1, k, numel, w.d1, w.S1, w.S2, st));
      }
      BS_TRY(launch_trial_se(w.S1, w.S2, io.K, numel, w.sek, st));
    }
    for (int i = 0; i < io.n_pol; ++i) {
      float* dst = io.dK.se + i * numel;
      if (io.pol[i] == BS_READ_N)
        BS_TRY(launch_combine(w.sek, nullptr, nullptr, numel, dst, nullptr, nullptr, st));
      else
        BS_TRY(launch_fill2d(dst, 1, numel, numel, 0.0f, st));
    }
  }
  return BS_OK;
}

}  // namespace bsp
