// C-ABI entry point of the attention backward with a policy-dependent correction term.
#include "bsp_kernels.h"
#include "k_attn.h"

using namespace bsp;

#define BS_TRY(x)               \
  do {                          \
    const bs_status _s = (x);   \
    if (_s != BS_OK) return _s; \
  } while (0)

namespace {
struct AttnWs {
  float *m, *l, *O, *D_ref, *dD_R, *dD_N, *sd_N;
};
AttnWs carve_attn(Carver& c, int64_t rows, int64_t numel, bool need_o, bool need_dref) {
  AttnWs w{};
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

extern "C" {

size_t bs_attn_workspace_size(int B, int H, int S, int dh, int n_pol, int K) {
  (void)n_pol;
  (void)K;
  if (B < 0 || H < 0 || S < 0 || dh < 0) return 0;
  Carver c;
  const int64_t rows = (int64_t)B * H * S;
  carve_attn(c, rows, rows * dh, true, true);
  return c.used();
}

bs_status bs_attn_bwd_policy(const void* Q, const void* Kt, const void* V, const void* dO, int B, int H, int S, int dh,
                             int causal, float softmax_scale, const float* O, bs_fp8 fmt, bs_round fwd_mode,
                             const bs_read* d_pol, int n_pol, int K, uint64_t seed, uint32_t store_id, float* O_out,
                             uint8_t* O_codes, float* O_scale, float* dQ_ref, float* dK_ref, float* dV, float* D_ref,
                             bs_est dQ, bs_est dK, bs_diag* diag, void* ws, size_t ws_bytes, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  if (!Q || !Kt || !V || !dO || !O_codes || !O_scale || !dQ_ref || !dK_ref || !dV || !diag || !d_pol) return BS_EINVAL;
  if (B < 1 || H < 1 || S < 1 || n_pol < 1 || n_pol > ATTN_MAX_POL || K < 1 || K > 4096) return BS_EINVAL;
  if (!(softmax_scale > 0.0f) || (fmt != BS_E4M3 && fmt != BS_E5M2) || (fwd_mode != BS_RNE && fwd_mode != BS_SR))
    return BS_EINVAL;
  if (dh != 64) return BS_ESHAPE;
  if ((int64_t)B * H > 65535) return BS_ESHAPE;
  if (dK.se) return BS_EUNSUPPORTED;
  bool want_r = false, want_n = false;
  for (int i = 0; i < n_pol; ++i) {
    if (d_pol[i] < BS_READ_U || d_pol[i] > BS_READ_N) return BS_EINVAL;
    want_r |= d_pol[i] == BS_READ_R;
    want_n |= d_pol[i] == BS_READ_N;
  }
  const int64_t rows = (int64_t)B * H * S, numel = rows * dh;
  const bool need_o = !O && !O_out;
  Carver probe;
  carve_attn(probe, rows, numel, need_o, !D_ref);
  if (!ws || ((uintptr_t)ws & 255) || ws_bytes < probe.used()) return BS_EWORKSPACE;
  Carver c(ws, ws_bytes);
  AttnWs w = carve_attn(c, rows, numel, need_o, !D_ref);
  float* dref = D_ref ? D_ref : w.D_ref;

  // forward: m, l (and O when the caller does not hand it in)
  AttnArgs fa{(const u16*)Q, (const u16*)Kt, (const u16*)V, S, causal, softmax_scale, w.m, w.l, nullptr};
  const float* Oorig = O;
  if (!O) {
    fa.O_out = O_out ? O_out : w.O;
    Oorig = fa.O_out;
  }
  BS_TRY(launch_attn_fwd(fa, B, H, st));
  if (O && O_out) {
    if (hipMemcpyAsync(O_out, O, sizeof(float) * numel, hipMemcpyDeviceToDevice, st) != hipSuccess) return BS_EHIP;
  }

  // the store of O (trial 0, use store_id*256), then the D variants
  const uint32_t base = store_id * 256u;
  BS_TRY(launch_store(Oorig, BS_F32, numel, fmt, fwd_mode, seed, 0, base, nullptr, O_codes, O_scale, diag, st, false));
  AttnDArgs da{Oorig, (const u16*)dO, O_codes, O_scale, rows, f8_format(fmt), seed, base + 1, K, want_n ? 1 : 0,
               dref, w.dD_R, w.dD_N, w.sd_N};
  BS_TRY(launch_attn_d(da, st));

  AttnBwdArgs ba{};
  ba.Q = (const u16*)Q;
  ba.K = (const u16*)Kt;
  ba.V = (const u16*)V;
  ba.dO = (const u16*)dO;
  ba.m = w.m;
  ba.l = w.l;
  ba.D_ref = dref;
  ba.dD_R = want_r ? w.dD_R : nullptr;
  ba.dD_N = want_n ? w.dD_N : nullptr;
  ba.sd_N = want_n ? w.sd_N : nullptr;
  ba.S = S;
  ba.causal = causal;
  ba.ntrial = K;
  ba.scale = softmax_scale;
  ba.dQ_ref = dQ_ref;
  ba.dK_ref = dK_ref;
  ba.dV = dV;
  ba.n_pol = n_pol;
  for (int i = 0; i < n_pol; ++i) {
    ba.pol[i] = d_pol[i];
    ba.mean[i] = dQ.mean ? dQ.mean + i * numel : nullptr;
    ba.bias[i] = dQ.bias ? dQ.bias + i * numel : nullptr;
    ba.se[i] = dQ.se ? dQ.se + i * numel : nullptr;
    ba.kmean[i] = dK.mean ? dK.mean + i * numel : nullptr;
    ba.kbias[i] = dK.bias ? dK.bias + i * numel : nullptr;
  }
  BS_TRY(launch_attn_bwd(ba, B, H, st));
  return BS_OK;
}

}  // extern "C"
