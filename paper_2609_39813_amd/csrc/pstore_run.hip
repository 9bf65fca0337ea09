// The runner and C-ABI entry of the FP8 store of attention probabilities and its two uses
// (App. B.2-B.4): the forward's row statistics, the store of P and O = p_q V, the per-row sums,
// the bias fields with dQ, then dK and dV; each policy's estimate is the reference plus the
// field its two reads select.
#include "k_attn.h"
#include "k_pstore.h"

#define BS_TRY(x)               \
  do {                          \
    const bs_status _s = (x);   \
    if (_s != BS_OK) return _s; \
  } while (0)

namespace bsp {

namespace {

struct PstoreWs {
  u16 *Qt, *Kt, *Vt, *dOt;
  float *m, *l, *D, *DR, *E, *Ee, *Ps1, *Ga, *Ha, *Gb, *O;
  float* fld[PF_COUNT];
  uint32_t* ubits;
};

PstoreWs carve_pstore(Carver& c, int64_t bh, int S, int K, int causal, bool need_o) {
  PstoreWs w{};
  const int64_t Sp = round_up(S, PSTORE_T), rows = bh * S, numel = rows * PSTORE_T;
  const int nqb = (int)(Sp / PSTORE_T);
  w.Qt = c.take<u16>(bh * PSTORE_T * Sp);
  w.Kt = c.take<u16>(bh * PSTORE_T * Sp);
  w.Vt = c.take<u16>(bh * PSTORE_T * Sp);
  w.dOt = c.take<u16>(bh * PSTORE_T * Sp);
  for (float** p : {&w.m, &w.l, &w.D, &w.DR, &w.E, &w.Ee, &w.Ps1}) *p = c.take<float>(rows);
  for (float** p : {&w.Ga, &w.Ha, &w.Gb}) *p = c.take<float>((int64_t)K * rows);
  const int64_t nf = bh * pstore_tiles(nqb, causal) * PSTORE_T * PSTORE_T;
  for (int i = 0; i < PF_COUNT; ++i) w.fld[i] = c.take<float>(nf);
  w.ubits = c.take<uint32_t>((int64_t)((K + PSTORE_RC - 1) / PSTORE_RC) * nf);
  if (need_o) w.O = c.take<float>(numel);
  return w;
}

// the bias field a softmax's-backward read selects (PF_REF: the reference J(p) itself, no bias)
int softmax_field(int r) {
  switch (r) {
    case BS_SM_R: return PF_R;
    case BS_SM_N: return PF_N;
    case BS_SM_K: return PF_K;
    case BS_SM_J2: return PF_J2;
    case BS_SM_Q2: return PF_Q2;
    default: return PF_REF;
  }
}

}  // namespace

size_t pstore_ws_size(int B, int H, int S, int dh, int K, int causal) {
  if (B < 1 || H < 1 || S < 1 || dh != PSTORE_T || K < 1 || K > PSTORE_KMAX) return 0;
  Carver c;
  carve_pstore(c, (int64_t)B * H, S, K, causal ? 1 : 0, true);
  return c.used();
}

struct PstoreIO {
  const void *Q, *K, *V, *dO;
  int B, H, S, dh, causal;
  float scale;
  int fmt, fwd_mode;
  const bs_pstore_policy* pol;
  int n_pol, ntrial;
  uint64_t seed;
  uint32_t store_id;
  float *O, *P_out;
  uint8_t* P_codes;
  float* P_scale;
  float *dQ_ref, *dK_ref, *dV_ref;
  bs_est dQ, dK, dV;
  bs_diag* diag;
};

bs_status pstore_run(const PstoreIO& io, void* ws, size_t ws_bytes, hipStream_t st) {
  if (!io.Q || !io.K || !io.V || !io.dO || !io.P_codes || !io.dQ_ref || !io.dK_ref || !io.dV_ref || !io.diag ||
      !io.pol)
    return BS_EINVAL;
  if (io.B < 1 || io.H < 1 || io.S < 1 || io.ntrial < 1 || io.ntrial > PSTORE_KMAX) return BS_EINVAL;
  if (io.n_pol < 1 || io.n_pol > PSTORE_MAXPOL) return BS_EINVAL;
  if (!(io.scale > 0.0f) || (io.fmt != BS_E4M3 && io.fmt != BS_E5M2) ||
      (io.fwd_mode != BS_RNE && io.fwd_mode != BS_SR))
    return BS_EINVAL;
  for (int i = 0; i < io.n_pol; ++i) {
    if (io.pol[i].softmax_read < BS_SM_U || io.pol[i].softmax_read > BS_SM_Q2) return BS_EINVAL;
    if (io.pol[i].v_read < BS_READ_U || io.pol[i].v_read > BS_READ_N) return BS_EINVAL;
  }
  if (io.dh != PSTORE_T || io.S % 4 != 0) return BS_ESHAPE;
  if ((int64_t)io.B * io.H > 65535 || (io.S + PSTORE_T - 1) / PSTORE_T > 65535) return BS_ESHAPE;
  if (io.dQ.se || io.dK.se || io.dV.se) return BS_EUNSUPPORTED;
  for (const void* p : {io.Q, io.K, io.V, io.dO, (const void*)io.O, (const void*)io.P_out, (const void*)io.P_codes})
    if ((uintptr_t)p & 15) return BS_EINVAL;  // 16-byte vector loads and stores
  const int64_t bh = (int64_t)io.B * io.H, Sp = round_up(io.S, PSTORE_T), rows = bh * io.S, numel = rows * PSTORE_T;
  Carver probe;
  carve_pstore(probe, bh, io.S, io.ntrial, io.causal ? 1 : 0, !io.O);
  if (!ws || ((uintptr_t)ws & 255) || ws_bytes < probe.used()) return BS_EWORKSPACE;
  Carver c(ws, ws_bytes);
  const PstoreWs w = carve_pstore(c, bh, io.S, io.ntrial, io.causal ? 1 : 0, !io.O);

  // transposed operand copies, then the forward's row max and row sum
  {
    const u16* src[4] = {(const u16*)io.V, (const u16*)io.Q, (const u16*)io.K, (const u16*)io.dO};
    u16* dst[4] = {w.Vt, w.Qt, w.Kt, w.dOt};
    BS_TRY(launch_attn_transpose(src, dst, 4, (int)bh, io.S, (int)Sp, st));
  }
  AttnArgs fa{(const u16*)io.Q, (const u16*)io.K, (const u16*)io.V, io.S, io.causal, io.scale, w.m, w.l, nullptr,
              w.Vt, (int)Sp};
  BS_TRY(launch_attn_fwd(fa, io.B, io.H, st));

  PstoreArgs a{};
  a.Q = (const u16*)io.Q;
  a.K = (const u16*)io.K;
  a.V = (const u16*)io.V;
  a.dO = (const u16*)io.dO;
  a.Qt = w.Qt;
  a.Kt = w.Kt;
  a.Vt = w.Vt;
  a.dOt = w.dOt;
  a.S = io.S;
  a.Sp = (int)Sp;
  a.causal = io.causal ? 1 : 0;
  a.BH = (int)bh;
  a.scale = io.scale;
  a.m = w.m;
  a.l = w.l;
  a.f = f8_format(io.fmt);
  a.fmt = io.fmt;
  a.fwd_mode = io.fwd_mode;
  a.seed = io.seed;
  a.use_fwd = io.store_id * 256u;
  a.use_a = a.use_fwd + 1u;
  a.use_b = a.use_fwd + 2u;
  a.ntrial = io.ntrial;
  a.diag = io.diag;
  a.P_scale = io.P_scale;
  a.codes = io.P_codes;
  a.P_out = io.P_out;
  a.O = io.O ? io.O : w.O;
  a.D = w.D;
  a.DR = w.DR;
  a.E = w.E;
  a.Ee = w.Ee;
  a.Ps1 = w.Ps1;
  a.Ga = w.Ga;
  a.Ha = w.Ha;
  a.Gb = w.Gb;
  for (int i = 0; i < PF_COUNT; ++i) a.fld[i] = w.fld[i];
  a.ubits = w.ubits;
  for (int i = 0; i < io.n_pol; ++i) {
    const int sm = io.pol[i].softmax_read;
    a.draw_a |= (sm == BS_SM_N || sm == BS_SM_K || sm == BS_SM_J2 || sm == BS_SM_Q2 || io.pol[i].v_read == BS_READ_N);
    a.draw_b |= sm == BS_SM_J2;
  }
  a.dQ_ref = io.dQ_ref;
  a.dK_ref = io.dK_ref;
  a.dV_ref = io.dV_ref;
  a.n_pol = io.n_pol;
  for (int i = 0; i < io.n_pol; ++i) {
    const int vr = io.pol[i].v_read;
    a.sm_field[i] = softmax_field(io.pol[i].softmax_read);
    a.v_field[i] = vr == BS_READ_U ? 1 : (vr == BS_READ_N ? 2 : 0);
    auto at = [&](float* base) { return base ? base + (int64_t)i * numel : nullptr; };
    a.dQ.mean[i] = at(io.dQ.mean);
    a.dQ.bias[i] = at(io.dQ.bias);
    a.dK.mean[i] = at(io.dK.mean);
    a.dK.bias[i] = at(io.dK.bias);
    a.dV.mean[i] = at(io.dV.mean);
    a.dV.bias[i] = at(io.dV.bias);
  }

  BS_TRY(launch_pstore_scale(a, st));
  BS_TRY(launch_pstore_fwd(a, st));
  BS_TRY(launch_pstore_rows(a, st));
  BS_TRY(launch_pstore_dq(a, st));
  BS_TRY(launch_pstore_dkv(a, st));

  return BS_OK;
}

}  // namespace bsp

using namespace bsp;

extern "C" {

size_t bs_attn_pstore_workspace_size(int B, int H, int S, int dh, int K, int causal) {
  return pstore_ws_size(B, H, S, dh, K, causal);
}

bs_status bs_attn_pstore_policy(const void* Q, const void* Kt, const void* V, const void* dO, int B, int H, int S,
                                int dh, int causal, float softmax_scale, bs_fp8 fmt, bs_round fwd_mode,
                                const bs_pstore_policy* pol, int n_pol, int K, uint64_t seed, uint32_t store_id,
                                float* O, float* P_out, uint8_t* P_codes, float* P_scale, float* dQ_ref,
                                float* dK_ref, float* dV_ref, bs_est dQ, bs_est dK, bs_est dV, bs_diag* diag,
                                void* ws, size_t ws_bytes, void* stream) {
  PstoreIO io{Q,     Kt,      V,      dO,     B,      H,      S,      dh,     causal, softmax_scale, fmt, fwd_mode,
              pol,   n_pol,   K,      seed,   store_id, O,    P_out,  P_codes, P_scale, dQ_ref, dK_ref, dV_ref,
              dQ,    dK,      dV,     diag};
  return pstore_run(io, ws, ws_bytes, (hipStream_t)stream);
}

}  // extern "C"
