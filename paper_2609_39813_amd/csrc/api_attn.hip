// C-ABI entry point of the attention backward with a policy-dependent correction term.
#include "attn_run.h"

using namespace bsp;

extern "C" {

size_t bs_attn_workspace_size(int B, int H, int S, int dh, int n_pol, int K, int want_dk_se) {
  (void)n_pol;
  return attn_ws_size(B, H, S, dh, K, want_dk_se != 0);
}

bs_status bs_attn_bwd_policy(const void* Q, const void* Kt, const void* V, const void* dO, bs_dtype dO_type, int B,
                             int H, int S, int dh,
                             int causal, float softmax_scale, const float* O, bs_fp8 fmt, bs_round fwd_mode,
                             const bs_read* d_pol, int n_pol, int K, uint64_t seed, uint32_t store_id, float* O_out,
                             uint8_t* O_codes, float* O_scale, float* dQ_ref, float* dK_ref, float* dV, float* D_ref,
                             bs_est dQ, bs_est dK, bs_diag* diag, void* ws, size_t ws_bytes, void* stream) {
  if (dO && dO_type != BS_BF16 && dO_type != BS_F32) return BS_EDTYPE;
  const bool f32 = dO_type == BS_F32;
  AttnIO io{Q, Kt, V, f32 ? nullptr : dO, f32 ? (const float*)dO : nullptr, B, H, S, dh, causal, softmax_scale, O, fmt, fwd_mode, d_pol, n_pol, K, seed,
            store_id, O_out, O_codes, O_scale, dQ_ref, dK_ref, dV, D_ref, dQ, dK, diag};
  return attn_run(io, ws, ws_bytes, (hipStream_t)stream);
}

bs_status bs_attn_level2_policy(const void* Q, const void* Kt, const void* V, const void* dO, int B, int H, int S,
                                int dh, int causal, float softmax_scale, const float* O, bs_fp8 fmt, bs_round fwd_mode,
                                float beta, const bs_read* d_pol, int n_pol, int K, uint64_t seed, uint32_t store_id,
                                float* O_out, float* O_scale, float* dO_mean, float* dQ_ref, float* dK_ref, float* dV,
                                float* D_ref, bs_est dQ, bs_est dK, float* d_use, float* T, bs_diag* diag, void* ws,
                                size_t ws_bytes, void* stream) {
  if (!dO) return BS_EINVAL;
  AttnIO io{Q, Kt, V, dO, nullptr, B, H, S, dh, causal, softmax_scale, O, fmt, fwd_mode, d_pol, n_pol, K, seed,
            store_id, O_out, nullptr, O_scale, dQ_ref, dK_ref, dV, D_ref, dQ, dK, diag};
  io.level2 = 1;
  io.beta = beta;
  io.d_use = d_use;
  io.T = T;
  io.dO_mean = dO_mean;
  return attn_run(io, ws, ws_bytes, (hipStream_t)stream);
}

}  // extern "C"
