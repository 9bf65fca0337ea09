/*
 * bsp.h -- per-use backward-state checks of emulated FP8 rounding on MI355X (gfx950).
 *
 * A "use" is a gradient computation that reads a rounded tensor; the backward-state
 * policy chooses, per use, whether it reads the original (U), the rounding the forward
 * used (R) or a new rounding from the same law (N) (paper Sec. 1; Sec. 3.1; App. B).
 * The reference gradient is the gradient of the forward as it actually ran, with
 * gradients passed through every rounding unchanged (Sec. 1; App. B.2, Eq. app-ref).
 * Each call below runs an operator's backward for every requested policy over K Monte
 * Carlo roundings with the forward held fixed, and returns the reference gradient and
 * each policy's mean gradient, its bias against the reference and its standard error
 * over trials (App. C.4; App. D.4).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Every pointer is DEVICE memory owned by the caller, row-major and contiguous,
 *    unless its comment says "host". The library keeps no pointer after a call
 *    returns and allocates no device memory: scratch comes from the caller's workspace
 *    `ws` of `ws_bytes` bytes (256-byte aligned), sized by the matching
 *    *_workspace_size() query with the same shape arguments.
 *  - Every call enqueues its kernels on `stream` (a hipStream_t; NULL = the null
 *    stream) and returns without waiting. Results are valid after the stream syncs.
 *  - The return code reports only what the host can check: argument, shape, dtype,
 *    workspace and launch errors. On a non-OK return nothing has been enqueued.
 *    Conditions found on the device go to the caller's `bs_diag` (device memory),
 *    which every call that takes one overwrites completely.
 *  - Results are deterministic: the same inputs and seed give the same bits.
 *  - The random word of element e of a rounding is Philox4x32-10 (Salmon et al.,
 *    SC'11) keyed by the 64-bit seed, counter (e >> 2 as 64 bits, trial, use),
 *    output word e & 3. The forward's own rounding of store `store_id` uses trial 0
 *    and use id store_id*256; new roundings use trials 1..K and use ids
 *    store_id*256 + j, j >= 1, as each call states.
 *  - FP8 store: amax = max|x| over the whole tensor; s = fl32(amax / FMAX) (s = 1 when
 *    amax = 0); y = fl32(x / s); |y| > FMAX is clamped and counted; then round to
 *    nearest even, or stochastic rounding with P(up) = floor(frac * 2^32) / 2^32 where
 *    frac is y's position between its two neighbouring FP8 values (Sec. 2.1, App. D.2).
 *    Codes are OCP E4M3 (FMAX 448) or E5M2 (FMAX 57344); -0 is code 0x80.
 *  - Policy estimates are written to bs_est arrays laid out [n_pol][numel] in the
 *    order the policies are given. Any of mean/bias/se may be NULL (not written).
 */
#ifndef BSP_H
#define BSP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BS_OK = 0,
  BS_EINVAL = 1,        /* a NULL required pointer, negative size, bad enum or option */
  BS_ESHAPE = 2,        /* sizes the kernels do not support (stated per call) */
  BS_EDTYPE = 3,        /* dtype not supported by this call */
  BS_EUNSUPPORTED = 4,  /* a valid request the library does not implement */
  BS_EWORKSPACE = 5,    /* ws is NULL, misaligned or smaller than *_workspace_size() */
  BS_EHIP = 6           /* a HIP runtime error while enqueueing */
} bs_status;

typedef enum { BS_F32 = 0, BS_BF16 = 1 } bs_dtype;
typedef enum { BS_E4M3 = 0, BS_E5M2 = 1 } bs_fp8;
typedef enum { BS_RNE = 0, BS_SR = 1 } bs_round;
typedef enum { BS_READ_U = 0, BS_READ_R = 1, BS_READ_N = 2 } bs_read;

/* Device-side diagnostics of one store. nonfinite != 0: the tensor held a NaN or an
 * infinity and no codes were produced (outputs are then unspecified). n_saturated:
 * entries with |x/s| > FMAX, clamped to +-FMAX (App. D.2 counts such entries). */
typedef struct {
  uint32_t nonfinite;
  uint32_t n_saturated;
  float amax;
  float scale;
} bs_diag;

/* Per-policy estimate arrays, each [n_pol][numel] fp32, NULL = not wanted.
 * mean = (1/K) sum_k g_k; bias = mean - g_ref; se = sample standard deviation of g_k
 * over the K trials divided by sqrt(K) (App. C.4), 0 for a policy that draws nothing. */
typedef struct {
  float* mean;
  float* bias;
  float* se;
} bs_est;

const char* bs_status_string(bs_status s);
/* Library version (major*10000 + minor*100 + patch). */
int bs_version(void);

/* ------------------------------------------------------------------------------------
 * bs_qround -- the FP8 store of one tensor (Sec. 2.1; App. D.2, "at the TE output scale").
 *   x        [n] fp32 or bf16 (xt).
 *   fmt/mode format and rounding rule; seed/trial/use key the Philox words (SR only).
 *   scale_in NULL: s = amax/FMAX from x; else s = *scale_in (device fp32, > 0), a delayed
 *            scale: it replaces s only; amax and the NaN / infinity check still run over x.
 *   codes    [n] uint8 out.  scale_out [1] fp32 out (the s used).
 *   diag     [1] out: amax of x (also with scale_in), scale, nonfinite, n_saturated.
 * n may be 0 (diag then reports amax 0, scale 1, or *scale_in). No workspace.
 * ---------------------------------------------------------------------------------- */
bs_status bs_qround(const void* x, bs_dtype xt, int64_t n, bs_fp8 fmt, bs_round mode,
                    uint64_t seed, uint32_t trial, uint32_t use, const float* scale_in,
                    uint8_t* codes, float* scale_out, bs_diag* diag, void* stream);

/* ------------------------------------------------------------------------------------
 * bs_rmsnorm_linear_fwd_bwd -- RMSNorm feeding a Linear through an FP8 store of the
 * normalized output, and the two uses of that store (Sec. 3.1, Eq. norm-uses; App. D.4,
 * Table "Store policies"; App. E.4 for the norm-input reading R).
 *
 * Forward: z = x * r_t with r_t = 1/sqrt(mean_j x_tj^2 + eps); u = gain * z, computed in
 * fp32 in a fixed order (sum of squares in 64 lane-strided partials, partial l taking
 * j = l, l+64, ... ascending, combined pairwise with offsets 32, 16, ..., 1; every step
 * rounded to fp32, no fused multiply-add); (C_u, s) = FP8 store of u (trial 0, use
 * store_id*256); Y = deq(C_u) W.
 * Backward: du = dY W^T; reference dW = deq(C_u)^T dY, dgain = sum_t z du, dX = the
 * RMSNorm backward with the unrounded z. Per policy: the gain use reads z (U),
 * deq(C_u)/gain (R) or deq(C_f)/gain (N); the weight use reads u (U), deq(C_u) (R) or
 * deq(C_f') (N); the norm-input use reads z (U) or deq(C_u)/gain (R). A new rounding is
 * stochastic rounding of y = fl32(u/s) at the forward's scale; its use id is
 * store_id*256+1 at the gain use and store_id*256+2 at the weight use, or +1 for both
 * when fresh_shared != 0.
 *
 *   X [T,d] dt; gain [d] fp32; W [d,n] dt; dY [T,n] dt (dt fp32 or bf16).
 *   T >= 0; d and n multiples of 8 with 8 <= d <= 8192, 8 <= n; K in [1, 4096].
 *   dY NULL: forward only (u_codes, u_scale, Y, diag); the backward outputs are not written.
 *   pol (host) [n_pol], n_pol in [1, 16].
 *   Y [T,n] fp32 (nullable); u_codes [T,d] uint8; u_scale [1] fp32;
 *   dgain_ref [d], dW_ref [d,n], dX_ref [T,d] fp32; estimates dgain [n_pol][d],
 *   dW [n_pol][d*n], dX [n_pol][T*d]. The other estimates collapse the K trials by
 *   linearity; a non-NULL dW.se with a policy that reads N at the weight use runs the K
 *   per-trial contractions (App. C.4's sample SD over trials; K x 2 d n T flop more).
 * ---------------------------------------------------------------------------------- */
typedef struct {
  bs_read gain_use;
  bs_read weight_use;
  bs_read norm_input_use;  /* U (default of the paper) or R */
  int fresh_shared;        /* 1: both N uses read one new rounding */
} bs_norm_policy;

size_t bs_rmsnorm_linear_workspace_size(int64_t T, int64_t d, int64_t n, int n_pol, int K);
bs_status bs_rmsnorm_linear_fwd_bwd(const void* X, const float* gain, const void* W, const void* dY,
                                    bs_dtype dt, int64_t T, int64_t d, int64_t n, float eps,
                                    bs_fp8 fmt, bs_round fwd_mode, const bs_norm_policy* pol, int n_pol,
                                    int K, uint64_t seed, uint32_t store_id, float* Y, uint8_t* u_codes,
                                    float* u_scale, float* dgain_ref, float* dW_ref, float* dX_ref,
                                    bs_est dgain, bs_est dW, bs_est dX, bs_diag* diag, void* ws,
                                    size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------------------
 * bs_rmsnorm_linear_grid_fwd_bwd -- RMSNorm feeding a Linear through the paper's own store of
 * the normalized output: a per-token b-bit uniform grid with stochastic rounding (App. D.4),
 * and the eight policies of its Table "Store policies" (Sec. 3.1, Eq. norm-uses).
 *
 * Forward as bs_rmsnorm_linear_fwd_bwd up to u (same fixed fp32 order). Store, per token t:
 * s_t = fl32(max_j |u_tj| / M) with M = 2^(bits-1) - 1 (s_t = 1 for an all-zero row);
 * y = fl32(u / s_t); |y| > M is clamped and counted (diag.n_saturated); with lo = floor(|y|)
 * and F = floor((|y| - lo) 2^32) the code rounds up iff R + F >= 2^32 (R the element's Philox
 * word: trial 0, use store_id*256; element t*d + j); code q = sign * (lo + up) in [-M, M];
 * u_q = fl32(q s_t); Y = u_q W. Backward: du = dY W^T; dW = u_W^T dY; dgain = sum_t z_g du,
 * dX with the unrounded z. The new rounding u_f (trials 1..K, use store_id*256 + 1, the same
 * law) is read by both uses. Policies (gain use first): the gain use reads z (U), u_q/gain (R)
 * or u_f/gain (N); the weight use reads u (U), u_q (R), u_f (N) or u_q + (u_f - u) (R+eps).
 * U/R is the reference: dgain_ref = sum z du, dW_ref = u_q^T dY.
 *
 *   X [T,d] dt, gain [d] fp32, W [d,n] dt, dY [T,n] dt (dt fp32 or bf16); 1 <= T <= 2^24 - 256;
 *   d, n multiples of 8, d <= 8192; bits in [2, 8]; K in [1, 4096]; pol (host) [n_pol] in [1, 16].
 *   Y [T,n] fp32 (nullable); u_codes [T,d] int8; u_step [T] fp32; dgain_ref [d], dW_ref [d,n],
 *   dX_ref [T,d] fp32; estimates dgain [n_pol][d], dW [n_pol][d*n] (se must be NULL:
 *   BS_EUNSUPPORTED otherwise). diag: nonfinite, n_saturated, amax = max |u| (scale unused).
 *   ws: bs_rmsnorm_linear_grid_workspace_size(T, d, n) bytes.
 * ---------------------------------------------------------------------------------- */
typedef enum { BS_WREAD_U = 0, BS_WREAD_R = 1, BS_WREAD_N = 2, BS_WREAD_R_EPS = 3 } bs_weight_read;
typedef struct {
  bs_read gain_use;
  bs_weight_read weight_use;
} bs_grid_policy;

size_t bs_rmsnorm_linear_grid_workspace_size(int64_t T, int64_t d, int64_t n);
bs_status bs_rmsnorm_linear_grid_fwd_bwd(const void* X, const float* gain, const void* W, const void* dY, bs_dtype dt,
                                         int64_t T, int64_t d, int64_t n, float eps, int bits,
                                         const bs_grid_policy* pol, int n_pol, int K, uint64_t seed,
                                         uint32_t store_id, float* Y, int8_t* u_codes, float* u_step,
                                         float* dgain_ref, float* dW_ref, float* dX_ref, bs_est dgain, bs_est dW,
                                         bs_diag* diag, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------------------
 * bs_attn_bwd_policy -- attention backward whose correction term D reads a stored
 * copy of the output (Sec. 2.1, Eq. dterm; App. D.2).
 *
 * Scores S = c Q K^T (c = softmax_scale; causal: key j <= query i), P = softmax(S),
 * O = P V. The store is the FP8 store of the fp32 O (mode fwd_mode, trial 0, use
 * store_id*256). Backward: dV = P^T dO, dP = dO V^T, dS = P * (dP - D), dQ = c dS K,
 * dK = c dS^T Q. The reference takes D = rowsum(dO * O) with the original O. Policy U
 * reads O, R the forward's rounding deq(C_O), N a new stochastic rounding at the same
 * scale (trials 1..K, use store_id*256+1). dV does not depend on the policy.
 *
 *   Q, Kt, V [B,H,S,dh] bf16; dO [B,H,S,dh] bf16 or fp32 (dO_type; fp32 enters the
 *   contractions as three exact bf16 terms). dO NULL: forward and store only (O_out,
 *   O_codes, O_scale, diag). dh == 64; S >= 1; B, H >= 1.
 *   O [B,H,S,dh] fp32: the original output to store; NULL = computed by the library's
 *   forward (written to O_out if O_out != NULL).
 *   d_pol (host) [n_pol] in {U, R, N}, n_pol in [1, 8]; K in [1, 4096].
 *   O_codes [B,H,S,dh] uint8; O_scale [1]; dQ_ref, dK_ref, dV [B,H,S,dh] fp32;
 *   D_ref [B,H,S] fp32 (nullable); estimates dQ, dK [n_pol][B*H*S*dh]. dQ's se under N is
 *   exact from the trial SD of the rows' dD (dQ moves by -c dD_k P K, row-scaled); a non-NULL
 *   dK.se runs the per-trial path: trial k's move -c (P dD_k)^T Q by one key-major pass per
 *   trial, shifted fp64 sums (App. C.4), with workspace
 *   bs_attn_workspace_size(..., want_dk_se = 1); 0 for U and R.
 * ---------------------------------------------------------------------------------- */
size_t bs_attn_workspace_size(int B, int H, int S, int dh, int n_pol, int K, int want_dk_se);
bs_status bs_attn_bwd_policy(const void* Q, const void* Kt, const void* V, const void* dO, bs_dtype dO_type,
                             int B, int H, int S, int dh, int causal, float softmax_scale, const float* O, bs_fp8 fmt,
                             bs_round fwd_mode, const bs_read* d_pol, int n_pol, int K, uint64_t seed,
                             uint32_t store_id, float* O_out, uint8_t* O_codes, float* O_scale,
                             float* dQ_ref, float* dK_ref, float* dV, float* D_ref, bs_est dQ, bs_est dK,
                             bs_diag* diag, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------------------
 * bs_attn_level2_policy -- the D use of the attention output store averaged over the
 * forward's own rounding as well (App. C.1's level of averaging, the forward's inputs fixed),
 * with an incoming gradient that can depend on that rounding (Sec. 4.2; App. B.3), and the
 * split of the use's average error into a mean error and a coupling (App. C.1).
 *
 * As bs_attn_bwd_policy, except: in trial k = 1..K the forward's store of O rounds anew
 * (mode fwd_mode, trial k, use store_id*256; scale s from amax(O) as always) with error
 * r_k = deq(C_k) - O, and the incoming gradient is g_k = dO + beta r_k (beta = 0: fixed;
 * beta = 1: the output's deviation added, as the loss 1/2 ||o||^2 gives up to its fixed part).
 * U reads O, R reads deq(C_k), N a new rounding (trial k, use store_id*256 + 1). Each trial's
 * reference is the backward of the forward as it ran (incoming g_k, D_ref,k = rowsum(g_k O)).
 * Outputs are means over the K trials: dQ_ref, dK_ref, dV (= P^T mean g), D_ref; per policy
 * dQ, dK mean and bias (the mean of the per-trial difference; se must be NULL). For the D use
 * of each policy, d_use [n_pol][4][B*H*S]: the mean of its error rowsum(g_k e_k) (e_k the
 * copy's deviation from O), the mean-error part rowsum(mean e * mean g), the coupling (the
 * remainder) and the se over trials of the error. T [2][B*H*S]: mean and se of the paired
 * statistic T_k = 1/2 rowsum((r_k - r'_k)(g(O + r_k) - g(O + r'_k))) of App. E.4, whose mean
 * is R's error minus N's. dO_mean [B,H,S,dh] (nullable): the mean incoming gradient.
 *
 *   Q, Kt, V, dO bf16 [B,H,S,dh], dh == 64; O, O_out, D_ref as bs_attn_bwd_policy; O_scale [1].
 *   d_pol (host) [n_pol] in {U, R, N}, n_pol in [1, 8]; K in [1, 4096].
 *   Workspace: bs_attn_workspace_size(B, H, S, dh, n_pol, K, 0).
 * Returns BS_EINVAL for a NULL dO or a NaN beta; otherwise as bs_attn_bwd_policy.
 * ---------------------------------------------------------------------------------- */
bs_status bs_attn_level2_policy(const void* Q, const void* Kt, const void* V, const void* dO, int B, int H, int S,
                                int dh, int causal, float softmax_scale, const float* O, bs_fp8 fmt, bs_round fwd_mode,
                                float beta, const bs_read* d_pol, int n_pol, int K, uint64_t seed, uint32_t store_id,
                                float* O_out, float* O_scale, float* dO_mean, float* dQ_ref, float* dK_ref, float* dV,
                                float* D_ref, bs_est dQ, bs_est dK, float* d_use, float* T, bs_diag* diag, void* ws,
                                size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------------------
 * bs_logsoftmax_reuse_check -- the log-softmax operator test (Sec. 4.3; App. C.5), in fp64.
 * The operator's backward returns h - exp(S) (1^T h) from a saved output S. Per trial k =
 * 1..K the saved output is S = l + r with l = log_softmax(logits) per row and r_j = +eps where
 * the element's Philox word (trial k, use store_id*256; element row*C + j) is >= 2^31, -eps
 * otherwise; reuse reads S, an independent copy reads l + r' (use store_id*256 + 1). With p =
 * exp(l), g the returned gradient and g* the operator's gradient from l, the trial's statistic
 * is the mean over rows and classes of (g - g*)/p for: [0] the likelihood (h = -e_y, y =
 * target) with reuse, [1] the likelihood with the independent copy, [2] the constructed loss
 * (h = r) with reuse, [3] the constructed loss with the independent copy. calibrate != 0
 * divides the reconstruction exp(S) by cosh(eps) (LS5a/LS5b).
 *
 *   logits [rows, C] fp64; target [rows] int32 (a value outside [0, C) matches no class);
 *   rows >= 1; C >= 4 a multiple of 4; 0 < eps < 1; K in [1, 2^20].
 *   stats [4][2] fp64 (device): mean over the K trials and its se (sample SD / sqrt(K)).
 *   ws: bs_logsoftmax_check_workspace_size(rows, C, K) bytes (0 for shapes the call rejects).
 * Returns BS_EINVAL for a NULL pointer or eps, K out of range; BS_ESHAPE for C.
 * ---------------------------------------------------------------------------------- */
size_t bs_logsoftmax_check_workspace_size(int64_t rows, int C, int K);
bs_status bs_logsoftmax_reuse_check(const double* logits, const int32_t* target, int64_t rows, int C, double eps,
                                    int K, uint64_t seed, uint32_t store_id, int calibrate, double* stats, void* ws,
                                    size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------------------
 * bs_attn_pstore_policy -- attention whose probabilities P pass through an FP8 store, and
 * the two uses of that store in the backward: the gradient of V and the softmax's backward
 * (App. B.2, Eq. app-ref and Eq. app-errors; App. B.3; App. B.4; Table app-theory-errors).
 *
 * Forward: P = softmax(c Q K^T) (causal: key j <= query i), computed in fp32 with the row
 * max m of x = fl32(c log2(e) S) and row sum l, p = fl32(2^(x - m)) / l rounded once more to
 * fp32 (so the largest entry of a row is exactly fl32(1/l)). (C_P, s) = FP8 store of P
 * (amax = max P, mode fwd_mode, trial 0, use store_id*256; element ((b H + h) S + i) S + j).
 * O = deq(C_P) V (the forward as it ran: p_q = deq(C_P)).
 * Backward with the forward held fixed and the incoming gradient dO: dp = dO V^T per row;
 * reference dV_ref = p_q^T dO, ds = J(p) dp with J(x) = diag(x) - x x^T, dQ_ref = c ds K,
 * dK_ref = c ds^T Q. A policy names the softmax's backward read first, then the dV read:
 *   softmax  U J(p)   R J(p_q)   N J(a)   K K(a) = diag(a 1^T a) - a a^T
 *            J2 (a+b)/2 diag - (a b^T + b a^T)/2 = J2(a, b)    Q2 J2(p_q, a)
 *   dV       U p      R p_q      N a
 * where a and b are new stochastic roundings of y = fl32(P/s) at the forward's scale, trial
 * k = 1..K, use ids store_id*256+1 (a) and +2 (b); a policy that reads N at both uses reads
 * the same a. The mean over the K trials is formed exactly from per-row and per-element sums
 * of the up-decisions (every trial's rounding is drawn; no trial's gradient materializes).
 *
 *   Q, Kt (the keys), V, dO [B,H,S,dh] bf16, 16-byte aligned; dh == 64; S >= 4 a multiple of 4;
 *   B*H <= 65535. pol (host) [n_pol], n_pol in [1, 8]; K in [1, 32].
 *   O [B,H,S,dh] fp32 (nullable); P_out [B,H,S,S] fp32 (nullable): the realized P;
 *   P_codes [B,H,S,S] uint8 (zero above the causal diagonal); P_scale [1] fp32 (nullable);
 *   dQ_ref, dK_ref, dV_ref [B,H,S,dh] fp32; estimates dQ, dK, dV [n_pol][B*H*S*dh]
 *   (se must be NULL: BS_EUNSUPPORTED otherwise). diag: the store's amax, scale, saturations;
 *   nonfinite != 0 when a row sum is not a positive finite number (then nothing else is written).
 *   ws: bs_attn_pstore_workspace_size(B, H, S, dh, K, causal) bytes (0 for shapes the call
 *   rejects); about 8 causal-half S^2 fp32 fields per head plus 12 [B,H,S,dh] fp32 arrays.
 * Returns BS_EINVAL for a null required pointer, a bad enum, K or n_pol out of range or a
 * misaligned pointer; BS_ESHAPE for dh != 64 or S not a multiple of 4.
 * ---------------------------------------------------------------------------------- */
typedef enum { BS_SM_U = 0, BS_SM_R = 1, BS_SM_N = 2, BS_SM_K = 3, BS_SM_J2 = 4, BS_SM_Q2 = 5 } bs_softmax_read;
typedef struct {
  bs_softmax_read softmax_read;
  bs_read v_read;
} bs_pstore_policy;

size_t bs_attn_pstore_workspace_size(int B, int H, int S, int dh, int K, int causal);
bs_status bs_attn_pstore_policy(const void* Q, const void* Kt, const void* V, const void* dO, int B, int H, int S,
                                int dh, int causal, float softmax_scale, bs_fp8 fmt, bs_round fwd_mode,
                                const bs_pstore_policy* pol, int n_pol, int K, uint64_t seed, uint32_t store_id,
                                float* O, float* P_out, uint8_t* P_codes, float* P_scale, float* dQ_ref,
                                float* dK_ref, float* dV_ref, bs_est dQ, bs_est dK, bs_est dV, bs_diag* diag,
                                void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------------------
 * bs_te_attn_bwd -- an emulation of an FP8 attention backward with delayed scaling, whose
 * correction term D reads a saved copy of the output (App. D.2, the forks' dense backward;
 * App. E.3, the saturated-row repair).
 *
 * With scales = (s_P, s_dO, s_dS, s_g) (device fp32, > 0; delayed scales from the caller's
 * amax histories) and Q8(x; s, F) = s * RNE_F(clamp(fl32(x / s), +-FMAX_F)):
 *   the operands Q, K, V are the forward's FP8 tensors, read as their dequantized values
 *   (qkv_scales != NULL: E4M3 codes at scales s_Q, s_K, s_V; App. D.2 recomputes the output from
 *   the dequantized FP8 Q, K and V), or bf16 tensors (qkv_scales NULL);
 *   dO_q = Q8(dO; s_dO, E5M2); P re-formed from Q, K (the forward's realized fp32 probabilities);
 *   P_q = Q8(P; s_P, E4M3); dV = P_q^T dO_q; dP = dO_q V^T; dS = P (dP - D) (zero above the
 *   causal diagonal); dS_q = Q8(dS; s_dS, E5M2); dQ = c dS_q K; dK = c dS_q^T Q; the three
 *   gradients return as the fp32 dequantization fl32(val(C) s_g) of C = RNE_E5M2(clamp(fl32(g /
 *   s_g))), in BF16 (grad_type BS_BF16, rounded to nearest even: App. D.2 returns them in BF16)
 *   or in fp32 (BS_F32).
 *   FP8 operands enter the products as their exact code values with the scales applied in fp32
 *   after the accumulation (s_Q s_K on the scores, s_V on dP and on P V, s_K on dQ, s_Q on dK), so
 *   the results differ from fp32-dequantized operands by rounding only.
 * D per row, by source: FROM_P rowsum(dO_q * P V) (equal to rowsum(P dP)); U rowsum(dO_q * O);
 *   R rowsum(dO_q * deq(O_codes)); N rowsum(dO_q * N(O)), N(O) a new stochastic rounding of
 *   fl32(O / O_scale) in E4M3 (trial `trial`, use store_id*256 + 1, element b,h,s,d row-major);
 *   REPAIR FROM_P on rows whose largest probability (exactly fl32(1/l)) is >= threshold, R on
 *   the others.
 *
 *   Q, Kt (the keys), V [B,H,S,dh] bf16, or uint8 E4M3 codes with qkv_scales [3] fp32 (device);
 *   dO [B,H,S,dh] bf16; all 16-byte aligned; dh == 64; S >= 4 a multiple of 4;
 *   B*H <= 65535. O [B,H,S,dh] fp32 (U, N; else nullable); O_codes [B,H,S,dh] uint8 E4M3
 *   (R, REPAIR) and O_scale [1] fp32 device (R, N, REPAIR): the forward's store of O.
 *   dQ, dK, dV [B,H,S,dh] out, bf16 or fp32 (grad_type): the returned (cast) gradients.
 *   amax [4] fp32 out, in the order of scales: max P (= max over rows of fl32(1/l)), max |dO|,
 *   max |dS| (pre-cast), max of the pre-cast gradients.
 *   counts [4] uint32 out: rows with fl32(1/l) >= threshold; clamped entries of dO, of dS and of
 *   the three gradients.
 *   Nullable outputs: P_out, dS_out [B,H,S,S] fp32 (the realized P and pre-cast dS), P_codes,
 *   dS_codes [B,H,S,S] uint8 (4-byte aligned) and grad_pre [3][B,H,S,dh] fp32 (pre-cast dQ,
 *   dK, dV); [B,H,S,S] entries above the causal diagonal's 64 x 64 tiles are not written.
 *   ws: bs_te_attn_workspace_size(B, H, S, dh, causal, source, fp8_qkv) bytes, fp8_qkv != 0 when
 *   qkv_scales is set (0 for shapes the call rejects); about 2 causal-half S^2 bytes per head
 *   plus 7 (10 with FP8 operands) [B,H,S,dh] bf16/fp32 arrays.
 * Returns BS_EINVAL for a null required pointer, a bad source, a misaligned pointer;
 * BS_EDTYPE for a grad_type other than BS_F32 / BS_BF16; BS_ESHAPE for dh != 64 or S not a
 * multiple of 4.
 * ---------------------------------------------------------------------------------- */
typedef enum { BS_D_FROM_P = 0, BS_D_U = 1, BS_D_R = 2, BS_D_N = 3, BS_D_REPAIR = 4 } bs_d_source;

/* bs_te_delayed_scales -- one step of delayed scaling for the four tensors of bs_te_attn_bwd
 * (TE's recipe as the forks ran it, App. D.1: amax history of `len` steps, the maximum, margin 0).
 *   amax [4] fp32 device (P, dO, dS, gradients: bs_te_attn_bwd's amax output); history [4][len]
 *   fp32 device, a ring buffer the caller zeroes once; scales [4] fp32 device, in/out.
 * The step's amax is stored at history[i][step % len]; then scales[i] = fl32(m_i / FMAX_i) with
 * m_i the largest |amax| in history i (FMAX 448 for P, 57344 for the others), left unchanged when
 * m_i is zero, infinite or NaN (a non-finite amax stays in the history). len >= 1, step >= 0.
 * Returns BS_EINVAL for a NULL pointer or a bad len / step. No workspace. */
bs_status bs_te_delayed_scales(const float* amax, float* history, int len, int64_t step, float* scales,
                               void* stream);

size_t bs_te_attn_workspace_size(int B, int H, int S, int dh, int causal, bs_d_source source, int fp8_qkv);
bs_status bs_te_attn_bwd(const void* Q, const void* Kt, const void* V, const float* qkv_scales, const void* dO, int B,
                         int H, int S, int dh, int causal, float softmax_scale, const float* O, const uint8_t* O_codes,
                         const float* O_scale, bs_d_source source, float threshold, const float* scales, uint64_t seed,
                         uint32_t store_id, uint32_t trial, bs_dtype grad_type, void* dQ, void* dK, void* dV,
                         float* amax, uint32_t* counts, float* P_out, float* dS_out, uint8_t* P_codes,
                         uint8_t* dS_codes, float* grad_pre, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------------------
 * bs_linear_bwd_policy -- Linear backward whose incoming gradient is stochastically
 * rounded to FP8 (E5M2 in the HYBRID recipe, App. D.1), read by two uses.
 *
 * y = X W. The reference uses the unrounded dY: dX_ref = dY W^T, dW_ref = X^T dY. In
 * trial k the rounding C_k of dY (per-tensor scale s = amax(dY)/FMAX) is read by
 * dX_k = deq(C_k) W^T and dW_k = X^T deq(C'_k): shared (sharing 0) means C' = C (use id
 * store_id*256+1); per use (sharing 1) draws C' separately (use id store_id*256+2).
 * Coupling: kappa = mean_k <dX_k - dX_ref, A> <dW_k - dW_ref, B> for fixed probes A, B
 * (the coupling part of the error split of App. C.1; App. C.2's two-stage example).
 *
 *   X [M,k] dt, W [k,n] dt, dY [M,n] dt; dt bf16; k and n multiples of 8; M >= 0.
 *   sharing (host) [n_pol] in {0, 1}, n_pol in [1, 4]; K in [1, 4096].
 *   dX_ref [M,k], dW_ref [k,n] fp32; estimates dX [n_pol][M*k], dW [n_pol][k*n]. The means
 *   collapse the K trials by linearity; a non-NULL dX.se or dW.se runs the per-trial path (App.
 *   C.4's sample SD over trials / sqrt(K)): trial k's residual fresh_k - dY moves dX and dW by K
 *   per-trial contractions (2 M k n flop each per gradient, three bf16 terms), and its
 *   workspace is bs_linear_bwd_workspace_size(..., want_se = 1).
 *   probeA [M,k], probeB [k,n] fp32 and coupling [n_pol] fp64: all NULL or all set.
 *   dY_scale [1] fp32 out.
 * ---------------------------------------------------------------------------------- */
size_t bs_linear_bwd_workspace_size(int64_t M, int64_t k, int64_t n, int n_pol, int K, int want_se);
bs_status bs_linear_bwd_policy(const void* X, const void* W, const void* dY, bs_dtype dt, int64_t M,
                               int64_t k, int64_t n, bs_fp8 fmt, const int* sharing, int n_pol, int K,
                               uint64_t seed, uint32_t store_id, float* dX_ref, float* dW_ref, bs_est dX,
                               bs_est dW, const float* probeA, const float* probeB, double* coupling,
                               float* dY_scale, bs_diag* diag, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------------------
 * bs_policy_bias_estimate -- trial statistics of any use (App. C.4; App. D.4).
 *   delta [K][m] fp32: per-trial gradient minus the reference, trials in order.
 *   g_ref [m] (nullable, only for its norm). mean_err [m] out; se [m] out (nullable).
 *   summary [3] fp64 out: ||mean_err||_2, ||g_ref||_2 (0 if g_ref NULL), and
 *   R = ||mean_err||^2 / sum_j se_j^2 (NaN when the sum is 0).
 *   K >= 1, m >= 0. Sums run in a fixed order (deterministic).
 * ---------------------------------------------------------------------------------- */
/* ------------------------------------------------------------------------------------
 * bs_estimate_summary -- App. D.4's detection summary of any call's estimate of one gradient
 * (for instance one policy's slice of a bs_est):
 *   bias [n] (required when n > 0), se [n] and ref [n] (each nullable: treated as zero) fp32.
 *   summary [3] fp64 out (device): ||bias||_2, ||ref||_2, R = ||bias||^2 / sum_j se_j^2 (NaN
 *   when the sum is 0: no spread over trials, e.g. a policy that draws nothing). Fixed-order sums.
 *   ws: bs_estimate_summary_workspace_size() bytes, 256-byte aligned. n >= 0.
 * ---------------------------------------------------------------------------------- */
size_t bs_estimate_summary_workspace_size(void);
bs_status bs_estimate_summary(const float* bias, const float* se, const float* ref, int64_t n, double* summary,
                              void* ws, size_t ws_bytes, void* stream);

size_t bs_policy_bias_workspace_size(int K, int64_t m);
bs_status bs_policy_bias_estimate(const float* delta, int K, int64_t m, const float* g_ref, float* mean_err,
                                  float* se, double* summary, void* ws, size_t ws_bytes, void* stream);

/* bs_policy_bias_estimate_noalloc -- bs_policy_bias_estimate for callers that cannot allocate:
 * code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc. It takes no
 * workspace and allocates nothing: its scratch (the per-block partials) is a file-scope device
 * array of the library, 6 MiB, which each GPU the library runs on holds until the process ends.
 * Arguments and results as bs_policy_bias_estimate; m <= bs_policy_bias_noalloc_max() (2^26),
 * BS_ESHAPE above. Calls on one GPU share that GPU's scratch: calls that overlap in time on one
 * GPU (different streams without ordering, several host threads) race and must not be issued;
 * calls ordered on one stream are safe. The first call on a device looks up the array's address
 * on that device (BS_EHIP if that fails). */
int64_t bs_policy_bias_noalloc_max(void);
bs_status bs_policy_bias_estimate_noalloc(const float* delta, int K, int64_t m, const float* g_ref, float* mean_err,
                                          float* se, double* summary, void* stream);

/* ------------------------------------------------------------------------------------
 * bs_gemm_bf16_nt -- the contraction the backward uses for dW/dX/du (building block).
 *   C[M,N] = alpha * A[M,K] B[N,K]^T (+ C if accumulate), A and B bf16 with K contiguous
 *   (leading dimensions lda, ldb in elements), C fp32 with leading dimension ldc.
 *   K, lda, ldb multiples of 8; M, N, K >= 0.
 * ---------------------------------------------------------------------------------- */
bs_status bs_gemm_bf16_nt(const void* A, int64_t lda, const void* B, int64_t ldb, float* C, int64_t ldc,
                          int64_t M, int64_t N, int64_t K, float alpha, int accumulate, void* stream);

/* ------------------------------------------------------------------------------------
 * bs_decoder_layer_policy -- one pre-norm decoder layer (RMSNorm, causal multi-head attention
 * with dh = 64, SwiGLU MLP, no biases; the block of App. D.1) with four FP8 stores, and the
 * per-use check of every store (Sec. 4.1): each use is evaluated at its own operator with the
 * incoming gradient the straight-through reference backward delivers there.
 *
 *   u1 = gain1*RMSNorm(x)  [store 0]  QKV = deq(C_u1) Wqkv;  Q, K, V = bf16(QKV) per head
 *   O = softmax(c Q K^T) V [store 1]  h = x + deq(C_O) Wo
 *   u2 = gain2*RMSNorm(h)  [store 2]  [g | hh] = deq(C_u2) [Wg | Wu];  a = silu(g) * hh
 *   a                      [store 3]  out = h + deq(C_a) Wd
 *
 * Every store rounds with fwd_mode at trial 0, use store*256. Uses and their new roundings:
 *   store 0 and 2 (normalization stores): gain use (+1), weight use (+2), normalization-input
 *   use (U or R only), as bs_rmsnorm_linear_fwd_bwd; store 1: D use (+1, head-major element
 *   order) as bs_attn_bwd_policy with the fp32 incoming gradient, weight use of Wo (+2,
 *   token-major order); store 3: weight use of Wd (+2).
 *
 *   x [T, d] bf16 with T = B*S (row t = b*S + s); dOut [T, d] bf16; d = 64*H, d and F
 *   multiples of 8; weights bf16 row-major Wqkv [d, 3d], Wo [d, d], Wg [d, F], Wu [d, F],
 *   Wd [F, d]; gains fp32 [d]. K in [1, 4096].
 *   fixed (nullable): the realized forward to hold fixed instead of computing it (all of
 *   its pointers set): Q, K, V bf16 [B, H, S, 64], O fp32 [B, H, S, 64], h fp32 [T, d],
 *   gh = [g | hh] fp32 [T, 2F], a fp32 [T, F].
 *   grads: reference gradients (each nullable): dx [T,d], dgain1 [d], dWqkv [d,3d], dWo [d,d],
 *   dgain2 [d], dWg [d,F], dWu [d,F], dWd [F,d].
 *   stores (each nullable): codes of u1 [T,d], O [B,H,S,64], u2 [T,d], a [T,F]; scales [4].
 *   table [BS_LAYER_ROWS][3 letters U,R,N][3] fp64: sum of squared bias, sum of squared
 *   reference, sum of squared se of the row's gradient under the letter; NaN where there is no
 *   estimate: N at a normalization-input use (read unrounded, App. D.4), and, unless
 *   per_use_se is set, the se of a weight use and of dK under N.
 *   per_use_se != 0: those se by per-trial paths (App. C.4): at each weight use trial k's
 *   residual enters its own contraction with the incoming gradient, at the D use one key-major
 *   attention pass per trial gives dK; shifted fp64 sums over the K trials. Costs K extra
 *   contractions per weight use and K key-major passes.
 *   Rows: 0 u1 gain, 1 u1 weight (dWqkv), 2 u1 norm-input (dX), 3 O D (dQ), 4 O D (dK),
 *   5 O weight (dWo), 6 u2 gain, 7 u2 weight ([dWg | dWu]), 8 u2 norm-input, 9 a weight (dWd).
 *   all (nullable): each letter read at every use of every store together, in one backward whose
 *   moved incoming gradients reach the earlier uses (the policy applied to every stored
 *   tensor): U reads every original, R every forward rounding, N per use a new rounding (trials
 *   1..K; use +1 at a gain use and at the D use, +2 at a weight use, +3 at a normalization-input
 *   use). Per letter l (U, R, N): bias[l] (mean over trials minus the reference) and se[l] of each
 *   of dx, dgain1, dWqkv, dWo, dgain2, dWg, dWu, dWd (each nullable; se 0 for U and R, NaN where
 *   N has no estimate: dWd, dWg, dWu, whose incoming gradients do not move, as at the per-use
 *   weight uses); table [8][3][3] fp64 (nullable) in that gradient order: sum of squared bias,
 *   squared reference, squared se. Runs K + 2 backward passes of the moved part of the layer.
 *   diags [4] (nullable; one per store). Every pointer is device memory (the structs themselves
 *   are host memory); outputs are owned by the caller.
 *   ws: device workspace, 256-byte aligned, of bs_decoder_layer_workspace_size(B,S,d,H,F,K,
 *   options) bytes, options = BS_LAYER_ALL_USES when `all` is set | BS_LAYER_PER_USE_SE when
 *   per_use_se is (0 for shapes the call rejects).
 *   Returns BS_EINVAL for a null required pointer, K outside [1, 4096], eps < 0, an unknown
 *   format or mode, or a partly set `fixed`; BS_ESHAPE unless d = 64*H <= 8192, F a multiple of
 *   8 and B*H <= 65535; BS_EWORKSPACE for a short or misaligned workspace; BS_EHIP on a failed
 *   launch. Work is enqueued on `stream` (nullable: the null stream) and is asynchronous.
 * ---------------------------------------------------------------------------------- */
#define BS_LAYER_ROWS 10
typedef struct {
  const float* gain1;
  const void* Wqkv;
  const void* Wo;
  const float* gain2;
  const void* Wg;
  const void* Wu;
  const void* Wd;
} bs_layer_weights;
typedef struct {
  const void *Q, *K, *V;
  const float *O, *h, *gh, *a;
} bs_layer_forward;
typedef struct {
  float *dx, *dgain1, *dWqkv, *dWo, *dgain2, *dWg, *dWu, *dWd;
} bs_layer_grads;
typedef struct {
  uint8_t *u1, *O, *u2, *a;
  float* scales;
} bs_layer_stores;
typedef struct {
  bs_layer_grads bias[3];  /* U, R, N */
  bs_layer_grads se[3];
  double* table;           /* [8][3][3] */
} bs_layer_all;

#define BS_LAYER_ALL_USES 1   /* workspace option: the every-use-at-once check */
#define BS_LAYER_PER_USE_SE 2 /* workspace option: the per-use se of the weight uses and of dK */
size_t bs_decoder_layer_workspace_size(int B, int S, int d, int H, int F, int K, int options);
bs_status bs_decoder_layer_policy(const void* x, const bs_layer_weights* w, const void* dOut, int B, int S, int d,
                                  int H, int F, float eps, bs_fp8 fmt, bs_round fwd_mode, int K, uint64_t seed,
                                  const bs_layer_forward* fixed, bs_layer_grads grads, bs_layer_stores stores,
                                  double* table, const bs_layer_all* all, int per_use_se, bs_diag* diags, void* ws,
                                  size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------------------
 * Kernel timing instrumentation (host calls; for benchmarks and profiling).
 *   bs_profile_enable(1) clears earlier records and starts recording a pair of HIP
 *   events on the launch stream around each launch of the instrumented kernels
 *   ("fresh_count", "fresh_count_se", "fresh_count_kappa", "amax", "quantize", "gemm",
 *   "rmsnorm_fwd", "attn_fwd", "attn_bwd", "attn_l2", "pstore_fwd", "pstore_rows", "pstore_dq",
 *   "pstore_dkv", "lsm_prep", "lsm_trial", "grid_store", "grid_fresh", "te_prep", "te_d", "te_dq",
 *   "te_dkv", "lsm_reduce");
 *   bs_profile_enable(0) stops and frees them. bs_profile_read waits for the recorded
 *   events of `kernel` (NULL: all) and returns their summed elapsed time and count.
 *   bs_profile_work returns the summed algorithmic work of those launches (work): for "gemm",
 *   2 M N K flop per distinct product (the extra terms of a split bf16 operand do not count), and
 *   the work the matrix cores execute (exec: 2 M N K per bf16 term product); 0 for kernels that
 *   record none. Either pointer may be NULL. Return values are bs_status codes.
 * ---------------------------------------------------------------------------------- */
int bs_profile_enable(int on);
int bs_profile_read(const char* kernel, double* total_ms, int* launches);
int bs_profile_work(const char* kernel, double* work, double* exec);

#ifdef __cplusplus
}
#endif
#endif /* BSP_H */
