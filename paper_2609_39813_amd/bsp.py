"""Python binding of libbsp.so (the C-ABI in include/bsp.h).

Argument marshalling only: every step of every call runs in the library's HIP kernels.
Tensors must be CUDA (HIP) tensors; outputs are allocated with torch and the work is
enqueued on torch's current stream. There is no CPU fallback: if the library is not
built, importing this module raises.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbsp.so")
if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_39813_amd.build`")
_lib = ctypes.CDLL(LIB_PATH)

F32, BF16 = 0, 1
E4M3, E5M2 = 0, 1
RNE, SR = 0, 1
READ = {"U": 0, "R": 1, "N": 2}
_FMT = {"e4m3": E4M3, "e5m2": E5M2, E4M3: E4M3, E5M2: E5M2}
_MODE = {"rne": RNE, "sr": SR, RNE: RNE, SR: SR}

_vp, _i64, _u64, _u32, _int, _f32, _sz = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_uint32,
                                         ctypes.c_int, ctypes.c_float, ctypes.c_size_t)


class Diag(ctypes.Structure):
    _fields_ = [("nonfinite", ctypes.c_uint32), ("n_saturated", ctypes.c_uint32), ("amax", ctypes.c_float),
                ("scale", ctypes.c_float)]


class Est(ctypes.Structure):
    _fields_ = [("mean", _vp), ("bias", _vp), ("se", _vp)]


class NormPolicy(ctypes.Structure):
    _fields_ = [("gain_use", _int), ("weight_use", _int), ("norm_input_use", _int), ("fresh_shared", _int)]


def _sig(name, res, args):
    f = getattr(_lib, name)
    f.restype = res
    f.argtypes = args
    return f


_status_string = _sig("bs_status_string", ctypes.c_char_p, [_int])
bs_version = _sig("bs_version", _int, [])
_qround = _sig("bs_qround", _int, [_vp, _int, _i64, _int, _int, _u64, _u32, _u32, _vp, _vp, _vp, _vp, _vp])
_gemm = _sig("bs_gemm_bf16_nt", _int, [_vp, _i64, _vp, _i64, _vp, _i64, _i64, _i64, _i64, _f32, _int, _vp])
_pb_ws = _sig("bs_policy_bias_workspace_size", _sz, [_int, _i64])
_pb = _sig("bs_policy_bias_estimate", _int, [_vp, _int, _i64, _vp, _vp, _vp, _vp, _vp, _sz, _vp])
_sum_ws = _sig("bs_estimate_summary_workspace_size", _sz, [])
_sum = _sig("bs_estimate_summary", _int, [_vp, _vp, _vp, _i64, _vp, _vp, _sz, _vp])
_pb_na_max = _sig("bs_policy_bias_noalloc_max", _i64, [])
_pb_na = _sig("bs_policy_bias_estimate_noalloc", _int, [_vp, _int, _i64, _vp, _vp, _vp, _vp, _vp])
_norm_ws = _sig("bs_rmsnorm_linear_workspace_size", _sz, [_i64, _i64, _i64, _int, _int])
_norm = _sig("bs_rmsnorm_linear_fwd_bwd", _int,
             [_vp, _vp, _vp, _vp, _int, _i64, _i64, _i64, _f32, _int, _int, ctypes.POINTER(NormPolicy), _int, _int,
              _u64, _u32, _vp, _vp, _vp, _vp, _vp, _vp, Est, Est, Est, _vp, _vp, _sz, _vp])
_attn_ws = _sig("bs_attn_workspace_size", _sz, [_int, _int, _int, _int, _int, _int, _int])
_attn = _sig("bs_attn_bwd_policy", _int,
             [_vp, _vp, _vp, _vp, _int, _int, _int, _int, _int, _int, _f32, _vp, _int, _int, ctypes.POINTER(_int), _int,
              _int, _u64, _u32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, Est, Est, _vp, _vp, _sz, _vp])


class PstorePolicy(ctypes.Structure):
    _fields_ = [("softmax_read", _int), ("v_read", _int)]


SOFTMAX_READ = {"U": 0, "R": 1, "N": 2, "K": 3, "J2": 4, "Q2": 5}
_ps_ws = _sig("bs_attn_pstore_workspace_size", _sz, [_int] * 6)
_ps = _sig("bs_attn_pstore_policy", _int,
           [_vp, _vp, _vp, _vp, _int, _int, _int, _int, _int, _f32, _int, _int, ctypes.POINTER(PstorePolicy), _int,
            _int, _u64, _u32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, Est, Est, Est, _vp, _vp, _sz, _vp])
_attn2 = _sig("bs_attn_level2_policy", _int,
              [_vp, _vp, _vp, _vp, _int, _int, _int, _int, _int, _f32, _vp, _int, _int, _f32, ctypes.POINTER(_int), _int,
               _int, _u64, _u32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, Est, Est, _vp, _vp, _vp, _vp, _sz, _vp])
D_SOURCE = {"P": 0, "U": 1, "R": 2, "N": 3, "repair": 4}
_te_ws = _sig("bs_te_attn_workspace_size", _sz, [_int] * 7)
_te = _sig("bs_te_attn_bwd", _int,
           [_vp, _vp, _vp, _vp, _vp, _int, _int, _int, _int, _int, _f32, _vp, _vp, _vp, _int, _f32, _vp, _u64, _u32,
            _u32, _int, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp])
_te_sc = _sig("bs_te_delayed_scales", _int, [_vp, _vp, _int, _i64, _vp, _vp])
_lsm_ws = _sig("bs_logsoftmax_check_workspace_size", _sz, [_i64, _int, _int])
_lsm = _sig("bs_logsoftmax_reuse_check", _int,
            [_vp, _vp, _i64, _int, ctypes.c_double, _int, _u64, _u32, _int, _vp, _vp, _sz, _vp])


class GridPolicy(ctypes.Structure):
    _fields_ = [("gain_use", _int), ("weight_use", _int)]


WEIGHT_READ = {"U": 0, "R": 1, "N": 2, "R+e": 3}
GRID_POLICIES = ("U/R", "U/U", "U/N", "R/R", "R/N", "N/R", "N/N", "U/R+e")
_grid_ws = _sig("bs_rmsnorm_linear_grid_workspace_size", _sz, [_i64, _i64, _i64])
_grid = _sig("bs_rmsnorm_linear_grid_fwd_bwd", _int,
             [_vp, _vp, _vp, _vp, _int, _i64, _i64, _i64, _f32, _int, ctypes.POINTER(GridPolicy), _int, _int, _u64,
              _u32, _vp, _vp, _vp, _vp, _vp, _vp, Est, Est, _vp, _vp, _sz, _vp])
_lin_ws = _sig("bs_linear_bwd_workspace_size", _sz, [_i64, _i64, _i64, _int, _int, _int])
_lin = _sig("bs_linear_bwd_policy", _int,
            [_vp, _vp, _vp, _int, _i64, _i64, _i64, _int, ctypes.POINTER(_int), _int, _int, _u64, _u32, _vp, _vp,
             Est, Est, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp])


class LayerWeights(ctypes.Structure):
    _fields_ = [(k, _vp) for k in ("gain1", "Wqkv", "Wo", "gain2", "Wg", "Wu", "Wd")]


class LayerForward(ctypes.Structure):
    _fields_ = [(k, _vp) for k in ("Q", "K", "V", "O", "h", "gh", "a")]


class LayerGrads(ctypes.Structure):
    _fields_ = [(k, _vp) for k in ("dx", "dgain1", "dWqkv", "dWo", "dgain2", "dWg", "dWu", "dWd")]


class LayerStores(ctypes.Structure):
    _fields_ = [(k, _vp) for k in ("u1", "O", "u2", "a", "scales")]


class LayerAll(ctypes.Structure):
    _fields_ = [("bias", LayerGrads * 3), ("se", LayerGrads * 3), ("table", _vp)]


_layer_ws = _sig("bs_decoder_layer_workspace_size", _sz, [_int] * 7)
_layer = _sig("bs_decoder_layer_policy", _int,
              [_vp, ctypes.POINTER(LayerWeights), _vp, _int, _int, _int, _int, _int, _f32, _int, _int, _int, _u64,
               ctypes.POINTER(LayerForward), LayerGrads, LayerStores, _vp, ctypes.POINTER(LayerAll), _int, _vp, _vp,
               _sz, _vp])

_prof_enable = _sig("bs_profile_enable", _int, [_int])
_prof_read = _sig("bs_profile_read", _int, [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_int)])
_prof_work = _sig("bs_profile_work", _int, [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                            ctypes.POINTER(ctypes.c_double)])


def profile_enable(on=True):
    _check(_prof_enable(int(on)), "bs_profile_enable")


def profile_read(kernel=None):
    """(total ms, launches) of the instrumented kernel since profile_enable."""
    ms, n = ctypes.c_double(), _int()
    _check(_prof_read(None if kernel is None else kernel.encode(), ctypes.byref(ms), ctypes.byref(n)),
           "bs_profile_read")
    return ms.value, n.value


def profile_work(kernel=None):
    """(algorithmic, executed) work (flop for "gemm") of the instrumented launches since profile_enable."""
    w, x = ctypes.c_double(), ctypes.c_double()
    _check(_prof_work(None if kernel is None else kernel.encode(), ctypes.byref(w), ctypes.byref(x)),
           "bs_profile_work")
    return w.value, x.value


EXPORTED = ["bs_status_string", "bs_version", "bs_qround", "bs_gemm_bf16_nt", "bs_policy_bias_workspace_size",
            "bs_policy_bias_estimate", "bs_policy_bias_noalloc_max", "bs_policy_bias_estimate_noalloc",
            "bs_estimate_summary_workspace_size", "bs_estimate_summary",
            "bs_rmsnorm_linear_workspace_size", "bs_rmsnorm_linear_fwd_bwd",
            "bs_attn_workspace_size", "bs_attn_bwd_policy", "bs_attn_pstore_workspace_size", "bs_attn_pstore_policy", "bs_attn_level2_policy",
            "bs_te_attn_workspace_size", "bs_te_attn_bwd", "bs_te_delayed_scales",
            "bs_logsoftmax_check_workspace_size", "bs_logsoftmax_reuse_check",
            "bs_rmsnorm_linear_grid_workspace_size", "bs_rmsnorm_linear_grid_fwd_bwd", "bs_linear_bwd_workspace_size", "bs_linear_bwd_policy",
            "bs_decoder_layer_workspace_size", "bs_decoder_layer_policy", "bs_profile_enable", "bs_profile_read",
            "bs_profile_work"]


class BspError(RuntimeError):
    def __init__(self, code, call):
        super().__init__(f"{call}: {_status_string(code).decode()} (status {code})")
        self.code = code


def _check(code, call):
    if code != 0:
        raise BspError(code, call)


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dev_check(*ts):
    for t in ts:
        if t is not None:
            if not t.is_cuda:
                raise ValueError("libbsp works on device tensors only")
            if not t.is_contiguous():
                raise ValueError("tensors must be contiguous")


def _dt(t):
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"dtype {t.dtype} not supported")


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _workspace(nbytes, device):
    # 256-byte aligned by torch's caching allocator
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def diag_dict(d):
    """Decode a device bs_diag (a 16-byte uint8 tensor) after a stream sync."""
    raw = d.cpu().numpy().tobytes()
    v = Diag.from_buffer_copy(raw)
    return {"nonfinite": v.nonfinite, "n_saturated": v.n_saturated, "amax": v.amax, "scale": v.scale}


def new_diag(device):
    return torch.zeros(16, dtype=torch.uint8, device=device)


# ----------------------------------------------------------------------------------
def qround(x, fmt="e4m3", mode="rne", seed=0, trial=0, use=0, scale=None):
    """FP8 store of x: returns (codes uint8, scale [1] fp32, diag tensor)."""
    _dev_check(x, scale)
    codes = torch.empty(x.shape, dtype=torch.uint8, device=x.device)
    s = torch.empty(1, dtype=torch.float32, device=x.device)
    dg = new_diag(x.device)
    _check(_qround(_p(x), _dt(x), x.numel(), _FMT[fmt], _MODE[mode], seed, trial, use, _p(scale), _p(codes), _p(s),
                   _p(dg), _stream()), "bs_qround")
    return codes, s, dg


def gemm_bf16_nt(A, B, alpha=1.0, out=None, accumulate=False):
    """C = alpha * A B^T for bf16 A [M, K], B [N, K] (K-contiguous), C fp32."""
    _dev_check(A, B)
    M, K = A.shape
    N = B.shape[0]
    C = out if out is not None else torch.empty(M, N, dtype=torch.float32, device=A.device)
    _check(_gemm(_p(A), K, _p(B), K, _p(C), N, M, N, K, alpha, int(accumulate), _stream()), "bs_gemm_bf16_nt")
    return C


def policy_bias_estimate(delta, g_ref=None):
    """Trial statistics of per-trial errors delta [K, m]: (mean_err, se, summary[3])."""
    _dev_check(delta, g_ref)
    if delta.dim() != 2 or delta.dtype != torch.float32:
        raise TypeError("delta must be a [K, m] float32 tensor")
    K, m = delta.shape
    if g_ref is not None and (g_ref.dtype != torch.float32 or g_ref.numel() != m):
        raise TypeError("g_ref must be a float32 tensor of m elements")
    mean = torch.empty(m, dtype=torch.float32, device=delta.device)
    se = torch.empty(m, dtype=torch.float32, device=delta.device)
    summ = torch.empty(3, dtype=torch.float64, device=delta.device)
    ws = _workspace(_pb_ws(K, m), delta.device)
    _check(_pb(_p(delta), K, m, _p(g_ref), _p(mean), _p(se), _p(summ), _p(ws), ws.numel(), _stream()),
           "bs_policy_bias_estimate")
    return mean, se, summ


def policy_bias_estimate_noalloc(delta, g_ref=None, out=None):
    """bs_policy_bias_estimate_noalloc: the same statistics with the library's own device scratch
    (no workspace; m <= policy_bias_noalloc_max()). out: optional (mean_err, se, summary) tensors
    to write into."""
    _dev_check(delta, g_ref)
    if delta.dim() != 2 or delta.dtype != torch.float32:
        raise TypeError("delta must be a [K, m] float32 tensor")
    K, m = delta.shape
    if g_ref is not None and (g_ref.dtype != torch.float32 or g_ref.numel() != m):
        raise TypeError("g_ref must be a float32 tensor of m elements")
    if out is None:
        out = (torch.empty(m, dtype=torch.float32, device=delta.device),
               torch.empty(m, dtype=torch.float32, device=delta.device),
               torch.empty(3, dtype=torch.float64, device=delta.device))
    mean, se, summ = out
    _check(_pb_na(_p(delta), K, m, _p(g_ref), _p(mean), _p(se), _p(summ), _stream()),
           "bs_policy_bias_estimate_noalloc")
    return mean, se, summ


def estimate_summary(bias, se=None, ref=None):
    """(||bias||, ||ref||, R = ||bias||^2 / sum se^2) of one gradient's estimate (bs_estimate_summary);
    fp32 device tensors of equal size, se / ref optional."""
    _dev_check(bias, se, ref)
    n = bias.numel()
    for t in (bias, se, ref):
        if t is not None and (t.dtype != torch.float32 or t.numel() != n):
            raise TypeError("bias, se and ref must be float32 tensors of one size")
    summ = torch.empty(3, dtype=torch.float64, device=bias.device)
    ws = _workspace(_sum_ws(), bias.device)
    _check(_sum(_p(bias), _p(se), _p(ref), n, _p(summ), _p(ws), ws.numel(), _stream()), "bs_estimate_summary")
    return summ


def policy_bias_noalloc_max():
    return int(_pb_na_max())


def _est(n_pol, numel, device, want_se):
    mean = torch.empty(n_pol, numel, dtype=torch.float32, device=device)
    bias = torch.empty(n_pol, numel, dtype=torch.float32, device=device)
    se = torch.empty(n_pol, numel, dtype=torch.float32, device=device) if want_se else None
    return {"mean": mean, "bias": bias, "se": se}, Est(_p(mean), _p(bias), _p(se))


def parse_norm_policy(code):
    """'G/W' letters, optional suffixes ':R' (norm-input reads R) and ':shared'."""
    parts = code.split(":")
    g, w = parts[0].split("/")
    return NormPolicy(READ[g], READ[w], READ["R"] if "R" in parts[1:] else READ["U"], 1 if "shared" in parts[1:] else 0)


def rmsnorm_linear(X, gain, W, dY, *, eps=1e-5, fmt="e4m3", fwd_mode="rne", policies=("U/U", "R/R", "N/N"), K=16,
                   seed=0, store_id=0, want_y=True, want_se=True, want_dw_se=False, ws=None):
    """RMSNorm -> FP8 store -> Linear and the per-use policy estimates (bs_rmsnorm_linear_fwd_bwd).
    want_dw_se: also the se of dW where the weight use reads a new rounding (K per-trial
    contractions; the other estimates collapse the trials)."""
    _dev_check(X, gain, W, dY)
    T, d = X.shape
    n = W.shape[1]
    dev = X.device
    pol = (NormPolicy * len(policies))(*[parse_norm_policy(p) for p in policies])
    out = {"u_codes": torch.empty(T, d, dtype=torch.uint8, device=dev),
           "u_scale": torch.empty(1, dtype=torch.float32, device=dev),
           "dgain_ref": torch.empty(d, dtype=torch.float32, device=dev),
           "dW_ref": torch.empty(d, n, dtype=torch.float32, device=dev),
           "dX_ref": torch.empty(T, d, dtype=torch.float32, device=dev),
           "Y": torch.empty(T, n, dtype=torch.float32, device=dev) if want_y else None,
           "diag": new_diag(dev)}
    weight_n = any(p.split(":")[0].split("/")[1] == "N" for p in policies)
    eg, cg = _est(len(policies), d, dev, want_se)
    ew, cw = _est(len(policies), d * n, dev, want_se and (want_dw_se or not weight_n))
    ex, cx = _est(len(policies), T * d, dev, want_se)
    if ws is None:
        ws = _workspace(_norm_ws(T, d, n, len(policies), K), dev)
    _check(_norm(_p(X), _p(gain), _p(W), _p(dY), _dt(X), T, d, n, eps, _FMT[fmt], _MODE[fwd_mode], pol, len(policies), K,
                 seed, store_id, _p(out["Y"]), _p(out["u_codes"]), _p(out["u_scale"]), _p(out["dgain_ref"]),
                 _p(out["dW_ref"]), _p(out["dX_ref"]), cg, cw, cx, _p(out["diag"]), _p(ws), ws.numel(), _stream()),
           "bs_rmsnorm_linear_fwd_bwd")
    out["dgain"], out["dW"], out["dX"] = eg, ew, ex
    out["policies"] = list(policies)
    return out


def rmsnorm_linear_grid(X, gain, W, dY, *, bits=6, eps=1e-5, policies=GRID_POLICIES, K=16, seed=0, store_id=0,
                        want_y=True, ws=None):
    """RMSNorm -> per-token b-bit grid store -> Linear, and the policies of the paper's table
    (bs_rmsnorm_linear_grid_fwd_bwd). Policy codes name the gain use first; 'U/R+e' reads
    u_q + (u_f - u) at the weight use."""
    _dev_check(X, gain, W, dY)
    T, d = X.shape
    n = W.shape[1]
    dev = X.device
    pol = (GridPolicy * len(policies))(*[GridPolicy(READ[c.split("/")[0]], WEIGHT_READ[c.split("/")[1]])
                                          for c in policies])
    out = {"u_codes": torch.empty(T, d, dtype=torch.int8, device=dev),
           "u_step": torch.empty(T, dtype=torch.float32, device=dev),
           "dgain_ref": torch.empty(d, dtype=torch.float32, device=dev),
           "dW_ref": torch.empty(d, n, dtype=torch.float32, device=dev),
           "dX_ref": torch.empty(T, d, dtype=torch.float32, device=dev),
           "Y": torch.empty(T, n, dtype=torch.float32, device=dev) if want_y else None,
           "diag": new_diag(dev)}
    eg, cg = _est(len(policies), d, dev, False)
    ew, cw = _est(len(policies), d * n, dev, False)
    if ws is None:
        ws = _workspace(_grid_ws(T, d, n), dev)
    _check(_grid(_p(X), _p(gain), _p(W), _p(dY), _dt(X), T, d, n, eps, bits, pol, len(policies), K, seed, store_id,
                 _p(out["Y"]), _p(out["u_codes"]), _p(out["u_step"]), _p(out["dgain_ref"]), _p(out["dW_ref"]),
                 _p(out["dX_ref"]), cg, cw, _p(out["diag"]), _p(ws), ws.numel(), _stream()),
           "bs_rmsnorm_linear_grid_fwd_bwd")
    out["dgain"], out["dW"] = eg, ew
    out["policies"] = list(policies)
    return out


def rmsnorm_linear_workspace(T, d, n, n_pol, K, device):
    return _workspace(_norm_ws(T, d, n, n_pol, K), device)


def attn_bwd_policy(Q, Kt, V, dO, *, causal=True, scale=None, O=None, fmt="e4m3", fwd_mode="sr",
                    policies=("U", "R", "N"), K=32, seed=0, store_id=0, want_o=True, want_se=True, want_dk_se=False,
                    ws=None):
    """Attention backward with D read from each policy's copy of O (bs_attn_bwd_policy).
    want_dk_se: also dK's se (the per-trial path: one key-major pass per trial under N)."""
    _dev_check(Q, Kt, V, dO, O)
    B, H, S, dh = Q.shape
    dev = Q.device
    c = 1.0 / dh ** 0.5 if scale is None else scale
    pol = (_int * len(policies))(*[READ[p] for p in policies])
    shp = (B, H, S, dh)
    out = {"O": torch.empty(shp, dtype=torch.float32, device=dev) if want_o else None,
           "O_codes": torch.empty(shp, dtype=torch.uint8, device=dev),
           "O_scale": torch.empty(1, dtype=torch.float32, device=dev),
           "dQ_ref": torch.empty(shp, dtype=torch.float32, device=dev),
           "dK_ref": torch.empty(shp, dtype=torch.float32, device=dev),
           "dV": torch.empty(shp, dtype=torch.float32, device=dev),
           "D_ref": torch.empty(B, H, S, dtype=torch.float32, device=dev),
           "diag": new_diag(dev)}
    numel = B * H * S * dh
    eq, cq = _est(len(policies), numel, dev, want_se)
    ek, ck = _est(len(policies), numel, dev, want_dk_se)
    if ws is None:
        ws = _workspace(_attn_ws(B, H, S, dh, len(policies), K, int(want_dk_se)), dev)
    _check(_attn(_p(Q), _p(Kt), _p(V), _p(dO), F32 if dO is not None and dO.dtype == torch.float32 else BF16,
                 B, H, S, dh, int(causal), c, _p(O), _FMT[fmt], _MODE[fwd_mode], pol,
                 len(policies), K, seed, store_id, _p(out["O"]), _p(out["O_codes"]), _p(out["O_scale"]),
                 _p(out["dQ_ref"]), _p(out["dK_ref"]), _p(out["dV"]), _p(out["D_ref"]), cq, ck, _p(out["diag"]),
                 _p(ws), ws.numel(), _stream()), "bs_attn_bwd_policy")
    out["dQ"], out["dK"] = eq, ek
    return out


def attn_level2_policy(Q, Kt, V, dO, *, causal=True, scale=None, O=None, fmt="e4m3", fwd_mode="sr", beta=1.0,
                       policies=("U", "R", "N"), K=32, seed=0, store_id=0, want_o=False, ws=None):
    """The D use averaged over the forward's rounding too, with incoming gradient dO + beta r_k
    (bs_attn_level2_policy)."""
    _dev_check(Q, Kt, V, dO, O)
    B, H, S, dh = Q.shape
    dev = Q.device
    c = 1.0 / dh ** 0.5 if scale is None else scale
    pol = (_int * len(policies))(*[READ[p] for p in policies])
    shp, rows = (B, H, S, dh), B * H * S
    out = {"O": torch.empty(shp, dtype=torch.float32, device=dev) if want_o else None,
           "O_scale": torch.empty(1, dtype=torch.float32, device=dev),
           "dO_mean": torch.empty(shp, dtype=torch.float32, device=dev),
           "dQ_ref": torch.empty(shp, dtype=torch.float32, device=dev),
           "dK_ref": torch.empty(shp, dtype=torch.float32, device=dev),
           "dV": torch.empty(shp, dtype=torch.float32, device=dev),
           "D_ref": torch.empty(B, H, S, dtype=torch.float32, device=dev),
           "d_use": torch.empty(len(policies), 4, rows, dtype=torch.float32, device=dev),
           "T": torch.empty(2, rows, dtype=torch.float32, device=dev),
           "diag": new_diag(dev)}
    numel = B * H * S * dh
    eq, cq = _est(len(policies), numel, dev, False)
    ek, ck = _est(len(policies), numel, dev, False)
    if ws is None:
        ws = _workspace(_attn_ws(B, H, S, dh, len(policies), K, 0), dev)
    _check(_attn2(_p(Q), _p(Kt), _p(V), _p(dO), B, H, S, dh, int(causal), c, _p(O), _FMT[fmt], _MODE[fwd_mode], beta,
                  pol, len(policies), K, seed, store_id, _p(out["O"]), _p(out["O_scale"]), _p(out["dO_mean"]),
                  _p(out["dQ_ref"]), _p(out["dK_ref"]), _p(out["dV"]), _p(out["D_ref"]), cq, ck, _p(out["d_use"]),
                  _p(out["T"]), _p(out["diag"]), _p(ws), ws.numel(), _stream()), "bs_attn_level2_policy")
    out["dQ"], out["dK"] = eq, ek
    return out


LSM_STATS = ("likelihood_reuse", "likelihood_independent", "constructed_reuse", "constructed_independent")


def logsoftmax_reuse_check(logits, target, *, eps=0.1, K=4096, seed=0, store_id=0, calibrate=False, ws=None):
    """The log-softmax operator test (bs_logsoftmax_reuse_check): {statistic: (mean, se)} over K trials."""
    _dev_check(logits, target)
    if logits.dtype != torch.float64 or target.dtype != torch.int32:
        raise ValueError("logits must be fp64 and target int32")
    rows, C = logits.shape
    stats = torch.empty(4, 2, dtype=torch.float64, device=logits.device)
    if ws is None:
        n = _lsm_ws(rows, C, K)
        if n == 0:
            raise BspError(2, "bs_logsoftmax_check_workspace_size")
        ws = _workspace(n, logits.device)
    _check(_lsm(_p(logits), _p(target), rows, C, eps, K, seed, store_id, int(calibrate), _p(stats), _p(ws), ws.numel(),
                _stream()), "bs_logsoftmax_reuse_check")
    return stats


def attn_workspace(B, H, S, dh, n_pol, K, device, want_dk_se=False):
    return _workspace(_attn_ws(B, H, S, dh, n_pol, K, int(want_dk_se)), device)


def parse_pstore_policy(code):
    """'J2/R' -> the softmax's backward read first, then the read at the gradient of V."""
    sm, v = code.split("/")
    return PstorePolicy(SOFTMAX_READ[sm], READ[v])


def attn_pstore_workspace(B, H, S, dh, K, causal, device):
    n = _ps_ws(B, H, S, dh, K, int(causal))
    if n == 0:
        raise BspError(2, "bs_attn_pstore_workspace_size")
    return _workspace(n, device)


def attn_pstore_policy(Q, Kt, V, dO, *, causal=True, scale=None, fmt="e4m3", fwd_mode="rne",
                       policies=("U/R", "R/R", "U/U", "N/N", "R/U", "K/R", "J2/R", "Q2/R"), K=16, seed=0, store_id=0,
                       want_p=False, ws=None):
    """Attention with an FP8 store of P and the per-policy estimates of its two uses
    (bs_attn_pstore_policy)."""
    _dev_check(Q, Kt, V, dO)
    B, H, S, dh = Q.shape
    dev = Q.device
    c = 1.0 / dh ** 0.5 if scale is None else scale
    pol = (PstorePolicy * len(policies))(*[parse_pstore_policy(p) for p in policies])
    shp = (B, H, S, dh)
    out = {"O": torch.empty(shp, dtype=torch.float32, device=dev),
           "P": torch.empty(B, H, S, S, dtype=torch.float32, device=dev) if want_p else None,
           "P_codes": torch.empty(B, H, S, S, dtype=torch.uint8, device=dev),
           "P_scale": torch.empty(1, dtype=torch.float32, device=dev),
           "dQ_ref": torch.empty(shp, dtype=torch.float32, device=dev),
           "dK_ref": torch.empty(shp, dtype=torch.float32, device=dev),
           "dV_ref": torch.empty(shp, dtype=torch.float32, device=dev),
           "diag": new_diag(dev)}
    numel = B * H * S * dh
    ests = [_est(len(policies), numel, dev, False) for _ in range(3)]
    if ws is None:
        ws = attn_pstore_workspace(B, H, S, dh, K, causal, dev)
    _check(_ps(_p(Q), _p(Kt), _p(V), _p(dO), B, H, S, dh, int(causal), c, _FMT[fmt], _MODE[fwd_mode], pol,
               len(policies), K, seed, store_id, _p(out["O"]), _p(out["P"]), _p(out["P_codes"]), _p(out["P_scale"]),
               _p(out["dQ_ref"]), _p(out["dK_ref"]), _p(out["dV_ref"]), ests[0][1], ests[1][1], ests[2][1],
               _p(out["diag"]), _p(ws), ws.numel(), _stream()), "bs_attn_pstore_policy")
    out["dQ"], out["dK"], out["dV"] = (e[0] for e in ests)
    out["policies"] = list(policies)
    return out


def te_attn_workspace(B, H, S, dh, causal, source, device, fp8_qkv=False):
    n = _te_ws(B, H, S, dh, int(causal), D_SOURCE[source], int(fp8_qkv))
    if n == 0:
        raise BspError(2, "bs_te_attn_workspace_size")
    return _workspace(n, device)


def te_attn_bwd(Q, Kt, V, dO, scales, *, qkv_scales=None, O=None, O_codes=None, O_scale=None, source="R",
                threshold=0.9, causal=True, scale=None, seed=0, store_id=0, trial=1, grad_dtype="bf16", want_p=False,
                want_ds=False, want_codes=False, want_pre=False, ws=None):
    """The emulated FP8 attention backward with delayed scales (bs_te_attn_bwd). scales: device
    fp32 [4] = (s_P, s_dO, s_dS, s_g). qkv_scales: None (Q, Kt, V bf16) or device fp32 [3] with
    Q, Kt, V the forward's E4M3 codes (uint8). grad_dtype: "bf16" or "f32" returned gradients."""
    _dev_check(Q, Kt, V, dO, scales, O, O_codes, O_scale, qkv_scales)
    want = torch.uint8 if qkv_scales is not None else torch.bfloat16
    if any(t.dtype != want for t in (Q, Kt, V)):
        raise TypeError(f"Q, K and V must be {want} {'(E4M3 codes)' if qkv_scales is not None else ''}")
    if qkv_scales is not None and (qkv_scales.dtype != torch.float32 or qkv_scales.numel() != 3):
        raise TypeError("qkv_scales must be a float32 tensor of 3 scales")
    gdt = {"bf16": torch.bfloat16, "f32": torch.float32}[grad_dtype]
    B, H, S, dh = Q.shape
    dev = Q.device
    c = 1.0 / dh ** 0.5 if scale is None else scale
    shp = (B, H, S, dh)
    sq = lambda dt, on: torch.zeros(B, H, S, S, dtype=dt, device=dev) if on else None
    out = {"dQ": torch.empty(shp, dtype=gdt, device=dev),
           "dK": torch.empty(shp, dtype=gdt, device=dev),
           "dV": torch.empty(shp, dtype=gdt, device=dev),
           "amax": torch.empty(4, dtype=torch.float32, device=dev),
           "counts": torch.empty(4, dtype=torch.int32, device=dev),
           "P": sq(torch.float32, want_p), "dS": sq(torch.float32, want_ds),
           "P_codes": sq(torch.uint8, want_codes), "dS_codes": sq(torch.uint8, want_codes),
           "pre": torch.empty((3,) + shp, dtype=torch.float32, device=dev) if want_pre else None}
    if ws is None:
        ws = te_attn_workspace(B, H, S, dh, causal, source, dev, qkv_scales is not None)
    _check(_te(_p(Q), _p(Kt), _p(V), _p(qkv_scales), _p(dO), B, H, S, dh, int(causal), c, _p(O), _p(O_codes),
               _p(O_scale), D_SOURCE[source], threshold, _p(scales), seed, store_id, trial,
               BF16 if grad_dtype == "bf16" else F32, _p(out["dQ"]), _p(out["dK"]),
               _p(out["dV"]), _p(out["amax"]), _p(out["counts"]), _p(out["P"]), _p(out["dS"]), _p(out["P_codes"]),
               _p(out["dS_codes"]), _p(out["pre"]), _p(ws), ws.numel(), _stream()), "bs_te_attn_bwd")
    return out


def te_delayed_scales(amax, history, step, scales):
    """One step of delayed scaling (bs_te_delayed_scales): history [4, len] and scales [4] are
    updated in place."""
    _dev_check(amax, history, scales)
    _check(_te_sc(_p(amax), _p(history), history.shape[1], step, _p(scales), _stream()), "bs_te_delayed_scales")
    return scales


def linear_bwd_policy(X, W, dY, *, fmt="e5m2", sharings=("shared", "per_use"), K=16, seed=0, store_id=0,
                      probeA=None, probeB=None, want_se=False, ws=None):
    """Linear backward with an FP8-rounded incoming gradient (bs_linear_bwd_policy). want_se: the
    se of dX and dW over trials (the per-trial path: K per-trial contractions per gradient)."""
    _dev_check(X, W, dY, probeA, probeB)
    M, k = X.shape
    n = W.shape[1]
    dev = X.device
    sh = (_int * len(sharings))(*[0 if s == "shared" else 1 for s in sharings])
    out = {"dX_ref": torch.empty(M, k, dtype=torch.float32, device=dev),
           "dW_ref": torch.empty(k, n, dtype=torch.float32, device=dev),
           "dY_scale": torch.empty(1, dtype=torch.float32, device=dev),
           "coupling": torch.empty(len(sharings), dtype=torch.float64, device=dev) if probeA is not None else None,
           "diag": new_diag(dev)}
    ex, cx = _est(len(sharings), M * k, dev, want_se)
    ew, cw = _est(len(sharings), k * n, dev, want_se)
    if ws is None:
        ws = _workspace(_lin_ws(M, k, n, len(sharings), K, int(want_se)), dev)
    _check(_lin(_p(X), _p(W), _p(dY), _dt(X), M, k, n, _FMT[fmt], sh, len(sharings), K, seed, store_id,
                _p(out["dX_ref"]), _p(out["dW_ref"]), cx, cw, _p(probeA), _p(probeB), _p(out["coupling"]),
                _p(out["dY_scale"]), _p(out["diag"]), _p(ws), ws.numel(), _stream()), "bs_linear_bwd_policy")
    out["dX"], out["dW"] = ex, ew
    return out


def linear_bwd_workspace(M, k, n, n_pol, K, device, want_se=False):
    return _workspace(_lin_ws(M, k, n, n_pol, K, int(want_se)), device)


LAYER_ROWS = (("u1", "gain", "dgain"), ("u1", "weight", "dW"), ("u1", "norm_input", "dX"), ("O", "D", "dQ"),
              ("O", "D", "dK"), ("O", "weight", "dW"), ("u2", "gain", "dgain"), ("u2", "weight", "dW"),
              ("u2", "norm_input", "dX"), ("a", "weight", "dW"))


LAYER_GRADS = ("dx", "dgain1", "dWqkv", "dWo", "dgain2", "dWg", "dWu", "dWd")


LAYER_ALL_USES, LAYER_PER_USE_SE = 1, 2


def decoder_layer_workspace(B, S, d, H, F, K, device, all_uses=False, per_use_se=False):
    n = _layer_ws(B, S, d, H, F, K, (LAYER_ALL_USES if all_uses else 0) | (LAYER_PER_USE_SE if per_use_se else 0))
    if n == 0:
        raise BspError(3, "bs_decoder_layer_workspace_size")
    return _workspace(n, device)


def decoder_layer_policy(x, p, dOut, *, B, S, H, eps=1e-5, fmt="e4m3", fwd_mode="rne", K=16, seed=0, fixed=None,
                         all_uses=False, all_outputs=True, per_use_se=False, ws=None):
    """One decoder layer with four FP8 stores and the per-use check of every store
    (bs_decoder_layer_policy). p: gain1, gain2 fp32 [d]; Wqkv, Wo, Wg, Wu, Wd bf16. fixed:
    None, or the realized forward {Q, K, V (bf16 [B,H,S,64]), O ([B,H,S,64]), h, gh ([T,2F]),
    a ([T,F]) fp32}. Returns the table as {(store, use, grad, letter): (bias^2, ref^2, se^2)}
    plus reference gradients, store codes and scales. all_uses: also each letter read at every use
    together ("all_bias" / "all_se": {letter: {gradient: tensor}}, only with all_outputs, and
    "all_table_raw" [8][3][3]). per_use_se: the table's se of the weight uses and of dK under N by
    per-trial paths (NaN without)."""
    T, d = x.shape
    F = p["Wg"].shape[1]
    dev = x.device
    ts = [x, dOut] + [p[k] for k in ("gain1", "Wqkv", "Wo", "gain2", "Wg", "Wu", "Wd")]
    if fixed is not None:
        ts += [fixed[k] for k in ("Q", "K", "V", "O", "h", "gh", "a")]
    _dev_check(*ts)
    wts = LayerWeights(*[p[k].data_ptr() for k in ("gain1", "Wqkv", "Wo", "gain2", "Wg", "Wu", "Wd")])
    fx = None
    if fixed is not None:
        fx = ctypes.byref(LayerForward(*[fixed[k].data_ptr() for k in ("Q", "K", "V", "O", "h", "gh", "a")]))
    e = lambda *shape: torch.empty(*shape, dtype=torch.float32, device=dev)
    out = {"dx": e(T, d), "dgain1": e(d), "dWqkv": e(d, 3 * d), "dWo": e(d, d), "dgain2": e(d), "dWg": e(d, F),
           "dWu": e(d, F), "dWd": e(F, d),
           "codes_u1": torch.empty(T, d, dtype=torch.uint8, device=dev),
           "codes_O": torch.empty(B, H, S, d // H, dtype=torch.uint8, device=dev),
           "codes_u2": torch.empty(T, d, dtype=torch.uint8, device=dev),
           "codes_a": torch.empty(T, F, dtype=torch.uint8, device=dev),
           "scales": e(4), "diags": torch.zeros(4, 16, dtype=torch.uint8, device=dev),
           "table_raw": torch.empty(len(LAYER_ROWS), 3, 3, dtype=torch.float64, device=dev)}
    grads = LayerGrads(*[out[k].data_ptr() for k in ("dx", "dgain1", "dWqkv", "dWo", "dgain2", "dWg", "dWu", "dWd")])
    stores = LayerStores(*[out[k].data_ptr() for k in ("codes_u1", "codes_O", "codes_u2", "codes_a", "scales")])
    allp = None
    if all_uses:
        shp = {"dx": (T, d), "dgain1": (d,), "dWqkv": (d, 3 * d), "dWo": (d, d), "dgain2": (d,), "dWg": (d, F),
               "dWu": (d, F), "dWd": (F, d)}
        out["all_table_raw"] = torch.empty(8, 3, 3, dtype=torch.float64, device=dev)
        al = LayerAll()
        al.table = out["all_table_raw"].data_ptr()
        if all_outputs:
            out["all_bias"] = {l: {g: e(*shp[g]) for g in LAYER_GRADS} for l in "URN"}
            out["all_se"] = {l: {g: e(*shp[g]) for g in LAYER_GRADS} for l in "URN"}
            for i, l in enumerate("URN"):
                al.bias[i] = LayerGrads(*[out["all_bias"][l][g].data_ptr() for g in LAYER_GRADS])
                al.se[i] = LayerGrads(*[out["all_se"][l][g].data_ptr() for g in LAYER_GRADS])
        allp = ctypes.byref(al)
    if ws is None:
        ws = decoder_layer_workspace(B, S, d, H, F, K, dev, all_uses, per_use_se)
    _check(_layer(_p(x), ctypes.byref(wts), _p(dOut), B, S, d, H, F, eps, _FMT[fmt], _MODE[fwd_mode], K, seed, fx,
                  grads, stores, _p(out["table_raw"]), allp, int(per_use_se), _p(out["diags"]), _p(ws), ws.numel(),
                  _stream()),
           "bs_decoder_layer_policy")
    return out


def layer_all_table(raw):
    """{(gradient, letter): (bias^2, ref^2, se^2)} from the [8][3][3] every-use table (host)."""
    raw = raw.cpu().numpy() if hasattr(raw, "cpu") else raw
    return {(g, l): tuple(float(v) for v in raw[r, i]) for r, g in enumerate(LAYER_GRADS) for i, l in enumerate("URN")}


def layer_table(raw):
    """{(store, use, grad, letter): (bias^2, ref^2, se^2)} from the [rows][3][3] table (host)."""
    raw = raw.cpu().numpy() if hasattr(raw, "cpu") else raw
    return {LAYER_ROWS[r] + (l,): tuple(float(v) for v in raw[r, i]) for r in range(len(LAYER_ROWS))
            for i, l in enumerate("URN")}
