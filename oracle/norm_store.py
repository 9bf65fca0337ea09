"""RMSNorm feeding a Linear, with an FP8 store of the normalized output.

Test infrastructure (see ``oracle/__init__``).

Sec. 3.1 (Eq. norm-uses) and App. D.4: the forward computes z, u = gamma * z,
the store u_q and y = u_q W. The backward passes du = dy W^T through the
rounding unchanged (the straight-through reference, Sec. 1 and App. B.2) and
returns

  dW = u_W^T dy            (weight use: needs the rounded value u_q)
  dgamma = sum_tokens z_g * du   (gain use: needs the original z)

with z_g and u_W from Table "Store policies": U reads z / u, R reads
u_q / gamma / u_q, N reads a new rounding u_f / gamma / u_f. The normalization
input gradient uses unrounded values (App. D.4); the option ``norm_input='R'``
instead reads u_q / gamma there, as a memory-efficient normalization backward
that rebuilds z from the saved output does (App. E.4).

Readings where the paper is silent:
* the store is the FP8 store of ``oracle.qround`` (per-tensor amax scale) in
  place of the paper's per-token b-bit grid;
* the quantizer input u is computed in fp32 in a fixed order, so that every
  implementation produces the same bits: ss = sum_j fl(x_j * x_j) accumulated
  in 64 partials, partial l taking j = l, l + 64, ... in ascending order, then
  combined pairwise as p_l += p_{l+o} for o = 32, 16, ..., 1; ms = ss / d;
  r = 1 / sqrt(ms + eps); z = x * r; u = gamma * z; every step rounded to fp32,
  no fused multiply-add;
* the forward's own rounding uses trial 0 and use id ``store_id*256``; new
  roundings use trials 1..K and use ids ``store_id*256 + 1`` (gain use) and
  ``store_id*256 + 2`` (weight use), or one shared id ``+1`` for both uses;
  a new rounding is stochastic rounding at the forward's scale s.

Everything after u is fp64. Each policy's statistics come from K plain
backward passes (``oracle.stats``).

Parity: the reference gradients are pinned to torch.autograd of the
straight-through program in fp64; the biases to the closed forms of Eq.
norm-uses (U at the weight use adds -r^T dy, R at the gain use adds
sum (r/gamma) du, the other two are exactly zero); the N mean to an exact
enumeration of all rounding outcomes on tiny tensors
(tests/test_oracle_norm_store.py).
"""
import numpy as np

from . import policy, qround, fp8, philox
from .stats import trial_stats

LANES = 64


def rmsnorm_fp32(X, gamma, eps):
    """z, u and the inverse rms r_t, in the fixed fp32 order described above."""
    X = np.asarray(X, dtype=np.float32)
    g = np.asarray(gamma, dtype=np.float32)
    T, d = X.shape
    sq = (X * X).astype(np.float32)
    part = np.zeros((T, LANES), dtype=np.float32)
    for j in range(d):
        part[:, j % LANES] = (part[:, j % LANES] + sq[:, j]).astype(np.float32)
    off = LANES // 2
    while off >= 1:
        part[:, :off] = (part[:, :off] + part[:, off:2 * off]).astype(np.float32)
        off //= 2
    ss = part[:, 0]
    ms = (ss / np.float32(d)).astype(np.float32)
    rstd = (np.float32(1.0) / np.sqrt((ms + np.float32(eps)).astype(np.float32))).astype(np.float32)
    z = (X * rstd[:, None]).astype(np.float32)
    u = (g[None, :] * z).astype(np.float32)
    return z, u, rstd


def norm_backward(zhat, rstd, dz):
    """dx_t = r_t (dz_t - zhat_t * (sum_j dz_tj zhat_tj) / d), fp64."""
    zhat = np.asarray(zhat, dtype=np.float64)
    dz = np.asarray(dz, dtype=np.float64)
    d = zhat.shape[-1]
    dot = (dz * zhat).sum(axis=-1, keepdims=True)
    return np.asarray(rstd, dtype=np.float64)[..., None] * (dz - zhat * dot / d)


def use_ids(store_id, fresh_shared):
    base = store_id * 256
    return base, base + 1, (base + 1 if fresh_shared else base + 2)


def fresh_values(y_sel, elems, fmt, s, seed, trial, use):
    """deq of a new stochastic rounding of scaled values y_sel (fp32) at elements elems."""
    a = np.abs(np.asarray(y_sel, dtype=np.float32)).astype(np.float64)
    a = np.minimum(a, fmt.fmax)
    R = philox.words(seed, trial, use, elems)
    mag = fp8.sr_mag(a, fmt, R)
    return np.where(np.signbit(y_sel), -mag, mag) * np.float64(s)


def check(X, gamma, W, dY, *, eps=1e-5, fmt=fp8.E4M3, fwd_mode=qround.RNE,
          policies=("U/U", "R/R", "N/N"), K=16, seed=0, store_id=0, fresh_shared=False,
          norm_input="U", dw_rows=None, gain_cols=None, dx_rows=None, need_dx=True):
    """Reference gradients and each policy's trial statistics.

    norm_input is 'U' (the paper's default) or 'R'.

    dw_rows / gain_cols / dx_rows select the entries of dW (rows i), dgamma
    (entries j) and dX (rows t) to compute; None means all.
    """
    X = np.asarray(X, dtype=np.float32)
    T, d = X.shape
    g64 = np.asarray(gamma, dtype=np.float32).astype(np.float64)
    W64 = np.asarray(W, dtype=np.float32).astype(np.float64)
    dY64 = np.asarray(dY, dtype=np.float32).astype(np.float64)
    rows = np.arange(d) if dw_rows is None else np.asarray(dw_rows)
    cols = np.arange(d) if gain_cols is None else np.asarray(gain_cols)
    xrows = np.arange(T) if dx_rows is None else np.asarray(dx_rows)

    z, u, rstd = rmsnorm_fp32(X, gamma, eps)
    base, use_g, use_w = use_ids(store_id, fresh_shared)
    q = qround.qround(u, fmt, fwd_mode, seed, 0, base)
    s = q.scale
    uq = qround.dequant(q.codes, s, fmt)
    y = qround.scaled(u, s)
    z64, u64 = z.astype(np.float64), u.astype(np.float64)

    du = dY64 @ W64.T
    out = {"codes": q.codes, "scale": s, "n_saturated": q.n_saturated, "z": z, "u": u,
           "rstd": rstd, "du": du, "rows": rows, "cols": cols, "xrows": xrows}
    out["Y"] = uq @ W64
    out["dW_ref"] = uq[:, rows].T @ dY64
    out["dgamma_ref"] = (z64[:, cols] * du[:, cols]).sum(axis=0)
    if need_dx:
        out["dX_ref"] = norm_backward(z64[xrows], rstd[xrows], (g64 * du)[xrows])

    tidx = np.arange(T)[:, None]
    el_g = (tidx * d + cols[None, :]).astype(np.uint64)
    el_w = (tidx * d + rows[None, :]).astype(np.uint64)

    for code in policies:
        lg, lw = policy.parse(code)
        draws = lg == "N" or lw == "N"
        ntr = K if draws else 1
        dg_tr, dw_tr, dx_tr = [], [], []
        for k in range(1, ntr + 1):
            fg = fresh_values(y[:, cols], el_g, fmt, s, seed, k, use_g) if lg == "N" else None
            fw = fresh_values(y[:, rows], el_w, fmt, s, seed, k, use_w) if lw == "N" else None
            zg = policy.read(lg, z64[:, cols], uq[:, cols] / g64[cols], None if fg is None else fg / g64[cols])
            uW = policy.read(lw, u64[:, rows], uq[:, rows], fw)
            dg_tr.append((zg * du[:, cols]).sum(axis=0))
            dw_tr.append(uW.T @ dY64)
            if need_dx:
                zx = z64[xrows] if norm_input == "U" else uq[xrows] / g64
                dx_tr.append(norm_backward(zx, rstd[xrows], (g64 * du)[xrows]))
        reps = K if ntr == 1 else 1
        res = {}
        for name, tr, ref in (("dgamma", dg_tr, out["dgamma_ref"]), ("dW", dw_tr, out["dW_ref"]),
                              ("dX", dx_tr, out.get("dX_ref"))):
            if not tr:
                continue
            arr = np.stack(tr * reps) if reps > 1 else np.stack(tr)
            res[name] = trial_stats(arr, ref)
        out[code] = res
    return out
