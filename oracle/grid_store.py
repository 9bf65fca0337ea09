"""The paper's own normalization store: a per-token b-bit uniform grid (App. D.4).

Test infrastructure (see ``oracle/__init__``).

RMSNorm feeds a Linear as in ``oracle.norm_store`` (z, u = gamma * z in its fixed fp32 order,
y = u_q W, du = dy W^T passed through the rounding), but the store is the paper's: for each
token t the grid step is s_t = max_j |u_tj| / (2^(b-1) - 1) and u_q = s_t floor(u / s_t + xi)
with independent uniform xi per entry, so that u_q averages to u with no clipping. The new
rounding u_f = u + r_f is drawn from a separate stream and is read by both uses (all policies
at one seed share it). The uses return dW = u_W^T dy and dgamma = sum_tokens z_g * du with
(Table "Store policies", gain use first):

    U/R (reference)  z            u_q          R/N   u_q/gamma   u_f
    U/U              z            u            N/R   u_f/gamma   u_q
    U/N              z            u_f          N/N   u_f/gamma   u_f
    R/R              u_q/gamma    u_q          U/R+e z           u_q + (u_f - u)

The normalization input gradient uses unrounded values (the reference dX).

Readings where the paper is silent:
* fp32 as the paper's store: s_t = fl32(max_j |u_tj| / (2^(b-1) - 1)) (s_t = 1 for an all-zero
  row), y = fl32(u / s_t) (IEEE division), |y| clamped to 2^(b-1) - 1 (and counted: fl32 can
  exceed it by an ulp), u_q = fl32(q s_t) with the integer code q in [-(2^(b-1) - 1), 2^(b-1) - 1];
* stochastic rounding acts on |y| and keeps the sign (the same law as floor(y + xi) on the
  signed value): with lo = floor(|y|) and F = floor((|y| - lo) 2^32), the code rounds up iff
  R + F >= 2^32 for the element's 32-bit Philox word R, so P(up) = F / 2^32, the exact fraction
  whenever it has at most 32 bits;
* the forward's rounding uses trial 0 and use id store_id*256; the new rounding trials 1..K
  and use id store_id*256 + 1; the element index of u[t, j] is t d + j.

Everything after the store is fp64; each policy's statistics come from K plain passes.

Parity: the codec's up-probability is pinned exactly (rationals) to the fraction; the means over
the new rounding are pinned by exact enumeration of every outcome on small tensors against the
closed forms (N at the weight use has U/U's mean, U/R+e the reference's, N at the gain use the
original's up to fl32(gamma z) - gamma z, R at the gain use its residual sum); the reference
gradients to torch.autograd of the straight-through program (tests/test_oracle_grid_store.py).
"""
import numpy as np

from . import philox
from .norm_store import norm_backward, rmsnorm_fp32
from .stats import trial_stats

POLICIES = ("U/R", "U/U", "U/N", "R/R", "R/N", "N/R", "N/N", "U/R+e")


def parse(code):
    g, w = code.split("/")
    assert g in ("U", "R", "N") and w in ("U", "R", "N", "R+e"), code
    return g, w


def step_of(u, bits):
    """Per-token grid step s_t (fp32), 1 for an all-zero row."""
    u = np.asarray(u, dtype=np.float32)
    M = np.float32(2 ** (bits - 1) - 1)
    amax = np.max(np.abs(u), axis=-1)
    s = (amax / M).astype(np.float32)
    return np.where(amax > 0, s, np.float32(1.0)).astype(np.float32)


def bracket(u, s, bits):
    """|y| clamped, its floor lo, the threshold F = floor(frac 2^32), the sign and the clamp count."""
    y = (np.asarray(u, dtype=np.float32) / np.asarray(s, dtype=np.float32)[..., None]).astype(np.float32)
    M = np.float32(2 ** (bits - 1) - 1)
    a = np.abs(y)
    nsat = int((a > M).sum())
    a = np.minimum(a, M).astype(np.float64)
    lo = np.floor(a)
    F = np.floor((a - lo) * 2.0 ** 32).astype(np.uint64)
    return lo, F, np.signbit(y), nsat


def rounded(lo, F, neg, R):
    """The integer code of a stochastic rounding with words R."""
    up = (np.asarray(R, dtype=np.uint64) + F) >= np.uint64(1 << 32)
    mag = lo + up
    return np.where(neg, -mag, mag)


def value(q, s):
    """u = fl32(q s_t)."""
    return (np.asarray(q, dtype=np.float32) * np.asarray(s, dtype=np.float32)[..., None]).astype(np.float32)


def store(u, bits, seed, trial, use, cols=None):
    """(codes q, steps s, values fl32(q s), clamp count) of one stochastic rounding of u (of its
    columns ``cols`` only, if given; the steps always come from whole rows)."""
    s = step_of(u, bits)
    T, d = np.asarray(u).shape
    cols = np.arange(d) if cols is None else np.asarray(cols)
    lo, F, neg, nsat = bracket(np.asarray(u)[:, cols], s, bits)
    elem = (np.arange(T, dtype=np.uint64)[:, None] * np.uint64(d) + cols.astype(np.uint64)[None, :])
    q = rounded(lo, F, neg, philox.words(seed, trial, use, elem))
    return q.astype(np.int32), s, value(q, s), nsat


def policy_grads(code, z, u, uq, uf, gamma, du, dY):
    """One pass's (dgamma, dW) under a policy, all fp64 (uf may be None if the policy draws none)."""
    lg, lw = parse(code)
    z, u, uq, g, du, dY = (np.asarray(a, dtype=np.float64) for a in (z, u, uq, gamma, du, dY))
    uf = None if uf is None else np.asarray(uf, dtype=np.float64)
    zg = {"U": z, "R": uq / g if lg == "R" else None, "N": uf / g if lg == "N" else None}[lg]
    uW = {"U": u, "R": uq, "N": uf, "R+e": (uq + (uf - u)) if lw == "R+e" else None}[lw]
    return (zg * du).sum(axis=0), uW.T @ dY


def draws(code):
    lg, lw = parse(code)
    return lg == "N" or lw in ("N", "R+e")


def check(X, gamma, W, dY, *, bits=6, eps=1e-5, policies=POLICIES, K=16, seed=0, store_id=0, dw_rows=None,
          dw_cols=None, gain_cols=None, full=True):
    """Reference gradients and each policy's trial statistics (mean, bias, se) of dgamma, dW.

    dw_rows / dw_cols select the entries of dW (rows i, columns j) and gain_cols those of dgamma
    to compute; None means all (the store is always of the whole tensor). full=False skips Y and
    dX_ref and forms du only on the selected columns."""
    X = np.asarray(X, dtype=np.float32)
    g64 = np.asarray(gamma, dtype=np.float32).astype(np.float64)
    W64 = np.asarray(W, dtype=np.float32).astype(np.float64)
    dY64 = np.asarray(dY, dtype=np.float32).astype(np.float64)
    z, u, rstd = rmsnorm_fp32(X, gamma, eps)
    base = store_id * 256
    q, s, uq, nsat = store(u, bits, seed, 0, base)
    uq64 = uq.astype(np.float64)
    T, d = u.shape
    rows = np.arange(d) if dw_rows is None else np.asarray(dw_rows)
    cols = np.arange(dY64.shape[1]) if dw_cols is None else np.asarray(dw_cols)
    gcols = np.arange(d) if gain_cols is None else np.asarray(gain_cols)
    if full:
        du = dY64 @ W64.T
    else:                                   # du on the selected columns only
        du = np.zeros((T, d))
        sel = np.union1d(rows, gcols)
        du[:, sel] = dY64 @ W64[sel].T
    out = {"codes": q, "step": s, "uq": uq, "n_saturated": nsat, "u": u, "z": z, "du": du,
           "dW_ref": uq64[:, rows].T @ dY64[:, cols],
           "dgamma_ref": (z.astype(np.float64)[:, gcols] * du[:, gcols]).sum(axis=0)}
    if full:
        out["Y"] = uq64 @ W64
        out["dX_ref"] = norm_backward(z, rstd, g64 * du)
    need = np.union1d(rows, gcols)
    at = {int(j): i for i, j in enumerate(need)}
    ir, ig = [at[int(j)] for j in rows], [at[int(j)] for j in gcols]
    fresh = ([store(u, bits, seed, k, base + 1, cols=need)[2] for k in range(1, K + 1)]
             if any(draws(c) for c in policies) else [])
    for code in policies:
        ntr = K if draws(code) else 1
        dg, dw = [], []
        for k in range(ntr):
            f = fresh[k] if draws(code) else None
            a, _ = policy_grads(code, z[:, gcols], u[:, gcols], uq[:, gcols], None if f is None else f[:, ig],
                                gamma[gcols], du[:, gcols], dY64[:, :1])
            _, b = policy_grads(code, z[:, rows], u[:, rows], uq[:, rows], None if f is None else f[:, ir],
                                gamma[rows], du[:, rows], dY64[:, cols])
            dg.append(a)
            dw.append(b)
        reps = 1 if draws(code) else K
        out[code] = {"dgamma": trial_stats(np.stack(dg * reps), out["dgamma_ref"]),
                     "dW": trial_stats(np.stack(dw * reps), out["dW_ref"])}
    return out
