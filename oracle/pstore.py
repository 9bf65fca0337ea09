"""The FP8 store of attention probabilities and its two uses.

Test infrastructure (see ``oracle/__init__``).

One row of attention (App. B.2): scores s, probabilities p = softmax(s), values V with rows
v_j. The forward rounds p to p_q = p + r and outputs o = V^T p_q. With h = dL/do the row's
incoming gradient and dp = V h, the reference (Eq. app-ref) computes

    dV = p_q h^T,        ds = J(p) dp,        J(x) = diag(x) - x x^T.

A policy reads a vector p_hat at the gradient of V and a matrix J_hat at the softmax's
backward (Eq. app-errors). Policy codes name the softmax's backward first (Table
"app-theory-errors"). The softmax's backward reads

    U  J(p)            R  J(p_q)           N  J(a)  (a a new rounding; App. B.3)
    K  K(a) = diag(a (1^T a)) - a a^T      (one new rounding; Eq. app-onecopy, App. B.4)
    J2 J2(a, b) = diag((a + b)/2) - (a b^T + b a^T)/2   (two new roundings; App. B.4)
    Q2 J2(p_q, a)      (the forward's own rounding as one of J2's two; App. B.4)

and the gradient of V reads U p, R p_q or N a. N/N reads the same new rounding a at both uses
(App. B.3: "a new rounding p_f ... read at both uses"). U/R is the reference.

The attention-level check (``check``) applies the row functions to every query row of a
(causal) softmax attention with a fixed incoming gradient dO (the forward held fixed):
dp = dO V^T per row, ds -> dQ = c ds K, dK = c ds^T Q, and dV = p_hat^T dO. The store is the
per-tensor FP8 codec of ``oracle.qround`` applied to P: amax = max P over the whole tensor,
s = fl32(amax / FMAX); the forward's rounding is RNE (TE's, Sec. 2.2) or SR with trial 0 and
use store_id*256; new roundings a and b are SR at the same scale with trials 1..K and uses
store_id*256 + 1 and + 2. The element index of P[b, h, i, j] is ((b H + h) S + i) S + j. The
forward output is O = p_q V. Everything except the store is fp64.

Parity: the row functions are pinned by exact enumeration (fractions) of every rounding
outcome in the paper's cells A and B under its two rounding laws, against the closed forms of
Table app-theory-errors, Eq. app-replay-error and App. B.4 (tests/test_oracle_pstore.py); the
attention-level reference is pinned to torch.autograd in fp64.
"""
import numpy as np

from . import fp8, philox, qround
from .stats import trial_stats

SOFTMAX_READS = ("U", "R", "N", "K", "J2", "Q2")
V_READS = ("U", "R", "N")


def parse(code):
    """'N/N' -> ('N', 'N'): softmax's backward first, then the gradient of V."""
    a, b = code.split("/")
    assert a in SOFTMAX_READS and b in V_READS, code
    return a, b


def draws(code):
    """New roundings a policy reads: 0 (none), 1 (a) or 2 (a and b)."""
    sm, v = parse(code)
    if sm == "J2":
        return 2
    return 1 if (sm in ("N", "K", "Q2") or v == "N") else 0


# -- the matrices of the softmax's backward applied to dp (rows on the last axis) --------

def _dot(x, y):
    return (x * y).sum(axis=-1, keepdims=True)


def J_apply(x, dp):
    """J(x) dp = x * dp - x (x . dp)."""
    return x * dp - x * _dot(x, dp)


def K_apply(a, dp):
    """K(a) dp = diag(a (1^T a)) dp - a (a . dp)."""
    return a * a.sum(axis=-1, keepdims=True) * dp - a * _dot(a, dp)


def J2_apply(a, b, dp):
    """J2(a, b) dp = (a + b)/2 * dp - (a (b . dp) + b (a . dp)) / 2."""
    return ((a + b) * dp - a * _dot(b, dp) - b * _dot(a, dp)) / 2


def softmax_backward(letter, p, pq, a, b, dp):
    """ds under the softmax's backward read ``letter``."""
    if letter == "U":
        return J_apply(p, dp)
    if letter == "R":
        return J_apply(pq, dp)
    if letter == "N":
        return J_apply(a, dp)
    if letter == "K":
        return K_apply(a, dp)
    if letter == "J2":
        return J2_apply(a, b, dp)
    if letter == "Q2":
        return J2_apply(pq, a, dp)
    raise ValueError(letter)


def v_read(letter, p, pq, a):
    """The probabilities the gradient of V reads."""
    return {"U": p, "R": pq, "N": a}[letter]


def row_uses(code, p, pq, a, b, V, h):
    """One row's (dV, ds) under a policy: dV = p_hat h^T ([n, d]), ds = J_hat (V h)."""
    sm, vl = parse(code)
    dp = V @ h
    ds = softmax_backward(sm, p, pq, a, b, dp)
    dV = np.outer(v_read(vl, p, pq, a), h)
    return dV, ds


# -- attention ------------------------------------------------------------------------------

def probabilities(Q, Kt, causal, c):
    """fp64 softmax probabilities P [..., S, S] of c Q K^T (causal: key j <= query i)."""
    Q, Kt = (np.asarray(x, dtype=np.float64) for x in (Q, Kt))
    S = Q.shape[-2]
    s = c * (Q @ np.swapaxes(Kt, -1, -2))
    if causal:
        s = np.where(np.tril(np.ones((S, S), dtype=bool)), s, -np.inf)
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def store(P32, fmt, fwd_mode, seed, store_id):
    """The forward's FP8 store of P: (codes, s, p_q, y = fl32(P / s))."""
    P32 = np.asarray(P32, dtype=np.float32)
    q = qround.qround(P32, fmt, fwd_mode, seed, 0, store_id * 256)
    pq = qround.dequant(q.codes, q.scale, fmt)
    return q.codes, q.scale, pq, qround.scaled(P32, q.scale)


def new_rounding(y, fmt, s, seed, trial, use, elems):
    """s * val of a stochastic rounding of the scaled probabilities y (all >= 0)."""
    a = np.minimum(np.asarray(y, dtype=np.float32).astype(np.float64), fmt.fmax)
    return fp8.sr_mag(a, fmt, philox.words(seed, trial, use, elems)) * np.float64(s)


def check(Q, Kt, V, dO, *, causal=True, c=None, fmt=fp8.E4M3, fwd_mode=qround.RNE,
          policies=("U/R", "R/R", "U/U", "N/N", "R/U", "K/R", "J2/R", "Q2/R"), K=16, seed=0,
          store_id=0, P=None, heads=None, rows=None):
    """Reference gradients and each policy's trial statistics for the P store.

    Q, Kt, V, dO: [B, H, S, dh]. P: the realized fp32 probabilities [B, H, S, S] to store
    (default: this oracle's fp64 P rounded to fp32). heads: list of (b, h) to compute
    (default all); the store's scale always comes from the whole P. rows: query indices to
    compute (default all): dQ is then exact on those rows, while dK and dV sum only over them
    (exact for a key whose every contributing query is among them).
    Returns the forward (codes, scale, O), the reference dQ, dK, dV per head and, per
    policy, (mean, bias, se) of dQ, dK and dV over the K trials.
    """
    Q, Kt, V, dO = (np.asarray(x, dtype=np.float32).astype(np.float64) for x in (Q, Kt, V, dO))
    B, H, S, dh = Q.shape
    c = 1.0 / np.sqrt(dh) if c is None else c
    P32 = (probabilities(Q, Kt, causal, c) if P is None else np.asarray(P, np.float64)).astype(np.float32)
    codes, s, pq, y = store(P32, fmt, fwd_mode, seed, store_id)
    p = P32.astype(np.float64)
    heads = [(b, h) for b in range(B) for h in range(H)] if heads is None else list(heads)
    rows = np.arange(S) if rows is None else np.asarray(rows)
    base = store_id * 256
    out = {"codes": codes, "scale": s, "O": pq @ V, "P": P32, "heads": heads, "rows": rows}
    refs = {"dQ": [], "dK": [], "dV": []}
    tr = {code: {"dQ": [], "dK": [], "dV": []} for code in policies}
    for (bb, hh) in heads:
        # the element index of P[bb, hh, i, j] is ((bb H + hh) S + i) S + j
        elem = ((bb * H + hh) * S + rows[:, None].astype(np.uint64)) * S + np.arange(S, dtype=np.uint64)[None, :]
        yi = y[bb, hh][rows]
        pi, pqi, Vi, dOi, Qi, Ki = p[bb, hh][rows], pq[bb, hh][rows], V[bb, hh], dO[bb, hh][rows], Q[bb, hh][rows], Kt[bb, hh]
        dp = dOi @ Vi.T
        grads = lambda ds, pv: (c * (ds @ Ki), c * (ds.T @ Qi), pv.T @ dOi)
        for name, g in zip(("dQ", "dK", "dV"), grads(J_apply(pi, dp), pqi)):
            refs[name].append(g)
        for code in policies:
            sm, vl = parse(code)
            nd = draws(code)
            per = {"dQ": [], "dK": [], "dV": []}
            for k in range(1, (K if nd else 1) + 1):
                a = new_rounding(yi, fmt, s, seed, k, base + 1, elem) if nd >= 1 else None
                b = new_rounding(yi, fmt, s, seed, k, base + 2, elem) if nd >= 2 else None
                ds = softmax_backward(sm, pi, pqi, a, b, dp)
                for name, g in zip(("dQ", "dK", "dV"), grads(ds, v_read(vl, pi, pqi, a))):
                    per[name].append(g)
            for name in per:
                tr[code][name].append(np.stack(per[name] * (1 if nd else K)))
    for name in refs:
        out[name + "_ref"] = np.stack(refs[name])
    for code in policies:
        out[code] = {name: trial_stats(np.stack(tr[code][name], axis=1), out[name + "_ref"])
                     for name in ("dQ", "dK", "dV")}
    return out
