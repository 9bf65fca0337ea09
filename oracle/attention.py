"""Attention backward whose correction term D reads a stored copy of O.

Test infrastructure (see ``oracle/__init__``).

Sec. 2.1 (Eq. dterm): the forward forms P = softmax(S) and O = P V. Given dO
the backward forms dV = P^T dO, dP = dO V^T and dS = P * (dP - D) with
D = rowsum(P * dP); FlashAttention takes D = rowsum(dO * O) from the saved
output instead, the same value at the original O. Reading a copy O + E adds
rowsum(dO * E) to D. The reference passes dO through the rounding of O
unchanged, so D needs the original O (App. D.2: the emulated backward takes D
from the assigned output copy, dV = P^T dO, dS = P * (dP - D)).

With scores S = c Q K^T (c the softmax scale; causal: key j <= query i), the
gradients are dQ = c dS K and dK = c dS^T Q.

Policies at the D use: U reads the original O (the fp32 forward output), R
the forward's FP8 rounding of O (stochastic by default, as in the forks of
Sec. 2.1, or to nearest), N a new stochastic rounding at the same scale. The
forward's rounding uses trial 0 and use id ``store_id*256``; new roundings use
trials 1..K and use id ``store_id*256 + 1``. The element index of O[b,h,i,c] is
((b H + h) S + i) dh + c. Everything except the store is fp64.

Parity: reference gradients pinned to torch.autograd in fp64; D from the
saved output pinned to rowsum(P * dP); the exact FP8 attention example of App.
C.6 (Table "FP8 attention") reproduced cell by cell (tests/test_oracle_attention.py).
"""
import numpy as np

from . import policy, qround, fp8
from .norm_store import fresh_values
from .stats import trial_stats


def forward(Q, Kt, V, causal=True, c=None):
    """fp64 forward: O, P, row max m, row sum l (P = exp(cS - m) / l)."""
    Q, Kt, V = (np.asarray(a, dtype=np.float64) for a in (Q, Kt, V))
    S = Q.shape[-2]
    c = 1.0 / np.sqrt(Q.shape[-1]) if c is None else c
    s = c * (Q @ np.swapaxes(Kt, -1, -2))
    if causal:
        mask = np.tril(np.ones((S, S), dtype=bool))
        s = np.where(mask, s, -np.inf)
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    l = e.sum(axis=-1, keepdims=True)
    P = e / l
    return P @ V, P, m[..., 0], l[..., 0]


def d_from_copy(dO, Ohat):
    """D = rowsum(dO * Ohat) (FlashAttention's correction term, Eq. dterm)."""
    return (np.asarray(dO, np.float64) * np.asarray(Ohat, np.float64)).sum(axis=-1)


def backward(Q, Kt, V, dO, P, D, c):
    """dQ, dK, dV of softmax attention given P and the correction term D."""
    Q, Kt, V, dO = (np.asarray(a, dtype=np.float64) for a in (Q, Kt, V, dO))
    dV = np.swapaxes(P, -1, -2) @ dO
    dP = dO @ np.swapaxes(V, -1, -2)
    dS = P * (dP - D[..., None])
    dQ = c * (dS @ Kt)
    dK = c * (np.swapaxes(dS, -1, -2) @ Q)
    return dQ, dK, dV


def check(Q, Kt, V, dO, *, causal=True, c=None, fmt=fp8.E4M3, fwd_mode=qround.SR,
          policies=("U", "R", "N"), K=32, seed=0, store_id=0, O=None, heads=None):
    """Reference gradients and each D policy's trial statistics.

    Q, Kt, V, dO: [B, H, S, dh]. O: the fp32 forward output to store (default:
    this oracle's forward rounded to fp32). heads: list of (b, h) to compute
    (default all); the store's scale always comes from the whole O.
    """
    Q, Kt, V, dO = (np.asarray(a, dtype=np.float32).astype(np.float64) for a in (Q, Kt, V, dO))
    B, H, S, dh = Q.shape
    c = 1.0 / np.sqrt(dh) if c is None else c
    O64, P, m, l = forward(Q, Kt, V, causal, c)
    O32 = O64.astype(np.float32) if O is None else np.asarray(O, dtype=np.float32)
    base = store_id * 256
    q = qround.qround(O32, fmt, fwd_mode, seed, 0, base)
    s = q.scale
    Oq = qround.dequant(q.codes, s, fmt)
    y = qround.scaled(O32, s)
    heads = [(b, h) for b in range(B) for h in range(H)] if heads is None else list(heads)
    out = {"O": O64, "O32": O32, "m": m, "l": l, "codes": q.codes, "scale": s,
           "n_saturated": q.n_saturated, "heads": heads}
    elem = np.arange(O32.size, dtype=np.uint64).reshape(O32.shape)
    refs = {"dQ": [], "dK": [], "dV": [], "D": []}
    pol_tr = {p: {"dQ": [], "dK": []} for p in policies}
    for (b, h) in heads:
        o32 = O32[b, h].astype(np.float64)
        D_ref = d_from_copy(dO[b, h], o32)
        dQ, dK, dV = backward(Q[b, h], Kt[b, h], V[b, h], dO[b, h], P[b, h], D_ref, c)
        for name, v in (("dQ", dQ), ("dK", dK), ("dV", dV), ("D", D_ref)):
            refs[name].append(v)
        for p in policies:
            ntr = K if p == "N" else 1
            tq, tk = [], []
            for k in range(1, ntr + 1):
                fresh = fresh_values(y[b, h], elem[b, h], fmt, s, seed, k, base + 1) if p == "N" else None
                Ohat = policy.read(p, o32, Oq[b, h], fresh)
                D = d_from_copy(dO[b, h], Ohat)
                gq, gk, _ = backward(Q[b, h], Kt[b, h], V[b, h], dO[b, h], P[b, h], D, c)
                tq.append(gq)
                tk.append(gk)
            reps = K if ntr == 1 else 1
            pol_tr[p]["dQ"].append(np.stack(tq * reps))
            pol_tr[p]["dK"].append(np.stack(tk * reps))
    for name in refs:
        out[name + "_ref"] = np.stack(refs[name])
    for p in policies:
        out[p] = {}
        for name in ("dQ", "dK"):
            tr = np.stack(pol_tr[p][name], axis=1)          # [K, heads, S, dh]
            out[p][name] = trial_stats(tr, out[name + "_ref"])
    return out
