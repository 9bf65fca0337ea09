"""Level-2 averaging at the D use of the attention output store.

Test infrastructure (see ``oracle/__init__``).

App. C.1 averages a use's error over the forward's own rounding as well as over any new
rounding, the forward's inputs fixed, and splits it in two: with Delta the use's backward rule
minus the reference's and h the incoming gradient,

    E[Delta h] = E[Delta] E[h] + E[(Delta - E Delta)(h - E h)]      (mean error + coupling).

At the D use of the attention output store (Sec. 2.1, Eq. dterm) the use reads a copy O + e
of the output, the incoming gradient is h = dO, and Delta h = rowsum(e * dO) is the copy's
error in D for each query row. A coupling needs an incoming gradient that depends on the
forward's rounding (Sec. 4.2: the incoming gradient can depend on the forward's rounding but
not on a new one); here the incoming gradient of trial k is

    g_k = g(O + r_k),   g(O + x) = dO + beta x,

with r_k = deq(C_k) - O the forward's rounding in that trial: beta = 0 holds the incoming
gradient fixed, beta = 1 adds the output's deviation (the loss 1/2 ||o||^2 of App. B.3 up to
its fixed part; the deviation-coupled gradient of the TE test of Sec. 4.3 and App. C.6).

Trials k = 1..K: the forward's rounding C_k is the FP8 store of O with trial k and use id
store_id*256 (the forward resampled); a new rounding C'_k is stochastic rounding at the same
scale with trial k and use id store_id*256 + 1. U reads O (e = 0), R reads deq(C_k)
(e = r_k), N reads deq(C'_k) (e = r'_k). The element index of O[b,h,i,c] is
((b H + h) S + i) dh + c, as in ``oracle.attention``.

Each trial's reference is the straight-through backward of the forward as it ran: incoming
gradient g_k and D_ref,k = rowsum(g_k * O); each policy's backward takes D_ref,k +
rowsum(g_k * e_k). Reported per policy: the mean over trials of dQ and dK and their bias
(mean of the per-trial difference from the reference), and per query row the D use's mean
error, its mean-error part rowsum(mean e * mean g), its coupling (the remainder: the sample
form of the split is an identity) and the se over trials of Delta h; further the paired
statistic of the normalization evidence (App. E.4), T_k = 1/2 rowsum((r_k - r'_k) *
(g(O + r_k) - g(O + r'_k))), whose mean is that of Delta h under R minus under N, with its se.
Everything except the store is fp64.

Parity: the split, the paired statistic and the D-use errors are pinned by exact enumeration
(fractions) of every rounding outcome of small rows against their closed forms (R: mean
error 0, coupling beta * sum_j sigma_j^2; N and U: 0; E[T] = beta * sum_j sigma_j^2; an RNE
forward moves R's error into the mean-error part) in tests/test_oracle_level2.py; the
backward is ``oracle.attention.backward`` (pinned to torch.autograd).
"""
import numpy as np

from . import fp8, qround
from .attention import backward, d_from_copy, forward
from .norm_store import fresh_values


def split(e, g, w):
    """Delta h = rowsum(e_k * g_k) over outcomes k with weights w (summing to 1).

    e, g: [n_outcomes, ..., dh] (object arrays of fractions or floats). Returns per row the
    mean of Delta h, its mean-error part rowsum(E[e] * E[g]) and the coupling (the rest).
    """
    w = np.asarray(w, dtype=object if np.asarray(e).dtype == object else np.float64)
    wk = w.reshape((-1,) + (1,) * (np.asarray(e).ndim - 1))
    mean = ((e * g).sum(axis=-1) * wk[..., 0]).sum(axis=0)
    me = ((e * wk).sum(axis=0) * (g * wk).sum(axis=0)).sum(axis=-1)
    return mean, me, mean - me


def paired_T(r, rp, beta):
    """T_k = 1/2 rowsum((r_k - r'_k) * (g(O + r_k) - g(O + r'_k))) with g(O + x) = dO + beta x."""
    gr, grp = beta * r, beta * rp          # the fixed part dO cancels in the difference
    return ((r - rp) * (gr - grp)).sum(axis=-1) / 2


def _mean_se(x):
    x = np.asarray(x, dtype=np.float64)
    K = x.shape[0]
    m = x.mean(axis=0)
    se = np.sqrt(((x - m) ** 2).sum(axis=0) / (K - 1)) / np.sqrt(K) if K > 1 else np.zeros_like(m)
    return m, se


def check(Q, Kt, V, dO, *, causal=True, c=None, fmt=fp8.E4M3, fwd_mode=qround.SR, beta=1.0,
          policies=("U", "R", "N"), K=32, seed=0, store_id=0, O=None, heads=None):
    """Level-2 means, biases and the D-use split of each policy over K trials.

    Q, Kt, V, dO: [B, H, S, dh]. O: the fp32 forward output (default: this oracle's forward
    rounded to fp32). heads: list of (b, h) to compute (default all); the store's scale always
    comes from the whole O.
    """
    Q, Kt, V, dO = (np.asarray(a, dtype=np.float32).astype(np.float64) for a in (Q, Kt, V, dO))
    B, H, S, dh = Q.shape
    c = 1.0 / np.sqrt(dh) if c is None else c
    O64, P, m, l = forward(Q, Kt, V, causal, c)
    O32 = O64.astype(np.float32) if O is None else np.asarray(O, dtype=np.float32)
    base = store_id * 256
    s = qround.qround(O32, fmt, fwd_mode, seed, 0, base).scale
    y = qround.scaled(O32, s)
    heads = [(b, h) for b in range(B) for h in range(H)] if heads is None else list(heads)
    elem = np.arange(O32.size, dtype=np.uint64).reshape(O32.shape)
    out = {"O32": O32, "scale": s, "heads": heads}
    acc = {"ref": {"dQ": [], "dK": [], "dV": [], "D": [], "g": []}}
    per = {p: {"dQ": [], "dK": [], "dh": []} for p in policies}
    T_h = []
    for (b, h) in heads:
        o = O32[b, h].astype(np.float64)
        # the forward's rounding of each trial (the store of O at the trials' common scale s)
        r = np.stack([qround.dequant(qround.round_scaled(y[b, h], fmt, fwd_mode, seed, k, base, elem[b, h])[0], s, fmt)
                      - o for k in range(1, K + 1)])                                 # [K, S, dh]
        rp = np.stack([fresh_values(y[b, h], elem[b, h], fmt, s, seed, k, base + 1) - o
                       for k in range(1, K + 1)])
        g = dO[b, h][None] + beta * r                                               # g_k
        refs = [backward(Q[b, h], Kt[b, h], V[b, h], g[k], P[b, h], d_from_copy(g[k], o), c) for k in range(K)]
        for i, name in enumerate(("dQ", "dK", "dV")):
            acc["ref"][name].append(np.stack([x[i] for x in refs]))
        acc["ref"]["D"].append(np.stack([d_from_copy(g[k], o) for k in range(K)]))
        acc["ref"]["g"].append(g.mean(axis=0))
        for p in policies:
            e = {"U": np.zeros_like(r), "R": r, "N": rp}[p]
            tq, tk = [], []
            for k in range(K):
                gq, gk, _ = backward(Q[b, h], Kt[b, h], V[b, h], g[k], P[b, h],
                                     d_from_copy(g[k], o) + d_from_copy(g[k], e[k]), c)
                tq.append(gq - refs[k][0])
                tk.append(gk - refs[k][1])
            per[p]["dQ"].append(np.stack(tq))
            per[p]["dK"].append(np.stack(tk))
            mean, me, cp = split(e, g, np.full(K, 1.0 / K))
            _, se = _mean_se((e * g).sum(axis=-1))
            per[p]["dh"].append(np.stack([mean, me, cp, se]))
        T_h.append(np.stack(_mean_se(paired_T(r, rp, beta))))
    for name in ("dQ", "dK", "dV", "D"):
        out[name + "_ref"] = np.stack([x.mean(axis=0) for x in acc["ref"][name]])  # mean over trials
    out["dO_mean"] = np.stack(acc["ref"]["g"])
    for p in policies:
        out[p] = {}
        for name in ("dQ", "dK"):
            diff = np.stack(per[p][name], axis=1)                                   # [K, heads, S, dh]
            bias, se = _mean_se(diff)
            out[p][name] = (out[name + "_ref"] + bias, bias, se)
        out[p]["D_use"] = np.stack(per[p]["dh"], axis=1)          # [4 (mean, mean error, coupling, se), heads, S]
    out["T"] = np.stack(T_h, axis=1)                              # [2 (mean, se), heads, S]
    return out
