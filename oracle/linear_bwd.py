"""Linear backward whose incoming gradient is rounded to E5M2.

Test infrastructure (see ``oracle/__init__``).

The HYBRID recipe rounds gradients to E5M2 (App. D.1). Here the incoming
gradient dY of y = X W is stochastically rounded at a per-tensor scale in the
backward, and two uses read it: dX = deq(C) W^T and dW = X^T deq(C). The
reference passes gradients through the rounding unchanged, so it uses the
unrounded dY: dX_ref = dY W^T, dW_ref = X^T dY (reading: the paper states no
reference for a gradient cast; this is its straight-through reference applied
to it).

Sharing: one rounding per trial read by both uses ("shared", use id
``store_id*256 + 1``), or separate draws per use ("per_use": ids ``+1`` for
dX and ``+2`` for dW); trials k = 1..K.

Coupling statistic: with fixed probes A [M, k] and B [k, n],
kappa = mean_k <dX_k - dX_ref, A> <dW_k - dW_ref, B>. It is the coupling part
of the split of App. C.1 between two uses of one draw; App. C.2 shows a shared
draw can bias a composed backward where separate draws do not.

Parity: exact enumeration over every rounding outcome on tiny tensors pins
E[kappa] (shared: sum sigma^2 (A W) (X B) plus the product of the mean
residuals; per use: the product of the mean residuals), and the K-trial means
lie within their Monte Carlo bands (tests/test_oracle_linear_bwd.py).
"""
import numpy as np

from . import qround, fp8
from .norm_store import fresh_values
from .stats import trial_stats

SHARED, PER_USE = "shared", "per_use"


def check(X, W, dY, *, fmt=fp8.E5M2, sharings=(SHARED, PER_USE), K=16, seed=0, store_id=0,
          A=None, B=None, dx_rows=None, dw_rows=None, dw_cols=None):
    """dx_rows selects rows of dX; dw_rows x dw_cols selects entries of dW (None: all). With a
    selection, the probes must vanish outside it (A outside the rows of dX, B outside the entries
    of dW), so that the coupling statistic needs the selected outputs only."""
    X64 = np.asarray(X, dtype=np.float32).astype(np.float64)
    W64 = np.asarray(W, dtype=np.float32).astype(np.float64)
    dY32 = np.asarray(dY, dtype=np.float32)
    dY64 = dY32.astype(np.float64)
    M, kdim = X64.shape
    n = W64.shape[1]
    xr = np.arange(M) if dx_rows is None else np.asarray(dx_rows)
    wr = np.arange(kdim) if dw_rows is None else np.asarray(dw_rows)
    wc = np.arange(n) if dw_cols is None else np.asarray(dw_cols)
    full = dx_rows is None and dw_rows is None and dw_cols is None
    amax = np.float32(np.max(np.abs(dY32)))
    s = qround.scale_of(amax, fmt)
    y = qround.scaled(dY32, s)
    elem = np.arange(dY32.size, dtype=np.uint64).reshape(dY32.shape)
    out = {"scale": s, "dX_ref": dY64[xr] @ W64.T, "dW_ref": X64[:, wr].T @ dY64[:, wc]}
    base = store_id * 256
    if A is not None and not full:
        A = np.asarray(A, dtype=np.float64)
        B = np.asarray(B, dtype=np.float64)
        inside_a = np.zeros(A.shape, dtype=bool)
        inside_a[xr] = True
        inside_b = np.zeros(B.shape, dtype=bool)
        inside_b[np.ix_(wr, wc)] = True
        if np.any(A[~inside_a] != 0) or np.any(B[~inside_b] != 0):
            raise ValueError("probes must vanish outside the selected outputs")
    for sh in sharings:
        use1, use2 = base + 1, (base + 1 if sh == SHARED else base + 2)
        tx, tw, kap = [], [], []
        for k in range(1, K + 1):
            if full:
                g1 = fresh_values(y, elem, fmt, s, seed, k, use1)
                g2 = g1 if use2 == use1 else fresh_values(y, elem, fmt, s, seed, k, use2)
                dXk, dWk = g1 @ W64.T, X64.T @ g2
                if A is not None:
                    kap.append(np.sum((dXk - out["dX_ref"]) * A) * np.sum((dWk - out["dW_ref"]) * B))
            else:
                g1 = fresh_values(y[xr], elem[xr], fmt, s, seed, k, use1)
                g2 = fresh_values(y[:, wc], elem[:, wc], fmt, s, seed, k, use2)
                dXk, dWk = g1 @ W64.T, X64[:, wr].T @ g2
                if A is not None:
                    kap.append(np.sum((dXk - out["dX_ref"]) * A[xr]) *
                               np.sum((dWk - out["dW_ref"]) * B[np.ix_(wr, wc)]))
            tx.append(dXk)
            tw.append(dWk)
        out[sh] = {"dX": trial_stats(np.stack(tx), out["dX_ref"]),
                   "dW": trial_stats(np.stack(tw), out["dW_ref"])}
        if kap:
            out[sh]["kappa"] = float(np.mean(kap))
            out[sh]["kappa_trials"] = np.array(kap)
    return out
