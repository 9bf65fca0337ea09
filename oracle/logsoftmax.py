"""The log-softmax operator test (Sec. 4.3; App. C.5).

Test infrastructure (see ``oracle/__init__``).

The operator's backward takes the incoming gradient h and the saved output S of a log-softmax
row and returns h - exp(S) (1^T h). The test saves S = l + r, with l the exact output and the
entries r_j independent, each +eps or -eps with probability 1/2; reuse reads this S, an
independent copy reads l + r' with r' drawn anew. With p = exp(l), g the returned gradient and
g* the operator's gradient from l with the same h, the per-trial statistic is the mean over
rows and classes of (g_j - g*_j) / p_j. Two losses:

  likelihood   h = -e_y (a fixed target y per row): the error per entry is e^{r_j} - 1, whose
               average is cosh(eps) - 1 under either copy;
  constructed  h = r (the loss 1/2 ||S - l||^2 with l held constant): the error per entry is
               -(e^{r_j} - 1) sum_k r_k, average -eps sinh(eps) under reuse, 0 with an
               independent copy.

Calibrated: the backward divides its reconstruction exp(S) by cosh(eps) (App. C.5, LS5a/LS5b):
the likelihood's error then averages to 0 and reuse's effect under the constructed loss to
-eps tanh(eps) (the coupling scaled by 1/cosh(eps)).

Draws: r_j of trial k is +eps where the element's Philox word (seed; trial k, use store_id*256)
is at least 2^31, -eps otherwise; r'_j likewise with use store_id*256 + 1. The element index of
row i, class j is i C + j. Everything is fp64, as the paper's test.

Parity: the backward is pinned to torch.autograd in fp64; the four per-entry averages are pinned
by exact enumeration of every sign pattern of small rows against cosh(eps) - 1,
-eps sinh(eps), 0 and (calibrated) 0, -eps tanh(eps) (tests/test_oracle_logsoftmax.py).
"""
import numpy as np

from . import philox

STATS = ("likelihood_reuse", "likelihood_independent", "constructed_reuse", "constructed_independent")


def log_softmax(z):
    z = np.asarray(z, dtype=np.float64)
    m = z.max(axis=-1, keepdims=True)
    return z - m - np.log(np.exp(z - m).sum(axis=-1, keepdims=True))


def backward(h, S, calibrate=1.0):
    """The operator's backward from the saved output S: h - exp(S) / calibrate * (1^T h)."""
    return h - np.exp(S) / calibrate * h.sum(axis=-1, keepdims=True)


def signs(eps, seed, trial, use, elements):
    """+eps where the element's Philox word is at least 2^31, else -eps."""
    w = philox.words(seed, trial, use, elements)
    return np.where(w >= np.uint64(1 << 31), eps, -eps)


def entry_errors(l, y, r, rp, calibrate=1.0):
    """(g - g*) / p per entry for the four (loss, copy) pairs, given the draws r (consumed) and rp."""
    p = np.exp(l)
    # h = -e_y; a target outside the classes selects none (h = 0 on that row)
    y = np.asarray(y)
    onehot = (np.arange(l.shape[-1])[None, :] == y[:, None]).astype(l.dtype)
    out = {}
    for loss, h in (("likelihood", -onehot), ("constructed", r)):
        gstar = backward(h, l)
        for copy, read in (("reuse", l + r), ("independent", l + rp)):
            out[f"{loss}_{copy}"] = (backward(h, read, calibrate) - gstar) / p
    return out


def check(z, y, *, eps=0.1, K=256, seed=0, store_id=0, calibrate=False):
    """Mean and se over the K trials of each per-trial statistic (mean over rows and classes)."""
    l = log_softmax(z)
    rows, C = l.shape
    elem = np.arange(rows * C, dtype=np.uint64).reshape(rows, C)
    cal = np.cosh(eps) if calibrate else 1.0
    base = store_id * 256
    per = {k: [] for k in STATS}
    for k in range(1, K + 1):
        r = signs(eps, seed, k, base, elem)
        rp = signs(eps, seed, k, base + 1, elem)
        errs = entry_errors(l, y, r, rp, cal)
        for name in STATS:
            per[name].append(errs[name].mean())
    out = {}
    for name in STATS:
        x = np.asarray(per[name])
        m = x.mean()
        se = np.sqrt(((x - m) ** 2).sum() / (K - 1)) / np.sqrt(K) if K > 1 else 0.0
        out[name] = (m, se)
    return out
