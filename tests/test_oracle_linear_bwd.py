"""Pins of the E5M2 Linear-backward oracle (oracle/linear_bwd.py).

E[kappa] is enumerated exactly over every rounding outcome on tiny tensors and
compared with its closed form; the oracle's K-trial statistics are checked
against those exact expectations within their Monte Carlo bands.
"""
import itertools
from fractions import Fraction as Fr

import numpy as np
import pytest

from oracle import fp8, linear_bwd, qround


def make(M, k, n, seed):
    rng = np.random.default_rng(seed)
    X = rng.normal(size=(M, k)).astype(np.float32)
    W = (rng.normal(size=(k, n)) / np.sqrt(k)).astype(np.float32)
    dY = (rng.normal(size=(M, n)) * 0.01).astype(np.float32)
    A = rng.normal(size=(M, k))
    B = rng.normal(size=(k, n))
    return X, W, dY, A, B


def outcomes(dY):
    amax = np.float32(np.abs(dY).max())
    s = qround.scale_of(amax, fp8.E5M2)
    y = qround.scaled(dY, s).astype(np.float64)
    lo, step = fp8.bracket(np.abs(y), fp8.E5M2)
    res = []
    for yi, li, si in zip(y.ravel(), lo.ravel(), step.ravel()):
        sg = -1 if yi < 0 else 1
        p = (Fr(abs(float(yi))) - Fr(float(li))) / Fr(float(si))
        res.append((sg * Fr(float(li)) * Fr(float(s)), sg * (Fr(float(li)) + Fr(float(si))) * Fr(float(s)), p))
    return res


def test_coupling_expectation_exact_and_closed_form():
    X, W, dY, A, B = make(2, 2, 2, seed=1)
    oc = outcomes(dY)
    Xf = [[Fr(float(v)) for v in r] for r in X]
    Wf = [[Fr(float(v)) for v in r] for r in W]
    Af = [[Fr(float(v)) for v in r] for r in A]
    Bf = [[Fr(float(v)) for v in r] for r in B]
    dYf = [Fr(float(v)) for v in dY.ravel()]
    M, k, n = 2, 2, 2
    AW = [[sum(Af[t][i] * Wf[i][j] for i in range(k)) for j in range(n)] for t in range(M)]
    XB = [[sum(Xf[t][i] * Bf[i][j] for i in range(k)) for j in range(n)] for t in range(M)]
    a = [AW[t][j] for t in range(M) for j in range(n)]
    b = [XB[t][j] for t in range(M) for j in range(n)]

    def kappa(e1, e2):        # <E1 W^T, A> <X^T E2, B> written out from the definitions
        dx = sum(sum(e1[t * n + j] * Wf[i][j] for j in range(n)) * Af[t][i] for t in range(M) for i in range(k))
        dw = sum(sum(Xf[t][i] * e2[t * n + j] for t in range(M)) * Bf[i][j] for i in range(k) for j in range(n))
        return dx * dw

    def prob(bits):
        p = Fr(1)
        for bt, (_, _, ph) in zip(bits, oc):
            p *= ph if bt else 1 - ph
        return p

    def resid(bits):
        return [(hi if bt else lo) - dYf[e] for e, (bt, (lo, hi, _)) in enumerate(zip(bits, oc))]

    shared = sum(prob(bb) * kappa(resid(bb), resid(bb)) for bb in itertools.product((0, 1), repeat=4))
    per_use = sum(prob(b1) * prob(b2) * kappa(resid(b1), resid(b2))
                  for b1 in itertools.product((0, 1), repeat=4) for b2 in itertools.product((0, 1), repeat=4))
    mu = [lo + ph * (hi - lo) - dYf[e] for e, (lo, hi, ph) in enumerate(oc)]
    var = [ph * (1 - ph) * (hi - lo) ** 2 for (lo, hi, ph) in oc]
    mm = sum(m * x for m, x in zip(mu, a)) * sum(m * x for m, x in zip(mu, b))
    assert shared == sum(v * x * y for v, x, y in zip(var, a, b)) + mm
    assert per_use == mm

    out = linear_bwd.check(X, W, dY, K=6000, seed=3, A=A, B=B)
    for sh, ex in (("shared", shared), ("per_use", per_use)):
        kt = out[sh]["kappa_trials"]
        se = kt.std(ddof=1) / np.sqrt(kt.size)
        assert abs(kt.mean() - float(ex)) <= 4.5 * se


def test_trial_means_within_band_and_reference():
    X, W, dY, _, _ = make(5, 3, 4, seed=2)
    out = linear_bwd.check(X, W, dY, K=3000, seed=5)
    oc = outcomes(dY)
    Ey = np.array([float(lo + ph * (hi - lo)) for lo, hi, ph in oc]).reshape(dY.shape)
    for sh in ("shared", "per_use"):
        m, _, se = out[sh]["dX"]
        assert np.all(np.abs(m - Ey @ W.astype(np.float64).T) <= 4.5 * se + 1e-15)
        m, _, se = out[sh]["dW"]
        assert np.all(np.abs(m - X.astype(np.float64).T @ Ey) <= 4.5 * se + 1e-15)
    assert np.allclose(out["dX_ref"], dY.astype(np.float64) @ W.astype(np.float64).T, rtol=1e-15)


def test_sampled_entries_equal_full():
    X, W, dY, _, _ = make(6, 5, 7, seed=4)
    full = linear_bwd.check(X, W, dY, K=5, seed=8)
    part = linear_bwd.check(X, W, dY, K=5, seed=8, dx_rows=[1, 4], dw_rows=[0, 3], dw_cols=[2, 6])
    for sh in ("shared", "per_use"):
        assert np.allclose(part[sh]["dX"][0], full[sh]["dX"][0][[1, 4]], rtol=1e-13, atol=0)
        assert np.allclose(part[sh]["dW"][0], full[sh]["dW"][0][np.ix_([0, 3], [2, 6])], rtol=1e-13, atol=0)


def test_coupling_on_selected_outputs_equals_the_full_statistic():
    """With probes that vanish outside the selected rows of dX and entries of dW, the selected
    outputs give the same coupling statistic, trial by trial, as the full tensors; probes that do
    not vanish there are refused."""
    rng = np.random.default_rng(12)
    M, k, n = 40, 16, 24
    X, W = rng.normal(size=(M, k)), rng.normal(size=(k, n)) / 4
    dY = (rng.normal(size=(M, n)) * 0.1).astype(np.float32)
    xr, wr, wc = np.array([3, 17, 39]), np.array([0, 5]), np.array([2, 11, 23])
    A = np.zeros((M, k))
    A[xr] = rng.normal(size=(len(xr), k))
    B = np.zeros((k, n))
    B[np.ix_(wr, wc)] = rng.normal(size=(len(wr), len(wc)))
    full = linear_bwd.check(X, W, dY, K=6, seed=4, A=A, B=B)
    part = linear_bwd.check(X, W, dY, K=6, seed=4, A=A, B=B, dx_rows=xr, dw_rows=wr, dw_cols=wc)
    for sh in ("shared", "per_use"):
        np.testing.assert_allclose(part[sh]["kappa_trials"], full[sh]["kappa_trials"], rtol=1e-12, atol=1e-18)
    A[0, 0] = 1.0
    with pytest.raises(ValueError):
        linear_bwd.check(X, W, dY, K=2, seed=4, A=A, B=B, dx_rows=xr, dw_rows=wr, dw_cols=wc)
