"""Pins of the normalization-store oracle (oracle/norm_store.py).

* reference gradients: torch.autograd in fp64 of the straight-through program
  u_store = u + (u_q - u).detach(), y = u_store W (Sec. 1; Sec. 3.1);
* per-use errors: the closed forms of Eq. norm-uses (U at the weight use adds
  -r^T dy; R at the gain use adds sum (r / gamma) du; U at the gain use and R
  at the weight use add exactly nothing);
* new rounding: its exact expectation, enumerated over every rounding outcome
  in rationals, lies within the Monte Carlo band of the oracle's K-trial mean;
* reuse vs new rounding (Sec. 4.2): averaged over an SR forward's rounding as
  well, R and N give the same mean gradient exactly when the incoming gradient
  does not depend on the rounding;
* the fixed fp32 order of u: checked against an explicit scalar loop.
"""
import itertools
from fractions import Fraction as Fr

import numpy as np
import pytest
import torch

from oracle import fp8, norm_store, policy, qround


def make(T, d, n, seed=0, scale=1.0):
    rng = np.random.default_rng(seed)
    X = (rng.normal(size=(T, d)) * scale).astype(np.float32)
    g = (1 + 0.1 * rng.normal(size=d)).astype(np.float32)
    W = (rng.normal(size=(d, n)) / np.sqrt(d)).astype(np.float32)
    dY = rng.normal(size=(T, n)).astype(np.float32)
    return X, g, W, dY


def test_u_follows_fixed_fp32_order():
    X, g, _, _ = make(3, 150, 4)
    z, u, r = norm_store.rmsnorm_fp32(X, g, 1e-5)
    f = np.float32
    for t in range(3):
        part = [f(0)] * 64
        for j in range(150):
            part[j % 64] = f(part[j % 64] + f(X[t, j] * X[t, j]))
        off = 32
        while off:
            for l in range(off):
                part[l] = f(part[l] + part[l + off])
            off //= 2
        rr = f(f(1) / np.sqrt(f(f(part[0] / f(150)) + f(1e-5))))
        assert rr == r[t]
        for j in range(150):
            assert u[t, j] == f(g[j] * f(X[t, j] * rr))


def test_reference_matches_autograd():
    X, g, W, dY = make(40, 24, 16, seed=1)
    out = norm_store.check(X, g, W, dY, policies=(), K=1, seed=3)
    uq = qround.dequant(out["codes"], out["scale"], fp8.E4M3)
    x = torch.tensor(X, dtype=torch.float64, requires_grad=True)
    gt = torch.tensor(g, dtype=torch.float64, requires_grad=True)
    Wt = torch.tensor(W, dtype=torch.float64, requires_grad=True)
    r = ((x * x).mean(-1, keepdim=True) + 1e-5).rsqrt()
    u = gt * (x * r)
    us = u + (torch.tensor(uq) - u).detach()
    ((us @ Wt) * torch.tensor(dY, dtype=torch.float64)).sum().backward()
    assert np.allclose(out["dW_ref"], Wt.grad.numpy(), rtol=0, atol=1e-12)
    rel = lambda a, b: np.linalg.norm(a - b) / np.linalg.norm(b)
    assert rel(out["dgamma_ref"], gt.grad.numpy()) < 1e-6
    assert rel(out["dX_ref"], x.grad.numpy()) < 1e-6
    # the wrong value at either use is far off: the reference is not U/U or R/R
    assert rel(np.asarray(out["u"], np.float64).T @ dY.astype(np.float64), Wt.grad.numpy()) > 1e-3


def test_closed_form_biases():
    X, g, W, dY = make(64, 32, 24, seed=2)
    out = norm_store.check(X, g, W, dY, policies=("U/U", "R/R", "U/R", "R/U"), K=4, seed=5)
    uq = qround.dequant(out["codes"], out["scale"], fp8.E4M3)
    r = uq - out["u"].astype(np.float64)
    du = out["du"]
    wu = -(r.T @ dY.astype(np.float64))
    # at the gain use the original is z, and u = fl32(gamma z) differs from gamma z in
    # its last bit, so the gain-use residual is taken against gamma z exactly
    rg = uq - g.astype(np.float64) * out["z"].astype(np.float64)
    gr = ((rg / g.astype(np.float64)) * du).sum(0)
    for code in ("U/U", "R/R", "U/R", "R/U"):
        bg = out[code]["dgamma"][1]
        bw = out[code]["dW"][1]
        if code[0] == "U":
            assert np.all(bg == 0)
        else:
            assert np.allclose(bg, gr, rtol=1e-9, atol=1e-12)
        if code[2] == "R":
            assert np.all(bw == 0)
        else:
            assert np.allclose(bw, wu, rtol=1e-9, atol=1e-12)
        assert np.all(out[code]["dX"][1] == 0)
        assert np.all(out[code]["dW"][2] == 0) and np.all(out[code]["dgamma"][2] == 0)


def exact_outcomes(y, fmt):
    """Per element: (lo, hi, P(hi)) of stochastic rounding, as rationals (grid in fp8 units)."""
    a = np.minimum(np.abs(y.astype(np.float64)), fmt.fmax)
    lo, step = fp8.bracket(a, fmt)
    res = []
    for ai, li, si, yi in zip(a.ravel(), lo.ravel(), step.ravel(), y.ravel()):
        sg = -1 if np.signbit(yi) else 1
        p = (Fr(float(ai)) - Fr(float(li))) / Fr(float(si))
        res.append((sg * Fr(float(li)), sg * (Fr(float(li)) + Fr(float(si))), p))
    return res


def expect(outcomes, f):
    """E[f(values)] over independent per-element outcomes, by enumeration."""
    tot = Fr(0)
    for bits in itertools.product((0, 1), repeat=len(outcomes)):
        p = Fr(1)
        vals = []
        for b, (lo, hi, ph) in zip(bits, outcomes):
            p *= ph if b else 1 - ph
            vals.append(hi if b else lo)
            if p == 0:
                break
        if p:
            tot += p * f(vals)
    return tot


def test_new_rounding_mean_within_band_of_exact_expectation():
    X, g, W, dY = make(3, 4, 3, seed=4)
    K = 4000
    out = norm_store.check(X, g, W, dY, policies=("N/N",), K=K, seed=11)
    s = Fr(float(out["scale"]))
    y = qround.scaled(out["u"], out["scale"])
    oc = exact_outcomes(y, fp8.E4M3)
    du = out["du"]
    gF = [Fr(float(v)) for v in g]
    T, d = y.shape
    mean, _, se = out["N/N"]["dgamma"]
    for j in range(d):
        ex = expect(oc, lambda v: sum(v[t * d + j] * s / gF[j] * Fr(float(du[t, j])) for t in range(T)))
        assert abs(mean[j] - float(ex)) <= 4.5 * se[j] + 1e-12
    mw, _, sw = out["N/N"]["dW"]
    for i in range(d):
        for jj in range(W.shape[1]):
            ex = expect(oc, lambda v: sum(v[t * d + i] * s * Fr(float(dY[t, jj])) for t in range(T)))
            assert abs(mw[i, jj] - float(ex)) <= 4.5 * sw[i, jj] + 1e-12


def test_reuse_equals_new_rounding_over_both_roundings():
    # SR forward; dY does not depend on the forward's rounding, so averaged over the
    # forward's rounding and the new one, R and N read values of equal mean at each use.
    X, g, W, dY = make(2, 3, 2, seed=6)
    out = norm_store.check(X, g, W, dY, fwd_mode=qround.SR, policies=(), K=1, seed=1)
    y = qround.scaled(out["u"], out["scale"])
    oc = exact_outcomes(y, fp8.E4M3)
    s = Fr(float(out["scale"]))
    du = [[Fr(float(v)) for v in row] for row in out["du"]]
    T, d = y.shape
    for j in range(d):
        gain = lambda v: sum(v[t * d + j] * s * du[t][j] for t in range(T))
        e_r = expect(oc, gain)                        # reads the forward's rounding
        e_n = expect(oc + oc, lambda v: gain(v[len(oc):]))   # reads a new, independent one
        assert e_r == e_n


def test_planted_reuse_original_swap_at_the_weight_use_fails_the_closed_forms(monkeypatch):
    """The weight use reading R where the policy says U and U where it says R (the gain use
    untouched) must fail the closed forms of Eq. norm-uses."""
    read = policy.read
    calls = {"n": 0}
    swap = {"U": "R", "R": "U", "N": "N"}

    def planted(letter, original, forward_rounding, fresh):
        calls["n"] += 1                      # per trial: the gain use, then the weight use
        return read(swap[letter] if calls["n"] % 2 == 0 else letter, original, forward_rounding, fresh)
    monkeypatch.setattr(policy, "read", planted)
    with pytest.raises(AssertionError):
        test_closed_form_biases()
