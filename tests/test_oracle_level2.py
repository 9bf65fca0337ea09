"""Pins of the level-2 oracle (oracle/level2.py).

Every rounding outcome of small rows is enumerated in rational arithmetic (the forward's
stochastic rounding r and an independent new rounding r', each entry on its own grid), and the
exact averages of the D use's error, its mean-error part, its coupling and the paired statistic
are compared with their closed forms: with sigma_j^2 the variance of entry j's rounding,
R (reads the forward's rounding): mean error 0, coupling beta * sum_j sigma_j^2;
N (reads a new rounding): 0 and 0; U: 0 and 0; E[T] = E[Delta h under R] - E[under N].
"""
from fractions import Fraction as Fr
import itertools

import numpy as np
import pytest
import torch

from oracle import fp8, level2, qround

ROWS = {
    # original row o, fixed incoming gradient dO, grid spacing of the rounding
    "a": ([Fr(3, 10), Fr(-7, 20), Fr(1, 8), Fr(1, 3)], [Fr(1), Fr(-2), Fr(1, 2), Fr(3)], Fr(1, 8)),
    "b": ([Fr(2, 5), Fr(-1, 6), Fr(5, 7)], [Fr(-1, 2), Fr(2), Fr(1)], Fr(1, 4)),
}


def law(o, step):
    """Per entry: [(rounding error r, probability)] of stochastic rounding onto the grid."""
    out = []
    for x in o:
        lo = (x // step) * step
        up = (x - lo) / step
        out.append([(Fr(0), Fr(1))] if up == 0 else [(lo - x, 1 - up), (lo + step - x, up)])
    return out


def outcomes(lw):
    for combo in itertools.product(*lw):
        pr = Fr(1)
        for _, q in combo:
            pr *= q
        yield np.array([v for v, _ in combo], dtype=object), pr


def enumerate_row(name, beta):
    """Stacked outcomes (r, r', weight) of the forward's and a new rounding, and sum sigma^2."""
    o, dO, step = ROWS[name]
    lw = law(o, step)
    rs, rps, ws = [], [], []
    for r, pr in outcomes(lw):
        for rp, prp in outcomes(lw):
            rs.append(r)
            rps.append(rp)
            ws.append(pr * prp)
    assert sum(ws) == 1
    var = sum(sum(q * v * v for v, q in e) for e in lw)
    assert all(sum(q * v for v, q in e) == 0 for e in lw)                 # unbiased rounding
    r, rp = np.array(rs, dtype=object), np.array(rps, dtype=object)
    g = np.array(dO, dtype=object)[None] + beta * r
    return r, rp, g, np.array(ws, dtype=object), var


@pytest.mark.parametrize("name", ["a", "b"])
@pytest.mark.parametrize("beta", [Fr(0), Fr(1), Fr(5, 2)])
def test_split_matches_closed_forms(name, beta):
    r, rp, g, w, var = enumerate_row(name, beta)
    assert var > 0
    zero = np.zeros_like(r) * Fr(0)
    got = {p: level2.split(e, g, w) for p, e in (("U", zero), ("R", r), ("N", rp))}
    assert got["U"] == (0, 0, 0)
    assert got["R"][1] == 0 and got["R"][2] == beta * var and got["R"][0] == beta * var
    assert got["N"] == (0, 0, 0)
    ET = (level2.paired_T(r, rp, beta) * w).sum()
    assert ET == got["R"][0] - got["N"][0] == beta * var


@pytest.mark.parametrize("name", ["a", "b"])
def test_rne_forward_is_a_mean_error_not_a_coupling(name):
    """A deterministic forward rounding: R's error is all mean error, its coupling is zero."""
    o, dO, step = ROWS[name]
    r1 = np.array([((x / step + Fr(1, 2)) // 1) * step - x for x in o], dtype=object)   # nearest (ties up)
    r = r1[None]
    g = np.array(dO, dtype=object)[None] + 2 * r
    mean, me, cp = level2.split(r, g, np.array([Fr(1)], dtype=object))
    assert cp == 0 and me == mean == sum(r1 * (np.array(dO, dtype=object) + 2 * r1))
    assert mean != 0


def test_sample_split_is_an_identity():
    """Over K equally weighted trials the split holds exactly: mean = mean-error part + coupling,
    the coupling being the sample covariance summed over the row."""
    rng = np.random.default_rng(1)
    e = rng.standard_normal((7, 3, 5))
    g = rng.standard_normal((7, 3, 5)) + 0.5 * e
    mean, me, cp = level2.split(e, g, np.full(7, 1 / 7))
    cov = ((e - e.mean(0)) * (g - g.mean(0))).mean(0).sum(-1)
    np.testing.assert_allclose(cp, cov, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(mean, (e * g).sum(-1).mean(0), rtol=1e-12)


def test_attention_level2_statistics():
    """check() on an attention head: U's error is exactly zero; with a fixed incoming gradient
    R's coupling vanishes exactly (g - mean g = 0); with the deviation added R's coupling is
    beta times the sample variance of the forward's rounding (close to sum_j sigma_j^2, computed
    from the grid) and N's is a covariance of independent draws (near 0); E[T] = beta sum sigma^2."""
    g = torch.Generator().manual_seed(8)
    B, H, S, dh = 1, 1, 40, 8
    Q, Kt, V, dO = (torch.randn(B, H, S, dh, generator=g).numpy() for _ in range(4))
    K = 64
    for beta in (0.0, 1.0):
        out = level2.check(Q, Kt, V, dO, causal=True, c=0.35, fmt=fp8.E4M3, fwd_mode=qround.SR, beta=beta,
                           K=K, seed=5, store_id=1)
        # sum of the per-element variances of stochastic rounding at the store's scale
        y = np.abs(qround.scaled(out["O32"], out["scale"])).astype(np.float64)
        F, lo, step = fp8.sr_threshold(np.minimum(y, fp8.E4M3.fmax), fp8.E4M3)
        f = np.asarray(F, np.float64) / 2.0 ** 32
        var = float(((np.float64(out["scale"]) * step) ** 2 * f * (1 - f)).sum())
        assert np.all(out["U"]["dQ"][1] == 0) and np.all(out["U"]["D_use"][:3] == 0)
        mR, meR, cpR, seR = out["R"]["D_use"]
        mN, meN, cpN, seN = out["N"]["D_use"]
        Tm, Tse = out["T"]
        if beta == 0:
            assert np.abs(cpR).max() < 1e-12 and np.abs(cpN).max() < 1e-12 and np.all(Tm == 0)
        else:
            assert abs(cpR.sum() - beta * var * (K - 1) / K) < 0.05 * var
            assert abs(cpN.sum()) < 0.05 * var
            assert abs(Tm.sum() - beta * var) < 0.05 * var
