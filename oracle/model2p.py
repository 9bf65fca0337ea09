"""The two-parameter model of the normalization store, averaged exactly.

Test infrastructure (see ``oracle/__init__``).

App. B.1 (Eqs. app-model-loss, app-model-update): a gain gamma in (0, 1] scales
an input of one; the forward consumes a rounding q in {0, 1} of gamma with
P(q = 1) = gamma; a weight w multiplies q. One draw's loss is

  l = (w q - 1)^2 / 2 + 2 (gamma - 3/8)^2 + (w - 1)^2 .

The backward passes zeta = dl/dq = w (w q - 1) through the rounding. A policy
that reads x_g at the gain use and x_w at the weight use updates

  d_gamma = zeta x_g / gamma + 4 (gamma - 3/8) + c,   c = w^2 (1/2 - gamma),
  d_w     = (w q - 1) x_w + 2 (w - 1).

The gain use needs the original (gamma), the weight use the rounded value (q).
A new rounding f is an independent draw with P(f = 1) = gamma; the N/N policy
hands both uses the same new draw (Fig. "policies").

Every average here is an exact enumeration over q and f in rationals.

Parity: pinned to the values the paper prints (App. B.1): minimum 9/32 at
(1/2, 1); average updates (1/2, 0) for R/R and (0, -1/4) for U/U at the
minimum; R/R at rest at gamma = 1/3, w = 1 with excess 1/18
(tests/test_oracle_model2p.py).
"""
from fractions import Fraction as Fr

from . import policy


def loss(gamma, w, q):
    return Fr(1, 2) * (w * q - 1) ** 2 + 2 * (gamma - Fr(3, 8)) ** 2 + (w - 1) ** 2


def expected_loss(gamma, w):
    """E_q[l], enumerated."""
    return (1 - gamma) * loss(gamma, w, 0) + gamma * loss(gamma, w, 1)


def update(pol, gamma, w, q, f):
    """One draw's (d_gamma, d_w) under policy pol = (gain letter, weight letter)."""
    gain_letter, weight_letter = pol
    zeta = w * (w * q - 1)
    x_g = policy.read(gain_letter, gamma, q, f)
    x_w = policy.read(weight_letter, gamma, q, f)
    c = w * w * (Fr(1, 2) - gamma)
    d_gamma = zeta * x_g / gamma + 4 * (gamma - Fr(3, 8)) + c
    d_w = (w * q - 1) * x_w + 2 * (w - 1)
    return d_gamma, d_w


def average_update(pol, gamma, w):
    """E over the forward's rounding q and the new rounding f, exactly."""
    gamma, w = Fr(gamma), Fr(w)
    tot_g, tot_w = Fr(0), Fr(0)
    for q in (0, 1):
        pq = gamma if q else 1 - gamma
        for f in (0, 1):
            pf = gamma if f else 1 - gamma
            dg, dw = update(pol, gamma, w, q, f)
            tot_g += pq * pf * dg
            tot_w += pq * pf * dw
    return tot_g, tot_w


def grad_expected_loss(gamma, w):
    """Gradient of E_q[l] by exact finite differences of the polynomial.

    E_q[l] is quadratic in w and in gamma, so a symmetric difference with any
    step is exact.
    """
    gamma, w = Fr(gamma), Fr(w)
    h = Fr(1, 1000)
    dg = (expected_loss(gamma + h, w) - expected_loss(gamma - h, w)) / (2 * h)
    dw = (expected_loss(gamma, w + h) - expected_loss(gamma, w - h)) / (2 * h)
    return dg, dw
