"""Pins of the log-softmax operator test oracle (oracle/logsoftmax.py).

The backward is checked against torch.autograd in fp64; the per-entry average errors are
computed by exact enumeration of every sign pattern of the saved and the independent copy's
rounding on small rows and compared with the closed forms of App. C.5: cosh(eps) - 1 under the
likelihood (either copy), -eps sinh(eps) under the constructed loss with reuse, 0 with an
independent copy; with the reconstruction divided by cosh(eps), 0 and -eps tanh(eps).
"""
import itertools

import numpy as np
import pytest
import torch

from oracle import logsoftmax as ls


def test_backward_is_the_log_softmax_gradient():
    g = torch.Generator().manual_seed(2)
    z = torch.randn(5, 7, generator=g, dtype=torch.float64, requires_grad=True)
    h = torch.randn(5, 7, generator=g, dtype=torch.float64)
    (torch.log_softmax(z, dim=-1) * h).sum().backward()
    l = ls.log_softmax(z.detach().numpy())
    np.testing.assert_allclose(ls.backward(h.numpy(), l), z.grad.numpy(), rtol=0, atol=1e-14)
    np.testing.assert_allclose(l, torch.log_softmax(z.detach(), -1).numpy(), rtol=0, atol=1e-14)


def enumerate_errors(eps, C, calibrate):
    """Average of each (loss, copy) entry error over every sign pattern of r and r'."""
    rng = np.random.default_rng(C)
    z = rng.standard_normal((1, C))
    y = np.array([C // 2])
    l = ls.log_softmax(z)
    acc = {k: np.zeros((1, C)) for k in ls.STATS}
    n = 0
    for sr in itertools.product((-eps, eps), repeat=C):
        for srp in itertools.product((-eps, eps), repeat=C):
            errs = ls.entry_errors(l, y, np.array([sr]), np.array([srp]), np.cosh(eps) if calibrate else 1.0)
            for k in ls.STATS:
                acc[k] += errs[k]
            n += 1
    return {k: v / n for k, v in acc.items()}


@pytest.mark.parametrize("eps", [0.1, 0.35])
@pytest.mark.parametrize("C", [2, 4])
def test_average_errors_match_closed_forms(eps, C):
    e = enumerate_errors(eps, C, calibrate=False)
    np.testing.assert_allclose(e["likelihood_reuse"], np.cosh(eps) - 1, rtol=1e-13)
    np.testing.assert_allclose(e["likelihood_independent"], np.cosh(eps) - 1, rtol=1e-13)
    np.testing.assert_allclose(e["constructed_reuse"], -eps * np.sinh(eps), rtol=1e-13)
    np.testing.assert_allclose(e["constructed_independent"], 0.0, atol=1e-15)
    c = enumerate_errors(eps, C, calibrate=True)
    np.testing.assert_allclose(c["likelihood_reuse"], 0.0, atol=1e-15)
    np.testing.assert_allclose(c["constructed_reuse"], -eps * np.tanh(eps), rtol=1e-13)
    np.testing.assert_allclose(c["constructed_independent"], 0.0, atol=1e-15)


def test_monte_carlo_statistics_at_the_papers_shape():
    """64 rows x 128 classes, eps = 0.1: the trial means land on the closed forms within a few se."""
    rng = np.random.default_rng(0)
    z = rng.standard_normal((64, 128)) * 2.0
    y = rng.integers(0, 128, 64)
    out = ls.check(z, y, eps=0.1, K=256, seed=3, store_id=1)
    targets = {"likelihood_reuse": np.cosh(0.1) - 1, "likelihood_independent": np.cosh(0.1) - 1,
               "constructed_reuse": -0.1 * np.sinh(0.1), "constructed_independent": 0.0}
    for k, t in targets.items():
        m, se = out[k]
        assert se > 0 and abs(m - t) < 5 * se, (k, m, t, se)
    assert abs(out["constructed_reuse"][0]) > 20 * out["constructed_reuse"][1]    # resolved


def test_target_outside_the_classes_selects_none():
    """h = -e_y has no entry for a target outside [0, C): the likelihood's errors vanish on that
    row (g = g* = 0), under reuse and with the independent copy; other rows are unchanged."""
    rng = np.random.default_rng(5)
    z = rng.normal(0, 2, size=(3, 6))
    l = ls.log_softmax(z)
    r = np.where(rng.random((3, 6)) < 0.5, 0.1, -0.1)
    rp = np.where(rng.random((3, 6)) < 0.5, 0.1, -0.1)
    base = ls.entry_errors(l, np.array([2, 4, 1]), r, rp)
    for bad in (-1, 6):
        e = ls.entry_errors(l, np.array([2, bad, 1]), r, rp)
        for k in ("likelihood_reuse", "likelihood_independent"):
            assert np.all(e[k][1] == 0.0)
            np.testing.assert_array_equal(e[k][[0, 2]], base[k][[0, 2]])
        for k in ("constructed_reuse", "constructed_independent"):
            np.testing.assert_array_equal(e[k], base[k])
