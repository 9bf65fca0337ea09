"""Pins of the per-token b-bit grid store oracle (oracle/grid_store.py).

* the codec: P(up) = F / 2^32 equals the exact fraction of |y| (rationals), so E[q] = y, and no
  code leaves [-(2^(b-1) - 1), 2^(b-1) - 1];
* the policies' means over the new rounding, by exact enumeration of every outcome on a small
  tensor (fractions): N at the weight use has U/U's mean and U/R+e the reference's, up to the fp32
  rounding of the grid values; N at the gain use reads the original's mean;
* the reference gradients against torch.autograd of the straight-through program (fp64).
"""
from fractions import Fraction as Fr
import itertools

import numpy as np
import pytest
import torch

from oracle import grid_store as gs
from oracle.norm_store import rmsnorm_fp32


def test_up_probability_is_the_exact_fraction_and_codes_stay_on_the_grid():
    rng = np.random.default_rng(0)
    for bits in (5, 6):
        u = (rng.standard_normal((64, 96)) * rng.uniform(0.01, 10, (64, 1))).astype(np.float32)
        s = gs.step_of(u, bits)
        lo, F, neg, nsat = gs.bracket(u, s, bits)
        M = 2 ** (bits - 1) - 1
        y = (u / s[:, None]).astype(np.float32)
        for a, l, f in zip(np.abs(y).ravel()[:2000], lo.ravel()[:2000], F.ravel()[:2000]):
            a = min(Fr(float(a)), Fr(M))
            frac = a - int(a)
            assert int(l) == int(a)
            if frac * 2 ** 32 == int(frac * 2 ** 32):           # at most 32 fraction bits
                assert Fr(int(f), 2 ** 32) == frac               # P(up) = frac: E[q] = y
        q, s2, v, _ = gs.store(u, bits, seed=3, trial=0, use=0)
        assert np.all(np.abs(q) <= M) and np.array_equal(s, s2)
        assert np.all(np.abs(q).max(axis=1) >= M - 1)            # every row spans its grid
        np.testing.assert_array_equal(v, (q.astype(np.float32) * s[:, None]).astype(np.float32))


def enumerate_means(z, u, uq, s, bits, gamma, du, dY):
    """Exact expectation of every policy's (dgamma, dW) over all outcomes of the new rounding."""
    lo, F, neg, _ = gs.bracket(u, s, bits)
    cells = []
    for l, f, n in zip(lo.ravel(), F.ravel(), neg.ravel()):
        p = Fr(int(f), 2 ** 32)
        cells.append([(gs.rounded(l, f, n, 0), 1 - p)] + ([(gs.rounded(l, f, n, 2 ** 32 - 1), p)] if f else []))
    acc = {c: None for c in gs.POLICIES}
    for combo in itertools.product(*cells):
        w = Fr(1)
        for _, pw in combo:
            w *= pw
        q = np.array([c for c, _ in combo]).reshape(u.shape)
        uf = gs.value(q, s)
        for c in gs.POLICIES:
            dg, dw = gs.policy_grads(c, z, u, uq, uf, gamma, du, dY)
            term = (np.vectorize(Fr)(dg) * w, np.vectorize(Fr)(dw) * w)
            acc[c] = term if acc[c] is None else (acc[c][0] + term[0], acc[c][1] + term[1])
    return {c: (v[0].astype(float), v[1].astype(float)) for c, v in acc.items()}


@pytest.mark.parametrize("bits", [3, 5])
def test_policy_means_by_exact_enumeration(bits):
    rng = np.random.default_rng(bits)
    X = rng.standard_normal((2, 4)).astype(np.float32)
    gamma = (1 + 0.1 * rng.standard_normal(4)).astype(np.float32)
    W = rng.standard_normal((4, 3)).astype(np.float32)
    dY = rng.standard_normal((2, 3)).astype(np.float32)
    z, u, _ = rmsnorm_fp32(X, gamma, 1e-5)
    q, s, uq, _ = gs.store(u, bits, seed=1, trial=0, use=0)
    du = dY.astype(np.float64) @ W.astype(np.float64).T
    m = enumerate_means(z, u, uq, s, bits, gamma, du, dY)
    dW_ref = uq.astype(np.float64).T @ dY
    dW_U = u.astype(np.float64).T @ dY
    dg_ref = (z.astype(np.float64) * du).sum(0)
    # policies that draw nothing are their single pass
    for c in ("U/R", "U/U", "R/R"):
        dg, dw = gs.policy_grads(c, z, u, uq, None, gamma, du, dY)
        np.testing.assert_allclose(m[c][0], dg, rtol=1e-15)
        np.testing.assert_allclose(m[c][1], dw, rtol=1e-15)
    np.testing.assert_allclose(m["U/R"][1], dW_ref, rtol=1e-15)
    np.testing.assert_allclose(m["U/U"][1], dW_U, rtol=1e-15)
    # N at the weight use has U/U's mean; U/R+e the reference's (fp32 values: ~1e-7)
    for c in ("U/N", "R/N", "N/N"):
        np.testing.assert_allclose(m[c][1], dW_U, rtol=2e-6, atol=2e-6 * np.abs(dW_U).max())
    np.testing.assert_allclose(m["U/R+e"][1], dW_ref, rtol=2e-6, atol=2e-6 * np.abs(dW_ref).max())
    # N at the gain use reads the original's mean; R at the gain use adds sum (u_q - u) / gamma du
    for c in ("N/R", "N/N"):
        np.testing.assert_allclose(m[c][0], dg_ref, rtol=2e-6, atol=2e-6 * np.abs(dg_ref).max())
    r_sum = (((uq.astype(np.float64) - u) / gamma.astype(np.float64)) * du).sum(0)
    np.testing.assert_allclose(m["R/R"][0] - dg_ref, r_sum, rtol=1e-5, atol=1e-6 * np.abs(dg_ref).max())
    assert np.abs(r_sum).max() > 1e-4 * np.abs(dg_ref).max()      # the gain use needs the original


def test_reference_matches_autograd():
    g = torch.Generator().manual_seed(5)
    T, d, n = 6, 16, 8
    X = torch.randn(T, d, generator=g)
    gamma = 1 + 0.1 * torch.randn(d, generator=g)
    W = torch.randn(d, n, generator=g) / d ** 0.5
    dY = torch.randn(T, n, generator=g)
    out = gs.check(X.numpy(), gamma.numpy(), W.numpy(), dY.numpy(), bits=6, K=2, seed=1, policies=("U/R",))
    Xr, gr, Wr = (t.double().clone().requires_grad_(True) for t in (X, gamma, W))
    z = Xr * torch.rsqrt((Xr * Xr).mean(-1, keepdim=True) + 1e-5)
    u = gr * z
    uq = torch.from_numpy(out["uq"].astype(np.float64))
    y = (u + (uq - u).detach()) @ Wr
    (y * dY.double()).sum().backward()
    np.testing.assert_allclose(out["dW_ref"], Wr.grad.numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(out["dgamma_ref"], gr.grad.numpy(), rtol=1e-5, atol=1e-6)
    np.testing.assert_allclose(out["dX_ref"], Xr.grad.numpy(), rtol=1e-5, atol=1e-6)
