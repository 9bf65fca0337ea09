"""Comparison helpers of the parity tests (no method arithmetic).

A floating-point output passes when both its normwise relative error ||a - b||_2 / ||b||_2 and
its element-wise error max |a - b| / max |b| are within the tolerance: the first bounds the error
over the whole tensor, the second catches an isolated wrong entry (a misindexed element, a dropped
tile edge) too small to move the norm. Both figures are reported on failure.
"""
import numpy as np


def to_np(t):
    return t.detach().float().cpu().numpy().astype(np.float64) if hasattr(t, "detach") else np.asarray(t, np.float64)


def rel_err(a, b):
    a, b = to_np(a), to_np(b)
    nb = np.linalg.norm(b)
    if nb == 0:
        return float(np.linalg.norm(a))
    return float(np.linalg.norm(a - b) / nb)


def max_rel_err(a, b):
    """max |a - b| / max |b| (max |a - b| when b is all zero)."""
    a, b = to_np(a), to_np(b)
    if a.size == 0 and b.size == 0:
        return 0.0
    mb = float(np.abs(b).max())
    d = float(np.abs(a - b).max())
    return d / mb if mb > 0 else d


def assert_rel(a, b, tol, what, elem_tol=None):
    """Normwise and element-wise relative error within tol (elem_tol, if given, for the second)."""
    a, b = to_np(a), to_np(b)
    assert a.shape == b.shape or a.size == b.size, f"{what}: shapes {a.shape} vs {b.shape}"
    a = a.reshape(b.shape)
    e = rel_err(a, b)
    m = max_rel_err(a, b)
    et = tol if elem_tol is None else elem_tol
    assert e <= tol and m <= et, (f"{what}: normwise relative error {e:.3e} (tol {tol:.1e}), "
                                  f"max|a-b|/max|b| {m:.3e} (tol {et:.1e})")
    return e


def assert_zero_where_oracle_zero(a, b, what):
    """Where the oracle's value is exactly zero in every draw, the kernel's must be too."""
    a, b = to_np(a), to_np(b)
    if np.all(b == 0):
        assert np.all(a == 0), f"{what}: oracle is exactly zero but kernel max |x| = {np.abs(a).max():.3e}"
        return True
    return False


def parity_ok(a, b, tol):
    """True when both relative errors of assert_rel are within tol (for planted-error tests)."""
    a, b = to_np(a), to_np(b)
    if a.size != b.size:
        return False
    a = a.reshape(b.shape)
    return rel_err(a, b) <= tol and max_rel_err(a, b) <= tol
