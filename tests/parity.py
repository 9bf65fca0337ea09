"""Comparison helpers of the parity tests (no method arithmetic)."""
import numpy as np


def to_np(t):
    return t.detach().float().cpu().numpy().astype(np.float64) if hasattr(t, "detach") else np.asarray(t, np.float64)


def rel_err(a, b):
    a, b = to_np(a), to_np(b)
    nb = np.linalg.norm(b)
    if nb == 0:
        return float(np.linalg.norm(a))
    return float(np.linalg.norm(a - b) / nb)


def assert_rel(a, b, tol, what):
    e = rel_err(a, b)
    assert e <= tol, f"{what}: normwise relative error {e:.3e} > {tol:.1e}"
    return e


def assert_zero_where_oracle_zero(a, b, what):
    """Where the oracle's value is exactly zero in every draw, the kernel's must be too."""
    a, b = to_np(a), to_np(b)
    if np.all(b == 0):
        assert np.all(a == 0), f"{what}: oracle is exactly zero but kernel max |x| = {np.abs(a).max():.3e}"
        return True
    return False
