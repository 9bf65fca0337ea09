"""The kernels form y = fl32(x / s) as fl32(fl64(x) * fl64(1 / s)) (one fp64 multiply instead of
an IEEE fp32 division per element). The two agree for all float x, s: the fp64 product is within
2^-52 relative of x / s, and a quotient of two floats is never a rounding midpoint and, when
inexact, lies at least 2^-49 relative away from every midpoint. This checks the claim on random
pairs across the exponent range, on quotients built to sit next to midpoints, and on special
values (numpy's float32 division is the IEEE reference)."""
import numpy as np


def both(x, s):
    with np.errstate(all="ignore"):
        ref = (x / s).astype(np.float32)
        got = (x.astype(np.float64) * (1.0 / s.astype(np.float64))).astype(np.float32)
    same = (ref.view(np.uint32) == got.view(np.uint32)) | (np.isnan(ref) & np.isnan(got))
    return same


def test_random_pairs_across_binades():
    rng = np.random.default_rng(7)
    n = 2_000_000
    s = ((rng.random(n, dtype=np.float32) + 0.5) * np.float32(2.0) ** rng.integers(-140, 120, n)).astype(np.float32)
    x = rng.integers(0, 0x7F800000, n, dtype=np.uint32).view(np.float32)
    x = np.where(rng.random(n) < 0.5, -x, x).astype(np.float32)
    assert both(x, s).all()


def test_quotients_next_to_midpoints():
    rng = np.random.default_rng(8)
    n = 2_000_000
    s = ((rng.random(n) + 0.5) * 2.0 ** rng.integers(-60, 60, n)).astype(np.float32)
    k = rng.integers(1 << 23, 1 << 24, n).astype(np.float64)
    with np.errstate(all="ignore"):
        x = (s.astype(np.float64) * (k + 0.5) * 2.0 ** rng.integers(-40, 0, n)).astype(np.float32)
    assert both(x, s).all()


def test_special_values():
    vals = np.array([0.0, -0.0, 1e-45, -1e-45, 1.17549435e-38, 3.4028235e38, -3.4028235e38, np.inf, -np.inf,
                     np.nan, 1.0, 448.0, 57344.0], dtype=np.float32)
    x, s = np.meshgrid(vals, vals)
    assert both(x.ravel(), s.ravel()).all()
