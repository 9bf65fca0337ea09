"""Pins of the per-tensor store (oracle/qround.py): scale, zero and non-finite cases."""
import numpy as np

from oracle import fp8, qround


def test_scale_is_ieee_single_division():
    x = np.array([0.1, -3.7, 2.5], dtype=np.float32)
    q = qround.qround(x, fp8.E4M3, qround.RNE)
    assert q.amax == np.float32(3.7)
    assert q.scale == np.float32(np.float32(3.7) / np.float32(448.0))
    # the largest entry maps to (at most one ulp around) FMAX
    assert abs(fp8.decode(q.codes, fp8.E4M3)[1]) == 448.0


def test_all_zero_tensor_has_unit_scale():
    q = qround.qround(np.zeros(10, np.float32), fp8.E5M2, qround.SR, seed=3)
    assert q.scale == 1.0 and np.all(q.codes == 0) and q.n_saturated == 0


def test_nonfinite_is_flagged():
    for bad in (np.nan, np.inf, -np.inf):
        q = qround.qround(np.array([1.0, bad], np.float32), fp8.E4M3, qround.RNE)
        assert q.nonfinite and q.codes is None


def test_sr_codes_bracket_the_scaled_value():
    rng = np.random.default_rng(5)
    x = rng.normal(size=4096).astype(np.float32)
    q = qround.qround(x, fp8.E4M3, qround.SR, seed=9, trial=2, use=1)
    y = qround.scaled(x, q.scale).astype(np.float64)
    v = fp8.decode(q.codes, fp8.E4M3)
    lo, step = fp8.bracket(np.minimum(np.abs(y), 448.0), fp8.E4M3)
    assert np.all((np.abs(v) == lo) | (np.abs(v) == lo + step))
    assert np.all((np.sign(v) == np.sign(y)) | (v == 0))
