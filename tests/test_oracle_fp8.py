"""Pins of the oracle's FP8 codec (oracle/fp8.py, oracle/qround.py).

* decode: every finite code against torch's float8 -> float32 conversion;
* round to nearest even: against torch's float32 -> float8 casts (round to
  nearest even, not saturating) for |y| <= FMAX, and against a brute-force
  nearest-of-all-codes search;
* stochastic rounding: the probability of rounding up equals the exact
  fraction of the step (rationals), the expectation equals y exactly, and
  Monte Carlo frequencies over Philox words agree with it.
"""
from fractions import Fraction as Fr

import numpy as np
import pytest
import torch

from oracle import fp8, philox, qround

TORCH = {"e4m3": torch.float8_e4m3fn, "e5m2": torch.float8_e5m2}
FMTS = [fp8.E4M3, fp8.E5M2]


def finite_codes(fmt):
    c = np.arange(256, dtype=np.uint8)
    t = torch.from_numpy(c).view(TORCH[fmt.name]).float().numpy()
    return c[np.isfinite(t)], t[np.isfinite(t)]


@pytest.mark.parametrize("fmt", FMTS, ids=lambda f: f.name)
def test_decode_matches_torch(fmt):
    c, t = finite_codes(fmt)
    assert np.array_equal(fp8.decode(c, fmt), t.astype(np.float64))


def sample_values(fmt, n=20000, seed=0):
    rng = np.random.default_rng(seed)
    _, grid = finite_codes(fmt)
    grid = np.unique(np.abs(grid.astype(np.float64)))
    mids = (grid[1:] + grid[:-1]) / 2                    # exact ties
    e = rng.uniform(np.log2(fmt.min_sub) - 3, np.log2(fmt.fmax), n)
    rnd = np.exp2(e) * rng.choice([-1, 1], n)
    near = np.concatenate([np.nextafter(mids.astype(np.float32), np.float32(0)),
                           np.nextafter(mids.astype(np.float32), np.float32(np.inf))])
    vals = np.concatenate([grid, -grid, mids, -mids, near, rnd, [0.0, -0.0, fmt.fmax, -fmt.fmax,
                                                                  fmt.min_sub / 2, -fmt.min_sub / 2]])
    vals = vals.astype(np.float32)
    return vals[np.abs(vals) <= fmt.fmax]


@pytest.mark.parametrize("fmt", FMTS, ids=lambda f: f.name)
def test_rne_matches_torch_cast(fmt):
    y = sample_values(fmt)
    codes, nsat = qround.round_scaled(y, fmt, qround.RNE)
    assert nsat == 0
    want = torch.from_numpy(y).to(TORCH[fmt.name]).view(torch.uint8).numpy()
    assert np.array_equal(codes, want)


@pytest.mark.parametrize("fmt", FMTS, ids=lambda f: f.name)
def test_rne_is_nearest_of_all_codes(fmt):
    y = sample_values(fmt, n=3000, seed=1).astype(np.float64)
    c, vals = finite_codes(fmt)
    vals = vals.astype(np.float64)
    got = fp8.decode(qround.round_scaled(y.astype(np.float32), fmt, qround.RNE)[0], fmt)
    dist = np.abs(y[:, None] - vals[None, :])
    best = dist.min(axis=1)
    assert np.all(np.abs(y - got) == best)


@pytest.mark.parametrize("fmt", FMTS, ids=lambda f: f.name)
def test_clamp_counts_out_of_range(fmt):
    y = np.array([fmt.fmax * 1.01, -fmt.fmax * 3, fmt.fmax], dtype=np.float32)
    codes, nsat = qround.round_scaled(y, fmt, qround.RNE)
    assert nsat == 2
    assert np.array_equal(fp8.decode(codes, fmt), [fmt.fmax, -fmt.fmax, fmt.fmax])


def test_negative_zero_result_keeps_sign():
    for fmt in FMTS:
        codes, _ = qround.round_scaled(np.array([-0.0, -fmt.min_sub / 4, 0.0], np.float32), fmt, qround.RNE)
        assert list(codes) == [0x80, 0x80, 0x00]


@pytest.mark.parametrize("fmt", FMTS, ids=lambda f: f.name)
def test_sr_probability_is_exact_fraction(fmt):
    y = sample_values(fmt, n=4000, seed=2)
    y = y[np.abs(y) >= (2.0 ** -18 if fmt is fp8.E4M3 else 2.0 ** -25)]
    a = np.abs(y).astype(np.float64)
    F, lo, step = fp8.sr_threshold(a, fmt)
    for ai, Fi, li, si in zip(a[:1500], F[:1500], lo[:1500], step[:1500]):
        frac = (Fr(float(ai)) - Fr(float(li))) / Fr(float(si))
        assert 0 <= frac < 1
        assert Fr(int(Fi), 2**32) == frac            # P(up) = frac exactly
        # E[value] = lo + P(up) * step equals the input exactly (unbiased)
        assert Fr(float(li)) + Fr(int(Fi), 2**32) * Fr(float(si)) == Fr(float(ai))


def test_sr_of_grid_values_is_identity():
    for fmt in FMTS:
        c, vals = finite_codes(fmt)
        R = np.full(vals.shape, 0xFFFFFFFF, dtype=np.uint64)
        got = fp8.sr_mag(np.abs(vals).astype(np.float64), fmt, R)
        assert np.array_equal(got, np.abs(vals))


def test_sr_threshold_boundaries():
    fmt = fp8.E4M3
    a = np.array([1.0 + 1 / 16], dtype=np.float64)       # half way between 1 and 1.125
    F, lo, step = fp8.sr_threshold(a, fmt)
    assert int(F[0]) == 2**31 and lo[0] == 1.0 and step[0] == 0.125
    R = np.array([2**31 - 1, 2**31], dtype=np.uint64)
    got = fp8.sr_mag(np.repeat(a, 2), fmt, R)
    assert list(got) == [1.0, 1.125]                    # up iff R + F >= 2**32


@pytest.mark.parametrize("fmt", FMTS, ids=lambda f: f.name)
def test_sr_monte_carlo_frequency(fmt):
    rng = np.random.default_rng(3)
    y = np.float32(rng.uniform(0.1, fmt.fmax / 2, 64))
    a = np.abs(y).astype(np.float64)
    F, lo, step = fp8.sr_threshold(a, fmt)
    p = F.astype(np.float64) / 2**32
    K = 4000
    ups = np.zeros(64)
    for k in range(K):
        R = philox.words(11, k, 3, np.arange(64, dtype=np.uint64))
        ups += fp8.sr_mag(a, fmt, R) > lo
    se = np.sqrt(p * (1 - p) / K) + 1e-12
    z = np.abs(ups / K - p) / se
    assert np.all(z[(p > 0.01) & (p < 0.99)] < 5)


def test_planted_sr_threshold_off_by_one_fails_the_pins(monkeypatch):
    """Round up only when R + F exceeds 2^32 (one too strict), or a threshold F one too large:
    the boundary pin and the exact-probability pin must fail."""
    threshold = fp8.sr_threshold

    def strict(a, fmt, R):
        F, lo, step = threshold(a, fmt)
        up = (np.asarray(R, dtype=np.uint64) + F) > np.uint64(1 << 32)
        return np.where(up & (F > 0), lo + step, lo)
    monkeypatch.setattr(fp8, "sr_mag", strict)
    with pytest.raises(AssertionError):
        test_sr_threshold_boundaries()
    monkeypatch.undo()
    monkeypatch.setattr(fp8, "sr_threshold", lambda a, fmt: (lambda F, lo, s: (F + np.uint64(1), lo, s))(
        *threshold(a, fmt)))
    with pytest.raises(AssertionError):
        test_sr_probability_is_exact_fraction(fp8.E4M3)
