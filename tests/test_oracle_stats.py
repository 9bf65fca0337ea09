"""Pins of the trial statistics (oracle/stats.py)."""
import numpy as np
import scipy.stats

from oracle import stats


def test_se_matches_scipy_sem():
    rng = np.random.default_rng(0)
    g = rng.normal(size=(37, 11))
    ref = rng.normal(size=11)
    mean, bias, se = stats.trial_stats(g, ref)
    assert np.allclose(mean, g.mean(0), rtol=0, atol=1e-15)
    assert np.allclose(bias, g.mean(0) - ref, rtol=0, atol=1e-15)
    assert np.allclose(se, scipy.stats.sem(g, axis=0, ddof=1), rtol=1e-13, atol=0)


def test_deterministic_trials_have_zero_se():
    g = np.tile(np.arange(5.0), (8, 1))
    _, bias, se = stats.trial_stats(g, np.arange(5.0))
    assert np.all(se == 0) and np.all(bias == 0)


def test_R_statistic_by_hand():
    # R = ||m||^2 / sum se^2 (App. D.4)
    s = stats.summary(np.array([3.0, 4.0]), np.array([1.0, 2.0]), np.array([0.0, 1.0]))
    assert s["bias_l2"] == 5.0 and s["ref_l2"] == 1.0 and s["R"] == 25.0 / 5.0
