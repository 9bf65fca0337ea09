"""Trial statistics of a policy's gradient estimate.

Test infrastructure (see ``oracle/__init__``).

App. C.4 takes a use's mean error over trials, its standard error over trials
and z = |m| / se. App. D.4 defines the detection statistic
R = ||m||^2 / sum_j se_j^2 (about one at zero mean). Here the trials are the K
Monte Carlo roundings with the forward held fixed, g_k is the policy's gradient
in trial k and g_ref the reference gradient:

  mean = (1/K) sum_k g_k           (evaluated as g_1 + (1/K) sum_k (g_k - g_1))
  bias = mean - g_ref
  se   = sqrt( sum_k (g_k - mean)^2 / (K - 1) ) / sqrt(K)      (0 when K == 1)

Parity: se pinned to scipy.stats.sem; R and z by their definitions on
hand-computed cases (tests/test_oracle_stats.py).
"""
import numpy as np


def trial_stats(g_trials, g_ref):
    g = np.asarray(g_trials, dtype=np.float64)
    K = g.shape[0]
    # mean = g_1 + (1/K) sum_k (g_k - g_1): equal to (1/K) sum_k g_k, and exactly g_1
    # when every trial gives the same gradient (a policy that reads no new rounding)
    mean = g[0] + (g - g[0]).sum(axis=0) / K
    bias = mean - np.asarray(g_ref, dtype=np.float64)
    if K > 1:
        se = np.sqrt(((g - mean) ** 2).sum(axis=0) / (K - 1)) / np.sqrt(K)
    else:
        se = np.zeros_like(mean)
    return mean, bias, se


def summary(bias, se, g_ref):
    """||bias||_2, ||g_ref||_2 and R = ||bias||^2 / sum se^2 (nan if sum se^2 == 0)."""
    b2 = float(np.sum(np.asarray(bias, dtype=np.float64) ** 2))
    s2 = float(np.sum(np.asarray(se, dtype=np.float64) ** 2))
    return {"bias_l2": np.sqrt(b2),
            "ref_l2": float(np.sqrt(np.sum(np.asarray(g_ref, dtype=np.float64) ** 2))),
            "R": b2 / s2 if s2 > 0 else float("nan")}


def zscore(m, se):
    return abs(m) / se
