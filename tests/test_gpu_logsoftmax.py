"""GPU parity: bs_logsoftmax_reuse_check against the oracle (oracle/logsoftmax.py).

Both sides run the test in fp64 on the same seeded logits and Philox draws; the trial means
and se of the four statistics must agree to 1e-9 of their size (fp64 sums in different orders).
The paper's configuration (eps = 0.1, 128 classes, 64 rows, 4096 trials) is also checked
against the closed forms within a few se.
"""
import numpy as np
import pytest
import torch

from oracle import logsoftmax as ls

pytestmark = pytest.mark.gpu


def inputs(rows, C, seed):
    g = torch.Generator().manual_seed(600 + seed)
    z = torch.randn(rows, C, generator=g, dtype=torch.float64) * 2.0
    y = torch.randint(0, C, (rows,), generator=g, dtype=torch.int32)
    return z, y


def run(lib, rows, C, K, eps, seed, calibrate=False):
    z, y = inputs(rows, C, seed)
    print(f"[lsm] rows={rows} C={C} K={K} eps={eps} calibrate={calibrate}", flush=True)
    got = lib.logsoftmax_reuse_check(z.cuda(), y.cuda(), eps=eps, K=K, seed=seed, store_id=1,
                                     calibrate=calibrate).cpu().numpy()
    return z, y, got


@pytest.mark.parametrize("rows,C,K,eps,calibrate", [(3, 8, 40, 0.1, False), (5, 132, 33, 0.35, True),
                                                    (1, 4, 1, 0.2, False), (7, 260, 70, 0.05, False),
                                                    (4, 16, 300, 0.1, False)])
def test_statistics_match_oracle(lib, rows, C, K, eps, calibrate):
    z, y, got = run(lib, rows, C, K, eps, seed=rows, calibrate=calibrate)
    ref = ls.check(z.numpy(), y.numpy(), eps=eps, K=K, seed=rows, store_id=1, calibrate=calibrate)
    for i, name in enumerate(ls.STATS):
        m, se = ref[name]
        scale = max(abs(m), se, 1e-300)
        assert abs(got[i, 0] - m) <= 1e-9 * scale, (name, got[i, 0], m)
        assert abs(got[i, 1] - se) <= 1e-9 * max(se, 1e-300) or (K == 1 and got[i, 1] == 0), (name, got[i, 1], se)


def test_targets_outside_the_classes_match_none(lib):
    """A target outside [0, C) makes the likelihood's h zero on that row, on both sides."""
    z, y = inputs(4, 12, 3)
    y[1], y[3] = -1, 12
    got = lib.logsoftmax_reuse_check(z.cuda(), y.cuda(), eps=0.1, K=50, seed=3, store_id=1).cpu().numpy()
    ref = ls.check(z.numpy(), y.numpy(), eps=0.1, K=50, seed=3, store_id=1)
    for i, name in enumerate(ls.STATS):
        m, se = ref[name]
        assert abs(got[i, 0] - m) <= 1e-9 * max(abs(m), se, 1e-300), (name, got[i, 0], m)


def test_papers_configuration_matches_closed_forms(lib):
    eps = 0.1
    _, _, got = run(lib, 64, 128, 4096, eps, seed=9)
    target = [np.cosh(eps) - 1, np.cosh(eps) - 1, -eps * np.sinh(eps), 0.0]
    for i, name in enumerate(ls.STATS):
        assert abs(got[i, 0] - target[i]) < 5 * got[i, 1], (name, got[i])
    assert abs(got[2, 0]) > 50 * got[2, 1]                 # reuse's effect is resolved
    _, _, cal = run(lib, 64, 128, 4096, eps, seed=9, calibrate=True)
    assert abs(cal[0, 0]) < 5 * cal[0, 1]                  # LS5a: the likelihood's error is removed
    assert abs(cal[2, 0] + eps * np.tanh(eps)) < 5 * cal[2, 1]   # LS5b: reuse's effect / cosh(eps)


def test_rejected_arguments(lib):
    z, y = inputs(2, 6, 0)
    with pytest.raises(lib.BspError):
        lib.logsoftmax_reuse_check(z.cuda(), y.cuda(), K=4, ws=torch.empty(1 << 16, dtype=torch.uint8, device="cuda"))
