"""GPU parity: bs_policy_bias_estimate (the generic trial reducer, App. C.4; App. D.4) against
oracle.stats: the mean error and se per output, ||mean error||, ||g_ref|| and R = ||m||^2 / sum se^2."""
import numpy as np
import pytest
import torch

from oracle import stats
from tests.parity import assert_rel, to_np

pytestmark = pytest.mark.gpu
TOL = 1e-5


def case(K, m, seed, with_ref=True, spread=1.0):
    g = torch.Generator().manual_seed(seed)
    ref = torch.randn(m, generator=g)
    bias = 0.01 * torch.randn(m, generator=g)
    delta = (bias[None, :] + spread * 0.1 * torch.randn(K, m, generator=g)).float()
    return delta, (ref if with_ref else None)


def run(lib, delta, ref):
    K, m = delta.shape
    print(f"[policy_bias] K={K} m={m} ref={ref is not None}", flush=True)
    mean, se, summ = lib.policy_bias_estimate(delta.cuda(), None if ref is None else ref.cuda())
    torch.cuda.synchronize()
    return to_np(mean), to_np(se), summ.cpu().numpy()


def oracle(delta, ref):
    d = delta.numpy().astype(np.float64)
    m_, b_, se_ = stats.trial_stats(d, np.zeros(d.shape[1]))   # delta is already a per-trial error
    s = stats.summary(m_, se_, np.zeros(1) if ref is None else ref.numpy())
    return m_, se_, s


@pytest.mark.parametrize("K,m,seed,with_ref", [
    (7, 1000003, 1, True),      # m not a multiple of the 256-wide blocks
    (32, 4099, 2, False),       # g_ref NULL: its norm reads 0
    (2, 1, 3, True),
])
def test_matches_oracle(lib, K, m, seed, with_ref):
    delta, ref = case(K, m, seed, with_ref)
    mean, se, summ = run(lib, delta, ref)
    om, ose, s = oracle(delta, ref)
    assert_rel(mean, om, TOL, "mean error")
    assert_rel(se, ose, TOL, "se")
    assert abs(summ[0] - s["bias_l2"]) <= 1e-12 * s["bias_l2"]
    assert abs(summ[1] - s["ref_l2"]) <= 1e-12 * max(s["ref_l2"], 1e-300)
    assert abs(summ[2] - s["R"]) <= 1e-10 * s["R"]


def test_one_trial_has_zero_se_and_undefined_R(lib):
    delta, ref = case(1, 5000, 4)
    mean, se, summ = run(lib, delta, ref)
    assert np.array_equal(mean, delta[0].numpy().astype(np.float64))
    assert np.all(se == 0) and np.isnan(summ[2])


def test_identical_trials_are_exact(lib):
    """Trials that all agree (a policy that draws nothing) give that value exactly and se 0."""
    row = torch.randn(3001, generator=torch.Generator().manual_seed(6))
    delta = row[None, :].repeat(5, 1).contiguous()
    mean, se, summ = run(lib, delta, None)
    assert np.array_equal(mean, row.numpy().astype(np.float64)) and np.all(se == 0)
    assert summ[1] == 0.0 and np.isnan(summ[2])


def test_empty(lib):
    mean, se, summ = run(lib, torch.zeros(3, 0), None)
    assert mean.size == 0 and summ[0] == 0.0 and summ[1] == 0.0 and np.isnan(summ[2])


def test_store_sized_output(lib):
    """m = 16384 x 1024 (a normalization store of the decoder layer's shape), K = 8: the summary
    reduces 65536 block partials."""
    delta, ref = case(8, 16384 * 1024, 7)
    mean, se, summ = run(lib, delta, ref)
    om, ose, s = oracle(delta, ref)
    assert_rel(mean, om, TOL, "mean error")
    assert_rel(se, ose, TOL, "se")
    assert abs(summ[0] - s["bias_l2"]) <= 1e-12 * s["bias_l2"]
    assert abs(summ[2] - s["R"]) <= 1e-10 * s["R"]


def test_binding_rejects_other_dtypes(lib):
    with pytest.raises(TypeError):
        lib.policy_bias_estimate(torch.zeros(2, 8, dtype=torch.float16, device="cuda"))
    with pytest.raises(TypeError):
        lib.policy_bias_estimate(torch.zeros(2, 8, device="cuda"), torch.zeros(8, dtype=torch.float64, device="cuda"))


def test_estimate_summary_of_a_call_against_the_oracle(lib):
    """App. D.4's R of a call's outputs (the N policy's dgain of the RMSNorm -> Linear check): the
    summary of the library's bias / se / ref arrays against oracle.stats.summary of the oracle's."""
    from oracle import fp8, norm_store, qround as oq
    from paper_2609_39813_amd import synth
    X, g, W, dY = synth.rmsnorm_linear_inputs(300, 128, 72, torch.float32, 2)
    out = lib.rmsnorm_linear(X.cuda(), g.cuda(), W.cuda(), dY.cuda(), policies=("U/U", "N/N"), K=24, seed=9)
    ref = norm_store.check(X.numpy(), g.numpy(), W.numpy(), dY.numpy(), fmt=fp8.E4M3, fwd_mode=oq.RNE,
                           policies=("U/U", "N/N"), K=24, seed=9)
    for i, code in enumerate(("U/U", "N/N")):
        b, s = out["dgain"]["bias"][i].contiguous(), out["dgain"]["se"][i].contiguous()
        summ = lib.estimate_summary(b, s, out["dgain_ref"]).cpu().numpy()
        torch.cuda.synchronize()
        _, ob, ose = ref[code]["dgamma"]
        want = stats.summary(ob, ose, ref["dgamma_ref"])
        assert abs(summ[0] - want["bias_l2"]) <= TOL * want["bias_l2"] + 1e-30
        assert abs(summ[1] - want["ref_l2"]) <= TOL * want["ref_l2"]
        if code == "U/U":
            assert np.isnan(summ[2]) and np.isnan(want["R"])
        else:
            assert abs(summ[2] - want["R"]) <= 3 * TOL * want["R"]
        # and exactly the summary of the library's own arrays
        bn, sn, rn = (to_np(t) for t in (b, s, out["dgain_ref"]))
        assert abs(summ[0] - np.sqrt(np.sum(bn ** 2))) <= 1e-12 * max(summ[0], 1e-300)
        if code == "N/N":
            assert abs(summ[2] - np.sum(bn ** 2) / np.sum(sn ** 2)) <= 1e-12 * summ[2]
    empty = lib.estimate_summary(torch.zeros(0, device="cuda")).cpu().numpy()
    assert empty[0] == 0 and empty[1] == 0 and np.isnan(empty[2])
