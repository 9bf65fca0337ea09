"""GPU parity: bs_linear_bwd_policy against the oracle (oracle/linear_bwd.py)."""
import numpy as np
import pytest
import torch

from oracle import fp8, linear_bwd
from paper_2609_39813_amd import synth
from tests.parity import assert_rel, assert_zero_where_oracle_zero, to_np

pytestmark = pytest.mark.gpu
TOL = 1e-5


def run_both(lib, M, k, n, K, sharings=("shared", "per_use"), seed=5, coupling=True, oracle_kw=None, stream=40,
             fmt="e5m2", probes=None, want_se=False):
    X, W, dY, A, B = synth.linear_bwd_inputs(M, k, n, torch.bfloat16, stream)
    if probes is not None:
        A, B = probes
    print(f"[linear_bwd] M={M} k={k} n={n} K={K} {sharings} coupling={coupling} fmt={fmt}", flush=True)
    out = lib.linear_bwd_policy(X.cuda(), W.cuda(), dY.cuda(), fmt=fmt, sharings=sharings, K=K, seed=seed, store_id=2,
                                probeA=A.cuda() if coupling else None, probeB=B.cuda() if coupling else None,
                                want_se=want_se)
    torch.cuda.synchronize()
    ref = linear_bwd.check(X.float().numpy(), W.float().numpy(), dY.float().numpy(),
                           fmt=fp8.E5M2 if fmt == "e5m2" else fp8.E4M3, sharings=sharings, K=K, seed=seed,
                           store_id=2, A=A.double().numpy() if coupling else None,
                           B=B.double().numpy() if coupling else None, **(oracle_kw or {}))
    return out, ref


def compare(out, ref, sharings, M, k, n, xr=None, wr=None, wc=None, coupling=True):
    assert float(out["dY_scale"].cpu()[0]) == float(ref["scale"])
    selx = (lambda a: a) if xr is None else (lambda a: a[xr])
    selw = (lambda a: a) if wr is None else (lambda a: a[np.ix_(wr, wc)])
    assert_rel(selx(to_np(out["dX_ref"])), ref["dX_ref"], TOL, "dX_ref")
    assert_rel(selw(to_np(out["dW_ref"])), ref["dW_ref"], TOL, "dW_ref")
    for i, sh in enumerate(sharings):
        for name, sel, shape in (("dX", selx, (M, k)), ("dW", selw, (k, n))):
            m = sel(to_np(out[name]["mean"][i]).reshape(shape))
            b = sel(to_np(out[name]["bias"][i]).reshape(shape))
            om, ob, _ = ref[sh][name]
            assert_rel(m, om, TOL, f"{sh} {name} mean")
            if not assert_zero_where_oracle_zero(b, ob, f"{sh} {name} bias"):
                assert_rel(b, ob, TOL, f"{sh} {name} bias")
            if out[name]["se"] is not None:
                se = sel(to_np(out[name]["se"][i]).reshape(shape))
                assert_rel(se, ref[sh][name][2], TOL, f"{sh} {name} se")
        if coupling:
            g = float(out["coupling"][i].cpu())
            r = ref[sh]["kappa"]
            assert abs(g - r) <= TOL * max(abs(r), 1e-300) + 1e-12 * np.abs(ref[sh]["kappa_trials"]).mean(), (sh, g, r)


@pytest.mark.parametrize("M,k,n", [(200, 72, 136), (64, 64, 64), (1, 8, 8)])
def test_ragged_shared_and_per_use_with_coupling(lib, M, k, n):
    out, ref = run_both(lib, M, k, n, 12, seed=M, want_se=M == 200)
    compare(out, ref, ("shared", "per_use"), M, k, n)


def test_se_over_trials_per_use_only_and_one_trial(lib):
    """The per-trial path: se of dX and dW for a per-use policy alone (its dW series is use +2),
    and K = 1 (se 0)."""
    for K in (9, 1):
        out, ref = run_both(lib, 130, 64, 96, K, sharings=("per_use",), seed=7 + K, want_se=True)
        compare(out, ref, ("per_use",), 130, 64, 96)


def test_e4m3_gradient_store_and_no_coupling(lib):
    out, ref = run_both(lib, 130, 64, 96, 7, sharings=("per_use",), coupling=False, fmt="e4m3", seed=3)
    compare(out, ref, ("per_use",), 130, 64, 96, coupling=False)


@pytest.mark.slow
def test_config4_full_size_sampled(lib):
    """The 16384 x 2048 x 8192 launch: sampled rows of dX and entries of dW, and the coupling
    statistic kappa with probes supported on exactly those outputs (A on the sampled rows, B on the
    sampled entries), so the oracle's plain K trials over the samples give kappa exactly."""
    cfg = synth.WORKLOADS["linear_bwd_e5m2_16384x2048x8192"]
    M, k, n = cfg["M"], cfg["k"], cfg["n"]
    rng = np.random.default_rng(4)
    xr = np.sort(rng.choice(M, 6, replace=False))
    wr = np.sort(rng.choice(k, 3, replace=False))
    wc = np.sort(rng.choice(n, 5, replace=False))
    g = torch.Generator().manual_seed(44)
    A = torch.zeros(M, k)
    A[xr] = torch.randn(len(xr), k, generator=g)
    B = torch.zeros(k, n)
    B[np.ix_(wr, wc)] = torch.randn(len(wr), len(wc), generator=g)
    out, ref = run_both(lib, M, k, n, cfg["K"], sharings=cfg["sharings"], seed=cfg["seed"], coupling=True,
                        oracle_kw=dict(dx_rows=xr, dw_rows=wr, dw_cols=wc), stream=4, probes=(A, B), want_se=True)
    compare(out, ref, cfg["sharings"], M, k, n, xr=xr, wr=wr, wc=wc, coupling=True)
