"""GPU parity: bs_attn_level2_policy against the oracle (oracle/level2.py).

The oracle's fp32 output O is handed to both sides, so every trial's store agrees; the means
over trials of the reference gradients and of each policy's dQ and dK, the mean incoming
gradient, the D use's split (mean error, mean-error part, coupling, se) and the paired
statistic must agree within 1e-5 (normwise relative; a split part that is zero in real
arithmetic is compared against the size of the error it splits).
"""
import numpy as np
import pytest
import torch

from oracle import fp8, level2, qround as oq
from paper_2609_39813_amd import synth
from tests.parity import assert_rel, assert_zero_where_oracle_zero, to_np

pytestmark = pytest.mark.gpu
TOL = 1e-5
FMTS = {"e4m3": fp8.E4M3, "e5m2": fp8.E5M2}
MODES = {"rne": oq.RNE, "sr": oq.SR}


def inputs(B, H, S, seed):
    return [t.to(torch.bfloat16) for t in synth.attention_inputs(B, H, S, 64, torch.float32, stream=400 + seed)]


def case(lib, B, H, S, *, seed, causal=True, fmt="e4m3", fwd_mode="sr", beta=1.0, pols=("U", "R", "N"), K=8,
         heads=None):
    Q, K_, V, dO = inputs(B, H, S, seed)
    ref = level2.check(Q.float().numpy(), K_.float().numpy(), V.float().numpy(), dO.float().numpy(), causal=causal,
                       fmt=FMTS[fmt], fwd_mode=MODES[fwd_mode], beta=beta, policies=tuple(dict.fromkeys(pols)), K=K,
                       seed=seed, store_id=1, heads=heads)
    print(f"[level2] shape={(B, H, S)} causal={causal} fmt={fmt} fwd={fwd_mode} beta={beta} pols={pols} K={K}",
          flush=True)
    out = lib.attn_level2_policy(Q.cuda(), K_.cuda(), V.cuda(), dO.cuda(), causal=causal,
                                 O=torch.from_numpy(np.ascontiguousarray(ref["O32"])).cuda(), fmt=fmt,
                                 fwd_mode=fwd_mode, beta=beta, policies=pols, K=K, seed=seed, store_id=1)
    torch.cuda.synchronize()
    return out, ref


def compare(out, ref, pols):
    B, H, S, dh = out["dQ_ref"].shape
    idx = [b * H + h for b, h in ref["heads"]]
    sel = lambda t: to_np(t).reshape(B * H, *t.shape[2:])[idx]
    assert float(out["O_scale"].cpu()[0]) == float(ref["scale"])
    assert_rel(sel(out["dO_mean"]), ref["dO_mean"], TOL, "mean incoming gradient")
    for name, got in (("dQ", "dQ_ref"), ("dK", "dK_ref"), ("dV", "dV"), ("D", "D_ref")):
        assert_rel(sel(out[got]), ref[name + "_ref"], TOL, name + "_ref")
    shp = out["dQ_ref"].shape
    rows = lambda t: to_np(t).reshape(B * H, S)[idx]
    for i, p in enumerate(pols):
        for name in ("dQ", "dK"):
            m = sel(out[name]["mean"][i].reshape(shp))
            b = sel(out[name]["bias"][i].reshape(shp))
            om, ob, _ = ref[p][name]
            assert_rel(m, om, TOL, f"{p} {name} mean")
            if not assert_zero_where_oracle_zero(b, ob, f"{p} {name} bias"):
                assert_rel(b, ob, TOL, f"{p} {name} bias")
        du = out["d_use"][i]
        om, ome, ocp, ose = ref[p]["D_use"]
        size = max(np.linalg.norm(om), np.linalg.norm(ome), 1e-30)
        for k, (name, o) in enumerate((("mean", om), ("mean-error part", ome), ("coupling", ocp), ("se", ose))):
            g = rows(du[k])
            if np.all(o == 0) and k < 3 and p == "U":
                assert np.all(g == 0), f"{p} {name}"
                continue
            err = np.linalg.norm(g - o)
            # an se that is zero in real arithmetic (an RNE forward repeats every trial) carries
            # only the oracle's fp64 rounding noise: it is compared at a millionth of the error's size
            scale = max(np.linalg.norm(o), 1e-6 * size) if k == 3 else max(np.linalg.norm(o), size)
            assert err <= TOL * max(scale, 1e-30), f"{p} D use {name}: {err:.3e} vs {scale:.3e}"
    Tm, Tse = ref["T"]
    for k, o in enumerate((Tm, Tse)):
        g = rows(out["T"][k])
        if np.all(o == 0):
            assert np.all(g == 0)
        else:
            assert_rel(g, o, TOL, f"T {'se' if k else 'mean'}")


@pytest.mark.parametrize("beta", [1.0, 0.0])
def test_ragged_sr_forward(lib, beta):
    out, ref = case(lib, 1, 2, 150, seed=1, beta=beta)
    compare(out, ref, ("U", "R", "N"))
    # the coupling of reading the forward's rounding: resolved when the gradient depends on it
    cp = to_np(out["d_use"][1][2]).sum()
    if beta == 0:
        assert abs(cp) < 1e-6 * np.abs(to_np(out["d_use"][1][0])).sum()


def test_rne_forward_and_policy_order(lib):
    pols = ("N", "R", "U", "R")
    out, ref = case(lib, 2, 1, 96, seed=2, fwd_mode="rne", pols=pols, K=5)
    compare(out, ref, pols)
    assert torch.equal(out["d_use"][1], out["d_use"][3])


def test_noncausal_e5m2(lib):
    out, ref = case(lib, 1, 1, 64, seed=3, causal=False, fmt="e5m2", beta=2.5, K=12)
    compare(out, ref, ("U", "R", "N"))


def test_single_trial_and_short_rows(lib):
    out, ref = case(lib, 1, 1, 7, seed=4, K=1)
    compare(out, ref, ("U", "R", "N"))


@pytest.mark.slow
def test_attention_shape_sampled_heads(lib):
    """B4 H16 S1024 at K = 32 (the bench's level-2 workload), two heads compared."""
    out, ref = case(lib, 4, 16, 1024, seed=5, K=32, heads=[(0, 0), (3, 15)])
    compare(out, ref, ("U", "R", "N"))
