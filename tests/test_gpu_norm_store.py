"""GPU parity: bs_rmsnorm_linear_fwd_bwd against the oracle (oracle/norm_store.py).

FP8 codes and the scale bit for bit; gradients, means and biases within 1e-5 normwise
relative error; exact zeros where the oracle's bias is zero in every draw.
"""
import numpy as np
import pytest
import torch

from oracle import fp8, norm_store, qround as oq
from paper_2609_39813_amd import synth
from tests.parity import assert_rel, assert_zero_where_oracle_zero, to_np

pytestmark = pytest.mark.gpu
TOL = 1e-5
MODES = {"rne": oq.RNE, "sr": oq.SR}


def run_both(lib, T, d, n, dtype, K, policies, fwd_mode="rne", seed=123, store_id=0, norm_input="U",
             shared=False, oracle_kw=None, stream=2):
    X, g, W, dY = synth.rmsnorm_linear_inputs(T, d, n, dtype, stream)
    codes = [p + (":R" if norm_input == "R" else "") + (":shared" if shared else "") for p in policies]
    print(f"[norm_store] T={T} d={d} n={n} {dtype} K={K} {codes} fwd={fwd_mode}", flush=True)
    out = lib.rmsnorm_linear(X.cuda(), g.cuda(), W.cuda(), dY.cuda(), fmt="e4m3", fwd_mode=fwd_mode,
                             policies=codes, K=K, seed=seed, store_id=store_id)
    torch.cuda.synchronize()
    ref = norm_store.check(X.float().numpy(), g.numpy(), W.float().numpy(), dY.float().numpy(), eps=1e-5,
                           fmt=fp8.E4M3, fwd_mode=MODES[fwd_mode], policies=policies, K=K, seed=seed,
                           store_id=store_id, fresh_shared=shared, norm_input=norm_input, **(oracle_kw or {}))
    return out, ref


def compare(out, ref, policies, rows=None, cols=None, xrows=None, d=None, n=None):
    assert np.array_equal(out["u_codes"].cpu().numpy(), ref["codes"])
    assert float(out["u_scale"].cpu()[0]) == float(ref["scale"])
    sel_w = (lambda a: a) if rows is None else (lambda a: a[rows])
    sel_g = (lambda a: a) if cols is None else (lambda a: a[cols])
    sel_x = (lambda a: a) if xrows is None else (lambda a: a[xrows])
    assert_rel(sel_w(out["dW_ref"]), ref["dW_ref"], TOL, "dW_ref")
    assert_rel(sel_g(out["dgain_ref"]), ref["dgamma_ref"], TOL, "dgain_ref")
    assert_rel(sel_x(out["dX_ref"]), ref["dX_ref"], TOL, "dX_ref")
    if out["Y"] is not None and xrows is not None:
        assert_rel(to_np(out["Y"])[xrows], ref["Y"][xrows], TOL, "Y")
    elif out["Y"] is not None:
        assert_rel(out["Y"], ref["Y"], TOL, "Y")
    for i, code in enumerate(policies):
        for name, sel, shape in (("dgain", sel_g, None), ("dW", sel_w, (d, n)), ("dX", sel_x, (-1, d))):
            est = out[name]
            m = to_np(est["mean"][i])
            b = to_np(est["bias"][i])
            if shape is not None:
                m, b = m.reshape(shape), b.reshape(shape)
            om, ob, ose = ref[code]["dgamma" if name == "dgain" else name]
            assert_rel(sel(m), om, TOL, f"{code} {name} mean")
            if not assert_zero_where_oracle_zero(sel(b), ob, f"{code} {name} bias"):
                assert_rel(sel(b), ob, TOL, f"{code} {name} bias")
            if est["se"] is not None:
                s = to_np(est["se"][i])
                s = s.reshape(shape) if shape is not None else s
                if not assert_zero_where_oracle_zero(sel(s), ose, f"{code} {name} se"):
                    assert_rel(sel(s), ose, TOL, f"{code} {name} se")


ALL = ("U/R", "U/U", "R/R", "N/N", "R/N", "N/R", "U/N", "R/U")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("fwd_mode", ["rne", "sr"])
def test_ragged_all_policies(lib, dtype, fwd_mode):
    T, d, n = 300, 192, 136          # several tiles, ragged against 128 / 64 / 32
    out, ref = run_both(lib, T, d, n, dtype, 16, ALL, fwd_mode=fwd_mode, seed=7)
    compare(out, ref, ALL, d=d, n=n)


def test_shared_new_rounding_and_norm_input_R(lib):
    T, d, n = 130, 64, 72
    pols = ("N/N", "U/N", "R/R")
    out, ref = run_both(lib, T, d, n, torch.bfloat16, 12, pols, seed=9, shared=True, norm_input="R")
    compare(out, ref, pols, d=d, n=n)


def test_k_above_256_uses_two_term_residual(lib):
    T, d, n = 96, 64, 64
    pols = ("N/N",)
    out, ref = run_both(lib, T, d, n, torch.bfloat16, 300, pols, seed=10)
    compare(out, ref, pols, d=d, n=n)


def test_single_row_and_single_trial(lib):
    pols = ("U/U", "R/R", "N/N")
    out, ref = run_both(lib, 1, 64, 64, torch.float32, 1, pols, seed=11)
    compare(out, ref, pols, d=64, n=64)


def test_config1_exact(lib):
    cfg = synth.WORKLOADS["rmsnorm_linear_256x64x64"]
    out, ref = run_both(lib, cfg["T"], cfg["d"], cfg["n"], cfg["dtype"], cfg["K"], cfg["policies"],
                        seed=cfg["seed"], stream=1)
    compare(out, ref, cfg["policies"], d=cfg["d"], n=cfg["n"])


@pytest.mark.slow
def test_config2_full_size_sampled(lib):
    cfg = synth.WORKLOADS["rmsnorm_linear_390m_mlp_up"]
    T, d, n = cfg["T"], cfg["d"], cfg["n"]
    rng = np.random.default_rng(2)
    rows = np.sort(rng.choice(d, 4, replace=False))
    cols = np.sort(rng.choice(d, 6, replace=False))
    xrows = np.sort(rng.choice(T, 16, replace=False))
    out, ref = run_both(lib, T, d, n, cfg["dtype"], cfg["K"], cfg["policies"], seed=cfg["seed"],
                        oracle_kw=dict(dw_rows=rows, gain_cols=cols, dx_rows=xrows), stream=2)
    compare(out, ref, cfg["policies"], rows=rows, cols=cols, xrows=xrows, d=d, n=n)


def test_weight_use_se_per_trial(lib):
    """se of dW where the weight use reads a new rounding: the K per-trial contractions (trial
    batches of 8 and a ragged last batch) against the oracle's sample SD over its K passes."""
    for (T, d, n, K, shared) in ((300, 192, 136, 12, False), (130, 64, 72, 9, True)):
        X, g, W, dY = synth.rmsnorm_linear_inputs(T, d, n, torch.bfloat16, 2)
        pols = ("N/N", "U/N", "R/R", "U/U")
        codes = [p + (":shared" if shared else "") for p in pols]
        print(f"[norm_store] dW se per trial T={T} d={d} n={n} K={K} shared={shared}", flush=True)
        out = lib.rmsnorm_linear(X.cuda(), g.cuda(), W.cuda(), dY.cuda(), policies=codes, K=K, seed=31,
                                 want_dw_se=True)
        torch.cuda.synchronize()
        ref = norm_store.check(X.float().numpy(), g.numpy(), W.float().numpy(), dY.float().numpy(), eps=1e-5,
                               fmt=fp8.E4M3, fwd_mode=oq.RNE, policies=pols, K=K, seed=31, fresh_shared=shared)
        assert out["dW"]["se"] is not None
        compare(out, ref, pols, d=d, n=n)


def test_forward_only_and_no_tokens(lib):
    """dY NULL: the store and Y only (against the oracle); T = 0 with a non-NULL dY: references
    and estimates are zero, the store reports amax 0 and scale 1."""
    X, g, W, dY = synth.rmsnorm_linear_inputs(40, 32, 16, torch.bfloat16, stream=41)
    print("[norm_store] forward only T=40 d=32 n=16", flush=True)
    out = lib.rmsnorm_linear(X.cuda(), g.cuda(), W.cuda(), None, K=4, seed=2)
    torch.cuda.synchronize()
    ref = norm_store.check(X.float().numpy(), g.numpy(), W.float().numpy(), dY.float().numpy(), fmt=fp8.E4M3,
                           fwd_mode=oq.RNE, policies=("U/U",), K=4, seed=2)
    assert np.array_equal(out["u_codes"].cpu().numpy(), ref["codes"])
    assert float(out["u_scale"].cpu()[0]) == float(ref["scale"])
    assert_rel(out["Y"], ref["Y"], TOL, "Y")
    print("[norm_store] no tokens T=0 d=32 n=16", flush=True)
    X0 = torch.empty(0, 32, dtype=torch.bfloat16, device="cuda")
    # torch gives an empty tensor a NULL pointer, which asks for the forward only: a one-row
    # gradient supplies a valid pointer, of which T = 0 rows are read
    dY0 = torch.zeros(1, 16, dtype=torch.bfloat16, device="cuda")
    out = lib.rmsnorm_linear(X0, g.cuda(), W.cuda(), dY0, K=4, seed=2)
    torch.cuda.synchronize()
    d = lib.diag_dict(out["diag"])
    assert d["amax"] == 0.0 and d["scale"] == 1.0 and d["nonfinite"] == 0
    for name in ("dgain_ref", "dW_ref"):
        assert not torch.any(out[name] != 0), name
    for name in ("dgain", "dW"):
        assert not torch.any(out[name]["mean"] != 0) and not torch.any(out[name]["bias"] != 0), name
