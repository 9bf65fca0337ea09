"""GPU parity: bs_rmsnorm_linear_grid_fwd_bwd against the oracle (oracle/grid_store.py).

The grid codes and per-token steps bit for bit; Y, the reference gradients and every policy's
mean and bias of dgain and dW within 1e-5 normwise relative error; exact zeros where the
oracle's bias is zero in every draw (U at the gain use, R at the weight use).
"""
import numpy as np
import pytest
import torch

from oracle import grid_store as gs
from paper_2609_39813_amd import synth
from tests.parity import assert_rel, assert_zero_where_oracle_zero, to_np

pytestmark = pytest.mark.gpu
TOL = 1e-5


def run_both(lib, T, d, n, dtype, K, bits, policies=gs.POLICIES, seed=11, stream=7, zero_row=None):
    X, g, W, dY = synth.rmsnorm_linear_inputs(T, d, n, dtype, stream)
    if zero_row is not None:
        X[zero_row] = 0
    print(f"[grid_store] T={T} d={d} n={n} {dtype} bits={bits} K={K} {policies}", flush=True)
    out = lib.rmsnorm_linear_grid(X.cuda(), g.cuda(), W.cuda(), dY.cuda(), bits=bits, policies=policies, K=K,
                                  seed=seed, store_id=3)
    torch.cuda.synchronize()
    ref = gs.check(X.float().numpy(), g.numpy(), W.float().numpy(), dY.float().numpy(), bits=bits,
                   policies=tuple(dict.fromkeys(policies)), K=K, seed=seed, store_id=3)
    return out, ref


def compare(lib, out, ref, policies, d, n):
    assert np.array_equal(out["u_codes"].cpu().numpy().astype(np.int32), ref["codes"])
    assert np.array_equal(out["u_step"].cpu().numpy(), ref["step"])
    assert_rel(out["Y"], ref["Y"], TOL, "Y")
    assert_rel(out["dW_ref"], ref["dW_ref"], TOL, "dW_ref")
    assert_rel(out["dgain_ref"], ref["dgamma_ref"], TOL, "dgain_ref")
    assert_rel(out["dX_ref"], ref["dX_ref"], TOL, "dX_ref")
    assert lib.diag_dict(out["diag"])["n_saturated"] == ref["n_saturated"]
    for i, code in enumerate(policies):
        for name, shape in (("dgain", None), ("dW", (d, n))):
            m, b = to_np(out[name]["mean"][i]), to_np(out[name]["bias"][i])
            if shape:
                m, b = m.reshape(shape), b.reshape(shape)
            om, ob, _ = ref[code]["dgamma" if name == "dgain" else name]
            assert_rel(m, om, TOL, f"{code} {name} mean")
            if not assert_zero_where_oracle_zero(b, ob, f"{code} {name} bias"):
                assert_rel(b, ob, TOL, f"{code} {name} bias")


@pytest.mark.parametrize("bits", [6, 5])
def test_table_policies_fp32(lib, bits):
    out, ref = run_both(lib, 256, 64, 64, torch.float32, 32, bits)
    compare(lib, out, ref, gs.POLICIES, 64, 64)


def test_bf16_ragged_tokens_and_a_zero_row(lib):
    out, ref = run_both(lib, 200, 96, 40, torch.bfloat16, 16, 6, zero_row=7)
    compare(lib, out, ref, gs.POLICIES, 96, 40)
    assert float(out["u_step"][7].cpu()) == 1.0 and not torch.any(out["u_codes"][7] != 0)


@pytest.mark.parametrize("bits", [2, 8])
def test_grid_widths_and_policy_order(lib, bits):
    pols = ("N/N", "U/R+e", "U/R", "N/N", "R/N")
    out, ref = run_both(lib, 70, 32, 16, torch.float32, 5, bits, policies=pols)
    compare(lib, out, ref, pols, 32, 16)
    assert torch.equal(out["dW"]["mean"][0], out["dW"]["mean"][3])


@pytest.mark.slow
def test_full_size_sampled_entries(lib):
    """X [8192, 1024] bf16, W [1024, 4096], K = 256 (the benchmark's launch): every code and step,
    dW on 2 x 64 sampled entries and dgain on 16 sampled entries."""
    T, d, n, K = 8192, 1024, 4096, 256
    X, g, W, dY = synth.rmsnorm_linear_inputs(T, d, n, torch.bfloat16, 8)
    print(f"[grid_store] full size T={T} d={d} n={n} K={K}", flush=True)
    out = lib.rmsnorm_linear_grid(X.cuda(), g.cuda(), W.cuda(), dY.cuda(), bits=6, K=K, seed=21, store_id=3)
    torch.cuda.synchronize()
    rng = np.random.default_rng(4)
    rows, cols, gcols = rng.choice(d, 2, replace=False), rng.choice(n, 64, replace=False), rng.choice(d, 16, replace=False)
    ref = gs.check(X.float().numpy(), g.numpy(), W.float().numpy(), dY.float().numpy(), bits=6, K=K, seed=21,
                   store_id=3, dw_rows=rows, dw_cols=cols, gain_cols=gcols, full=False)
    assert np.array_equal(out["u_codes"].cpu().numpy().astype(np.int32), ref["codes"])
    assert np.array_equal(out["u_step"].cpu().numpy(), ref["step"])
    pick_w = lambda a: to_np(a).reshape(d, n)[np.ix_(rows, cols)]
    assert_rel(pick_w(out["dW_ref"]), ref["dW_ref"], TOL, "dW_ref")
    assert_rel(to_np(out["dgain_ref"])[gcols], ref["dgamma_ref"], TOL, "dgain_ref")
    for i, code in enumerate(gs.POLICIES):
        om, ob, _ = ref[code]["dW"]
        assert_rel(pick_w(out["dW"]["mean"][i]), om, TOL, f"{code} dW mean")
        if not assert_zero_where_oracle_zero(pick_w(out["dW"]["bias"][i]), ob, f"{code} dW bias"):
            assert_rel(pick_w(out["dW"]["bias"][i]), ob, TOL, f"{code} dW bias")
        om, ob, _ = ref[code]["dgamma"]
        assert_rel(to_np(out["dgain"]["mean"][i])[gcols], om, TOL, f"{code} dgain mean")
        if not assert_zero_where_oracle_zero(to_np(out["dgain"]["bias"][i])[gcols], ob, f"{code} dgain bias"):
            assert_rel(to_np(out["dgain"]["bias"][i])[gcols], ob, TOL, f"{code} dgain bias")
