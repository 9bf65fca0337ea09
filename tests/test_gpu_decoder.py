"""GPU parity: bs_decoder_layer_policy against the oracle (oracle/decoder.py).

The oracle's realized forward (Q, K, V, O, h, [g | hh], a) is handed to the library, so all four
FP8 stores are compared bit for bit, and the reference gradients and the per-use table within
the fp32 tolerance. The table holds sums of squares: a vector within normwise relative error e
has a sum of squares within 2e + e^2 of the oracle's, hence TOL2 below. Where the oracle's bias
is exactly zero (the letter that reads what its use needs) the library's must be exactly zero.
The library's own forward is checked separately: the first store (which depends on x only) bit
for bit, the others as valid roundings of nearly equal inputs.
"""
import numpy as np
import pytest
import torch

from oracle import decoder, fp8, qround as oq
from paper_2609_39813_amd import synth
from tests.parity import assert_rel, to_np

pytestmark = pytest.mark.gpu
TOL = 1e-5
TOL2 = 2 * TOL + TOL * TOL
FMTS = {"e4m3": fp8.E4M3, "e5m2": fp8.E5M2}
MODES = {"rne": oq.RNE, "sr": oq.SR}


def oracle_case(B, S, d, H, F, K, seed, fmt, mode, stream):
    (x, p, dOut), _ = synth.decoder_inputs(B, S, d, H, F, stream=stream)
    pn = {k: v.float().numpy() for k, v in p.items()}
    f = decoder.forward(x.float().numpy(), pn, B=B, S=S, H=H, fmt=FMTS[fmt], fwd_mode=MODES[mode], seed=seed)
    r = decoder.reference_backward(f, pn, dOut.float().numpy())
    t = decoder.per_use_table(f, pn, r, K=K, seed=seed, fmt=FMTS[fmt])
    return (x, p, dOut), f, r, t


def fixed_of(f):
    cu = lambda a, dt=torch.float32: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dt).cuda()
    return {"Q": cu(f["Q"], torch.bfloat16), "K": cu(f["K"], torch.bfloat16), "V": cu(f["V"], torch.bfloat16),
            "O": cu(f["O"]), "h": cu(f["h"]), "gh": cu(np.concatenate([f["g"], f["hh"]], axis=1)), "a": cu(f["a"])}


def run(lib, inputs, B, S, H, K, seed, fmt, mode, fixed, per_use_se=False):
    x, p, dOut = inputs
    print(f"[layer] B={B} S={S} d={x.shape[1]} H={H} F={p['Wg'].shape[1]} K={K} fmt={fmt} mode={mode} "
          f"fixed={fixed is not None} per_use_se={per_use_se}", flush=True)
    out = lib.decoder_layer_policy(x.cuda(), {k: v.cuda() for k, v in p.items()}, dOut.cuda(), B=B, S=S, H=H,
                                   fmt=fmt, fwd_mode=mode, K=K, seed=seed, fixed=fixed, per_use_se=per_use_se)
    torch.cuda.synchronize()
    return out


def check_sumsq(got, want, what):
    if want == 0.0:
        assert got == 0.0, (what, got)
    else:
        assert abs(got - want) <= TOL2 * want, (what, got, want, abs(got - want) / want)


@pytest.mark.parametrize("B,S,d,H,F,K,seed,fmt,mode,per_use_se", [
    (2, 40, 128, 2, 256, 8, 11, "e4m3", "rne", False),   # T = 80: one full and one ragged 64-row tile
    (1, 72, 64, 1, 136, 5, 12, "e5m2", "sr", False),     # F = 136: ragged GEMM columns
    (2, 40, 128, 2, 256, 11, 13, "e4m3", "rne", True),   # the per-use se (K = 11: a partial trial batch)
    (1, 72, 64, 1, 136, 1, 14, "e5m2", "sr", True),      # K = 1: se 0
])
def test_layer_matches_oracle_with_fixed_forward(lib, B, S, d, H, F, K, seed, fmt, mode, per_use_se):
    inputs, f, r, table = oracle_case(B, S, d, H, F, K, seed, fmt, mode, stream=600 + seed)
    out = run(lib, inputs, B, S, H, K, seed, fmt, mode, fixed_of(f), per_use_se)
    # the four stores, bit for bit
    for name, q in (("u1", f["q1"]), ("O", f["qO"]), ("u2", f["q2"]), ("a", f["qa"])):
        codes = to_np(out["codes_" + name])
        assert np.array_equal(codes.reshape(q.codes.shape), q.codes), name
    assert np.array_equal(to_np(out["scales"]), np.array([f[k].scale for k in ("q1", "qO", "q2", "qa")], np.float32))
    # reference gradients
    for name in ("dx", "dgain1", "dWqkv", "dWo", "dgain2", "dWg", "dWu", "dWd"):
        assert_rel(to_np(out[name]), r[name], TOL, name)
    # per-use table
    got = lib.layer_table(out["table_raw"])
    for key, (m, b, s, ref) in table.items():
        b2, r2, s2 = got[key]
        check_sumsq(b2, float(np.sum(np.asarray(b, np.float64) ** 2)), key + ("bias^2",))
        check_sumsq(r2, float(np.sum(np.asarray(ref, np.float64) ** 2)), key + ("ref^2",))
        if not np.isnan(s2):
            check_sumsq(s2, float(np.sum(np.asarray(s, np.float64) ** 2)), key + ("se^2",))
    # rows without an estimate in the library are NaN; every other row is present
    for key, (b2, r2, s2) in got.items():
        if key in table:
            assert not np.isnan(b2) and not np.isnan(r2), key
        else:
            assert key[1] == "norm_input" and key[3] == "N" and np.isnan(b2), key
        if np.isnan(s2):
            if per_use_se:
                assert key[3] == "N" and key[1] == "norm_input", key
            else:
                assert key[3] == "N" and (key[1] in ("weight", "norm_input") or key[2] == "dK"), key
    if per_use_se:  # every N row but the normalization inputs has its se
        for key in table:
            if key[3] == "N":
                assert not np.isnan(got[key][2]), key


def test_layer_own_forward_is_a_valid_realization(lib):
    B, S, d, H, F, K, seed = 2, 40, 128, 2, 256, 4, 21
    inputs, f, r, _ = oracle_case(B, S, d, H, F, K, seed, "e4m3", "rne", stream=621)
    out = run(lib, inputs, B, S, H, K, seed, "e4m3", "rne", None)
    assert np.array_equal(to_np(out["codes_u1"]), f["q1"].codes)
    scales = to_np(out["scales"])
    for i, name in enumerate(("u1", "O", "u2", "a")):
        q = f[("q1", "qO", "q2", "qa")[i]]
        assert abs(scales[i] - q.scale) <= 1e-5 * q.scale, name
        codes = to_np(out["codes_" + name]).reshape(q.codes.shape).astype(np.int64)
        # sign-magnitude codes of nearly equal inputs: equal, or one step apart in magnitude
        mag = lambda c: np.where(c >= 128, -(c - 128), c)
        diff = np.abs(mag(codes) - mag(q.codes.astype(np.int64)))
        zero_flip = (codes & 127) + (q.codes.astype(np.int64) & 127) <= 1
        assert np.all((diff <= 1) | zero_flip), name
        assert np.mean(diff != 0) < 1e-2, name
    for name in ("dx", "dWqkv", "dWo", "dWd"):
        assert_rel(to_np(out[name]), r[name], 2e-2, name)
