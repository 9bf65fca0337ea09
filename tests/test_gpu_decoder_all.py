"""GPU parity: the decoder layer's every-use-at-once check (bs_decoder_layer_policy with `all`)
against oracle.decoder.all_uses: each letter read at every use of every store together, K plain
backward passes in the oracle. The oracle's realized forward is handed to the library. Biases and
se of the eight gradients within 1e-5 (normwise and element-wise), the table's sums of squares
within the implied tolerance, exact zeros where the oracle's bias is zero in every draw."""
import numpy as np
import pytest
import torch

from oracle import decoder
from tests.parity import assert_rel, assert_zero_where_oracle_zero, to_np
from tests.test_gpu_decoder import FMTS, MODES, TOL, TOL2, check_sumsq, fixed_of, oracle_case

pytestmark = pytest.mark.gpu


def run_all(lib, B, S, d, H, F, K, seed, fmt, mode):
    inputs, f, r, _ = oracle_case(B, S, d, H, F, K, seed, fmt, mode, stream=640 + seed)
    x, p, dOut = inputs
    pn = {k: v.float().numpy() for k, v in p.items()}
    print(f"[layer all uses] B={B} S={S} d={d} H={H} F={F} K={K} fmt={fmt} mode={mode}", flush=True)
    out = lib.decoder_layer_policy(x.cuda(), {k: v.cuda() for k, v in p.items()}, dOut.cuda(), B=B, S=S, H=H,
                                   fmt=fmt, fwd_mode=mode, K=K, seed=seed, fixed=fixed_of(f), all_uses=True)
    torch.cuda.synchronize()
    ref = decoder.all_uses(f, pn, dOut.float().numpy(), r, K=K, seed=seed, fmt=FMTS[fmt])
    return out, ref, r


@pytest.mark.parametrize("B,S,d,H,F,K,seed,fmt,mode", [
    (2, 40, 128, 2, 256, 5, 31, "e4m3", "rne"),   # T = 80: a full and a ragged 64-row tile
    (1, 72, 64, 1, 136, 4, 32, "e5m2", "sr"),     # F = 136: ragged contraction columns
    (1, 16, 1088, 17, 128, 2, 34, "e4m3", "sr"),  # d > 1024: u1's gain and norm-input uses in two kernels
])
def test_every_use_at_once_matches_oracle(lib, B, S, d, H, F, K, seed, fmt, mode):
    out, ref, r = run_all(lib, B, S, d, H, F, K, seed, fmt, mode)
    tab = lib.layer_all_table(out["all_table_raw"])
    for l in "URN":
        for g in decoder.GRADS:
            m_o, b_o, se_o = ref[l][g]
            b = to_np(out["all_bias"][l][g]).reshape(b_o.shape)
            if not assert_zero_where_oracle_zero(b, b_o, f"{l} {g} bias"):
                assert_rel(b, b_o, TOL, f"{l} {g} bias")
            se = to_np(out["all_se"][l][g]).reshape(se_o.shape)
            b2, r2, s2 = tab[(g, l)]
            check_sumsq(b2, float(np.sum(b_o ** 2)), (g, l, "bias^2"))
            check_sumsq(r2, float(np.sum(np.asarray(r[g], np.float64) ** 2)), (g, l, "ref^2"))
            if l == "N" and g in ("dWd", "dWg", "dWu"):
                assert np.all(np.isnan(se)) and np.isnan(s2), (g, "se not estimated here")
                continue
            if not assert_zero_where_oracle_zero(se, se_o, f"{l} {g} se"):
                assert_rel(se, se_o, TOL, f"{l} {g} se")
            check_sumsq(s2, float(np.sum(se_o ** 2)), (g, l, "se^2"))
    # the letter that reads what every use needs does not exist: R and U both move some gradient
    for l in "UR":
        assert any(np.any(to_np(out["all_bias"][l][g]) != 0) for g in decoder.GRADS), l


def test_every_use_at_once_leaves_the_per_use_outputs_unchanged(lib):
    """Asking for the every-use check does not change the reference gradients, stores or table."""
    B, S, d, H, F, K, seed = 1, 40, 64, 1, 96, 3, 33
    inputs, f, r, _ = oracle_case(B, S, d, H, F, K, seed, "e4m3", "rne", stream=640 + seed)
    x, p, dOut = inputs
    args = (x.cuda(), {k: v.cuda() for k, v in p.items()}, dOut.cuda())
    kw = dict(B=B, S=S, H=H, fmt="e4m3", fwd_mode="rne", K=K, seed=seed, fixed=fixed_of(f))
    a = lib.decoder_layer_policy(*args, **kw)
    b = lib.decoder_layer_policy(*args, all_uses=True, **kw)
    torch.cuda.synchronize()
    for k in ("dx", "dgain1", "dWqkv", "dWo", "dgain2", "dWg", "dWu", "dWd", "codes_u1", "codes_O", "codes_u2",
              "codes_a", "scales"):
        assert torch.equal(a[k], b[k]), k
    assert np.array_equal(a["table_raw"].cpu().numpy(), b["table_raw"].cpu().numpy(), equal_nan=True)
