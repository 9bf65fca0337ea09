"""Planted errors on the GPU: a call made with a wrong argument (a Philox key, a use id, a policy
letter at one use, the copy D reads) must fail parity against the oracle computed with the right
one, while the same call with the right argument passes. The SR threshold, which no argument
changes, is planted on the CPU in the oracle: the GPU's codes at the 2^32 boundary must then
disagree with it."""
import numpy as np
import pytest
import torch

from oracle import attention, fp8, norm_store, philox, qround as oq
from paper_2609_39813_amd import synth
from tests.parity import parity_ok, to_np

pytestmark = pytest.mark.gpu
TOL = 1e-5


def test_wrong_philox_key_or_use_changes_the_codes(lib):
    g = torch.Generator().manual_seed(3)
    x = torch.randn(65536, generator=g) * 2
    ref = oq.qround(x.numpy(), fp8.E4M3, oq.SR, 0xB5F1, 2, 513)
    print("[mutant] qround seed / use", flush=True)
    for seed, use, right in ((0xB5F1, 513, True), (0xB5F1 ^ (1 << 32), 513, False), (0xB5F1, 514, False)):
        codes, _, _ = lib.qround(x.cuda(), "e4m3", "sr", seed, 2, use)
        torch.cuda.synchronize()
        same = np.array_equal(codes.cpu().numpy(), ref.codes)
        assert same == right, (hex(seed), use)


def _norm(lib, policies_gpu, store_id_gpu, policies_ref=None):
    T, d, n, K, seed = 160, 64, 72, 8, 31
    X, g, W, dY = synth.rmsnorm_linear_inputs(T, d, n, torch.float32, 2)
    print(f"[mutant] norm store gpu={policies_gpu} store={store_id_gpu}", flush=True)
    out = lib.rmsnorm_linear(X.cuda(), g.cuda(), W.cuda(), dY.cuda(), policies=policies_gpu, K=K, seed=seed,
                             store_id=store_id_gpu)
    torch.cuda.synchronize()
    ref = norm_store.check(X.numpy(), g.numpy(), W.numpy(), dY.numpy(), policies=policies_ref or policies_gpu, K=K,
                           seed=seed, store_id=0)
    return out, ref


def test_weight_use_reading_the_wrong_value_fails(lib):
    out, ref = _norm(lib, ("U/U",), 0)
    assert parity_ok(out["dW"]["bias"][0].reshape(64, 72), ref["U/U"]["dW"][1], TOL)
    out, ref = _norm(lib, ("U/R",), 0, policies_ref=("U/U",))          # R read where U is asked
    assert not parity_ok(out["dW"]["bias"][0].reshape(64, 72), ref["U/U"]["dW"][1], TOL)


def test_new_roundings_under_the_wrong_use_id_fail(lib):
    out, ref = _norm(lib, ("N/N",), 0)
    assert parity_ok(out["dW"]["bias"][0].reshape(64, 72), ref["N/N"]["dW"][1], TOL)
    out, ref = _norm(lib, ("N/N",), 1)                                   # use ids 256 + j for 0 + j
    assert not parity_ok(out["dW"]["bias"][0].reshape(64, 72), ref["N/N"]["dW"][1], TOL)


def test_d_from_the_wrong_copy_fails(lib):
    Q, K, V, dO = (t.to(torch.bfloat16) for t in synth.attention_inputs(1, 2, 96, 64, torch.float32, stream=140))
    ref = attention.check(*(t.float().numpy() for t in (Q, K, V, dO)), policies=("U", "R"), K=2, seed=9, store_id=1)
    O = torch.from_numpy(np.ascontiguousarray(ref["O32"])).cuda()
    print("[mutant] attention D copy", flush=True)
    for gpu_pol, want in (("R", True), ("U", False)):                 # U reads O where R's copy is asked
        out = lib.attn_bwd_policy(Q.cuda(), K.cuda(), V.cuda(), dO.cuda(), causal=True, O=O, policies=(gpu_pol,),
                                  K=2, seed=9, store_id=1)
        torch.cuda.synchronize()
        got = to_np(out["dQ"]["bias"][0]).reshape(2, 96, 64)
        assert parity_ok(got, ref["R"]["dQ"][1], TOL) == want, gpu_pol


def test_sr_threshold_off_by_one_in_the_oracle_disagrees_with_the_gpu(lib):
    """Normal magnitudes placed so that R + F = 2^32 exactly for each element's word: the GPU rounds
    them up, as the oracle does; an oracle planted to round up only above 2^32 disagrees."""
    seed, trial, use, n = 0xB5FB, 4, 9, 1 << 16
    f = fp8.E4M3
    R = philox.words(seed, trial, use, np.arange(n, dtype=np.uint64)).astype(np.int64)
    w = 23 - f.mbits
    D = -((R - (1 << 32)) // (1 << (32 - w)))        # smallest fraction that rounds up
    keep = (D < (1 << w)) & ((((1 << 32) - R) % (1 << (32 - w))) == 0)
    x = np.ldexp(((1 << w) * (1 << f.mbits) + D).astype(np.float64), -23).astype(np.float32)
    x[~keep] = 1.0
    codes, _, _ = lib.qround(torch.from_numpy(x).cuda(), "e4m3", "sr", seed, trial, use, torch.ones(1).cuda())
    torch.cuda.synchronize()
    codes = codes.cpu().numpy()
    ref, _ = oq.round_scaled(x, f, oq.SR, seed, trial, use)
    assert np.array_equal(codes, ref)
    F, lo, step = fp8.sr_threshold(np.abs(x).astype(np.float64), f)
    planted = fp8.encode(np.where((R.astype(np.uint64) + F > np.uint64(1 << 32)) & (F > 0), lo + step, lo),
                         np.signbit(x), f)
    assert keep.sum() > 0 and not np.array_equal(codes, planted)
