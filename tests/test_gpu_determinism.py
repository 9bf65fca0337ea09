"""Every call returns the same bits for the same inputs and seed (the C-ABI's determinism claim):
each entry point runs twice on one stream and every output tensor is compared bit for bit."""
import pytest
import torch

from paper_2609_39813_amd import synth

pytestmark = pytest.mark.gpu


def tensors(x):
    """Every tensor in a (possibly nested) output structure, in a fixed order."""
    if isinstance(x, torch.Tensor):
        yield x
    elif isinstance(x, dict):
        for k in sorted(x):
            yield from tensors(x[k])
    elif isinstance(x, (list, tuple)):
        for v in x:
            yield from tensors(v)


def same_bits(a, b, what):
    ta, tb = list(tensors(a)), list(tensors(b))
    assert len(ta) == len(tb) and ta, what
    for i, (u, v) in enumerate(zip(ta, tb)):
        assert u.shape == v.shape and torch.equal(u.view(torch.uint8) if u.dtype != torch.uint8 else u,
                                                  v.view(torch.uint8) if v.dtype != torch.uint8 else v), (what, i)


def twice(fn, what):
    print(f"[determinism] {what}", flush=True)
    a = fn()
    torch.cuda.synchronize()
    b = fn()
    torch.cuda.synchronize()
    same_bits(a, b, what)


def test_rmsnorm_linear_and_grid_store(lib):
    X, g, W, dY = (t.cuda() for t in synth.rmsnorm_linear_inputs(200, 96, 40, torch.bfloat16, stream=51))
    twice(lambda: lib.rmsnorm_linear(X, g, W, dY, K=24, seed=5, want_dw_se=True), "rmsnorm_linear")
    twice(lambda: lib.rmsnorm_linear_grid(X, g, W, dY, bits=6, K=24, seed=5), "rmsnorm_linear_grid")


def test_attention_paths(lib):
    Q, K, V, dO = (t.cuda() for t in synth.attention_inputs(1, 2, 136, 64, torch.bfloat16, stream=52))
    twice(lambda: lib.attn_bwd_policy(Q, K, V, dO, policies=("U", "R", "N"), K=8, seed=3), "attn_bwd_policy")
    twice(lambda: lib.attn_level2_policy(Q, K, V, dO, K=8, seed=3), "attn_level2_policy")
    twice(lambda: lib.attn_pstore_policy(Q, K, V, dO, K=8, seed=3, want_p=True), "attn_pstore_policy")
    O = torch.randn(1, 2, 136, 64, device="cuda") * 0.3
    codes, s, _ = lib.qround(O, fmt="e4m3", mode="sr", seed=4)
    sc = torch.tensor([1 / 448, 1e-4, 5e-5, 5e-5], device="cuda")
    twice(lambda: lib.te_attn_bwd(Q, K, V, dO, sc, O=O, O_codes=codes, O_scale=s, source="repair",
                                  want_ds=True, want_pre=True), "te_attn_bwd")


def test_linear_and_logsoftmax(lib):
    X, W, dY, _, _ = synth.linear_bwd_inputs(192, 64, 96, torch.bfloat16, 53)
    X, W, dY = X.cuda(), W.cuda(), dY.cuda()
    pa, pb = torch.randn(192, 64, device="cuda"), torch.randn(64, 96, device="cuda")
    twice(lambda: lib.linear_bwd_policy(X, W, dY, K=16, seed=6, probeA=pa, probeB=pb), "linear_bwd_policy")
    gz = torch.Generator().manual_seed(54)
    z = (torch.randn(9, 132, generator=gz, dtype=torch.float64) * 2).cuda()
    y = torch.randint(0, 132, (9,), generator=gz, dtype=torch.int32).cuda()
    twice(lambda: lib.logsoftmax_reuse_check(z, y, eps=0.1, K=300, seed=7), "logsoftmax_reuse_check")
