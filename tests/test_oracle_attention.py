"""Pins of the attention oracle (oracle/attention.py)."""
import numpy as np
import pytest
import torch

from oracle import attention, fp8, policy, qround
from tests import attn_example


def make(B, H, S, dh, seed=0):
    rng = np.random.default_rng(seed)
    return [rng.normal(size=(B, H, S, dh)).astype(np.float32) for _ in range(4)]


def test_reference_matches_autograd():
    Q, K, V, dO = make(1, 2, 37, 16)
    out = attention.check(Q, K, V, dO, policies=(), K=1, seed=1)
    q, k, v = (torch.tensor(a, dtype=torch.float64, requires_grad=True) for a in (Q, K, V))
    c = 1 / 4.0
    s = c * q @ k.transpose(-1, -2)
    mask = torch.tril(torch.ones(37, 37, dtype=torch.bool))
    o = torch.softmax(s.masked_fill(~mask, float("-inf")), -1) @ v
    oq = torch.tensor(qround.dequant(out["codes"], out["scale"], fp8.E4M3))
    stored = o + (oq - o).detach()
    (stored * torch.tensor(dO, dtype=torch.float64)).sum().backward()
    rel = lambda a, b: np.linalg.norm(a - b) / np.linalg.norm(b)
    assert rel(out["dV_ref"], v.grad.numpy()[0]) < 1e-12
    assert rel(out["dQ_ref"], q.grad.numpy()[0]) < 1e-6
    assert rel(out["dK_ref"], k.grad.numpy()[0]) < 1e-6
    assert rel(out["O"], o.detach().numpy()) < 1e-12


def test_d_from_output_equals_rowsum_p_dp():
    Q, K, V, dO = make(1, 1, 29, 8, seed=2)
    O, P, _, _ = attention.forward(Q, K, V, True, 0.3)
    dP = dO.astype(np.float64) @ np.swapaxes(V.astype(np.float64), -1, -2)
    assert np.allclose(attention.d_from_copy(dO, O), (P * dP).sum(-1), rtol=1e-12, atol=1e-12)


def test_fp8_attention_example_cells_exact():
    ex = attn_example.load()
    Q, K, V = attn_example.inputs(ex)
    O, P, _, _ = attention.forward(Q, K, V, True, ex["c"])
    assert O[0, 0, -1, 0] == ex["s"]
    a, c = ex["a"], ex["c"]
    means = {"dev": 0.0, "fix": 0.0}
    for cell in ex["cells"]:
        for key, h in (("T_h_shared_deviation", cell["sigma"] * a), ("T_h_fixed", a)):
            dq = {}
            for which, sign in (("shared", cell["sigma"]), ("indep", cell["tau"])):
                Os, dO = attn_example.saved_and_grad(ex, O, sign, h)
                D = attention.d_from_copy(dO, Os)
                dq[which] = attention.backward(Q, K, V, dO, P, D, c)[0][0, 0, -1, 0]
            T = (dq["indep"] - dq["shared"]) / c
            assert T == cell[key]
            means["dev" if key.endswith("deviation") else "fix"] += T / 4
    assert means["dev"] == ex["predicted_mean_h_shared_deviation"]
    assert means["fix"] == ex["predicted_mean_h_fixed"]


def test_policy_biases_have_row_scaled_form():
    Q, K, V, dO = make(1, 2, 20, 8, seed=3)
    out = attention.check(Q, K, V, dO, policies=("U", "R", "N"), K=8, seed=4)
    Oq = qround.dequant(out["codes"], out["scale"], fp8.E4M3)
    c = 1 / np.sqrt(8)
    _, P, _, _ = attention.forward(Q, K, V, True, c)
    for hh, (b, h) in enumerate(out["heads"]):
        dD = attention.d_from_copy(dO[b, h], Oq[b, h] - out["O32"][b, h].astype(np.float64))
        want_q = -c * dD[:, None] * (P[b, h] @ K[b, h].astype(np.float64))
        want_k = -c * (P[b, h] * dD[:, None]).T @ Q[b, h].astype(np.float64)
        assert np.allclose(out["R"]["dQ"][1][hh], want_q, rtol=1e-9, atol=1e-13)
        assert np.allclose(out["R"]["dK"][1][hh], want_k, rtol=1e-9, atol=1e-13)
    assert np.all(out["U"]["dQ"][1] == 0) and np.all(out["U"]["dK"][1] == 0)


def test_new_rounding_mean_within_band():
    Q, K, V, dO = make(1, 1, 12, 4, seed=5)
    Kt = 3000
    out = attention.check(Q, K, V, dO, policies=("N",), K=Kt, seed=6)
    s = out["scale"]
    y = qround.scaled(out["O32"], s).astype(np.float64)
    # E[new rounding] = s * y exactly for stochastic rounding (no value is clamped here)
    assert out["n_saturated"] == 0 or np.abs(y).max() <= 448.0
    c = 0.5
    _, P, _, _ = attention.forward(Q, K, V, True, c)
    D = attention.d_from_copy(dO[0, 0], s * y[0, 0])
    dq, dk, _ = attention.backward(Q[0, 0], K[0, 0], V[0, 0], dO[0, 0], P[0, 0], D, c)
    mean, _, se = out["N"]["dQ"]
    assert np.all(np.abs(mean[0] - dq) <= 4.5 * se[0] + 1e-12)
    mean, _, se = out["N"]["dK"]
    assert np.all(np.abs(mean[0] - dk) <= 4.5 * se[0] + 1e-12)


def test_planted_d_from_the_wrong_copy_fails_the_pins(monkeypatch):
    """D read from the forward's rounded copy where the original was handed in (the reference's
    D), or the R policy reading the original: the autograd pin, resp. the closed form of R's bias,
    must fail."""
    d_from = attention.d_from_copy

    def rounded_copy(dO, Ohat):
        q = qround.qround(np.asarray(Ohat, np.float32), fp8.E4M3, qround.RNE)
        return d_from(dO, qround.dequant(q.codes, q.scale, fp8.E4M3))
    monkeypatch.setattr(attention, "d_from_copy", rounded_copy)
    with pytest.raises(AssertionError):
        test_reference_matches_autograd()
    monkeypatch.undo()
    read = policy.read
    monkeypatch.setattr(policy, "read", lambda l, o, r, f: read({"R": "U"}.get(l, l), o, r, f))
    with pytest.raises(AssertionError):
        test_policy_biases_have_row_scaled_form()
