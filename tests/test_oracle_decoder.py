"""Pins of the decoder-layer oracle (oracle/decoder.py)."""
import numpy as np
import torch

from oracle import decoder, fp8, qround
from paper_2609_39813_amd import synth


def small(seed=0, B=2, S=24, d=128, H=2, F=256):
    return synth.decoder_inputs(B, S, d, H, F, config=500 + seed)


def test_reference_backward_matches_autograd():
    (x, p, dOut), (B, S, H) = small()
    f = decoder.forward(x.float().numpy(), {k: v.float().numpy() for k, v in p.items()}, B=B, S=S, H=H, seed=3)
    pn = {k: v.float().numpy() for k, v in p.items()}
    r = decoder.reference_backward(f, pn, dOut.float().numpy())
    t = lambda a: torch.tensor(np.asarray(a, np.float64), requires_grad=True)
    X = t(x.float().numpy())
    P = {k: t(v) for k, v in pn.items()}
    ste = lambda v, target: v + (torch.tensor(np.asarray(target, np.float64)) - v).detach()

    def rms(v, g):
        return g * (v * ((v * v).mean(-1, keepdim=True) + 1e-5).rsqrt())
    T, d = X.shape
    u1 = ste(rms(X, P["gain1"]), f["u1q"])
    qkv = ste(u1 @ P["Wqkv"], f["QKV"])
    hs = lambda m: m.reshape(B, S, H, d // H).permute(0, 2, 1, 3)
    Q, K, V = (ste(hs(qkv[:, i * d:(i + 1) * d]), f[n]) for i, n in enumerate("QKV"))
    sc = f["c"] * Q @ K.transpose(-1, -2)
    mask = torch.tril(torch.ones(S, S, dtype=torch.bool))
    O = torch.softmax(sc.masked_fill(~mask, float("-inf")), -1) @ V
    O = ste(ste(O, f["O"]), f["Oq"])
    Ot = O.permute(0, 2, 1, 3).reshape(T, d)
    h = ste(X + Ot @ P["Wo"], f["h"])
    u2 = ste(rms(h, P["gain2"]), f["u2q"])
    g = ste(u2 @ P["Wg"], f["g"])
    hh = ste(u2 @ P["Wu"], f["hh"])
    a = ste(ste(torch.nn.functional.silu(g) * hh, f["a"]), f["aq"])
    out = h + a @ P["Wd"]
    (out * torch.tensor(dOut.double().numpy())).sum().backward()
    rel = lambda a, b: np.linalg.norm(np.asarray(a) - b.detach().numpy()) / np.linalg.norm(b.detach().numpy())
    for name, grad in (("dx", X.grad), ("dgain1", P["gain1"].grad), ("dWqkv", P["Wqkv"].grad), ("dWo", P["Wo"].grad),
                       ("dgain2", P["gain2"].grad), ("dWg", P["Wg"].grad), ("dWu", P["Wu"].grad),
                       ("dWd", P["Wd"].grad)):
        assert rel(r[name], grad) < 2e-6, (name, rel(r[name], grad))


def test_per_use_reference_letters_are_exact_zeros_and_weight_closed_form():
    (x, p, dOut), (B, S, H) = small(seed=1, S=16)
    pn = {k: v.float().numpy() for k, v in p.items()}
    f = decoder.forward(x.float().numpy(), pn, B=B, S=S, H=H, seed=5)
    r = decoder.reference_backward(f, pn, dOut.float().numpy())
    t = decoder.per_use_table(f, pn, r, K=4, seed=5)
    need_original = {("u1", "gain"), ("u2", "gain"), ("u1", "norm_input"), ("u2", "norm_input"), ("O", "D")}
    for (store, use, grad, letter), (m, b, s, ref) in t.items():
        ref_letter = "U" if (store, use) in need_original else "R"
        if letter == ref_letter:
            assert np.all(b == 0), (store, use, grad, letter)
            assert np.allclose(m, ref, rtol=0, atol=0), (store, use, grad)
    # weight use of a: U adds (a - deq(C_a))^T dOut exactly
    m, b, s, ref = t[("a", "weight", "dW", "U")]
    want = (f["a"].astype(np.float64) - f["aq"]).T @ r["dOut"]
    assert np.allclose(b, want, rtol=1e-10, atol=1e-14)
    rows = decoder.table(t)
    assert rows[("a", "weight", "dW", "R")]["rel_bias"] == 0.0
    assert rows[("O", "D", "dQ", "R")]["rel_bias"] > 0.0
