"""Pins of the decoder-layer oracle (oracle/decoder.py)."""
import numpy as np
import pytest
import torch

from oracle import decoder, fp8, qround
from paper_2609_39813_amd import synth


def small(seed=0, B=2, S=24, d=128, H=2, F=256):
    return synth.decoder_inputs(B, S, d, H, F, stream=500 + seed)


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


# ---------------------------------------------------------------------------------------------
# The forward itself, pinned stage by stage against an independent torch fp64 program written
# from App. D.1's block (pre-norm RMSNorm, causal multi-head attention, SwiGLU MLP, no biases),
# with torch's own float8 casts (round to nearest even) as the codec of the four stores. Each
# stage is recomputed from the oracle's realized value of the stage before it, so a wrong
# formula anywhere (a swapped weight or gain, a dropped residual, a wrong mask) fails at its own
# stage, while fp32 rounding of the oracle's values stays within FWD_TOL.
# ---------------------------------------------------------------------------------------------
FWD_TOL = 1e-6


def _torch_store(u, fmax=448.0):
    """Per-tensor FP8 E4M3 store by torch's cast: s = fl32(amax / FMAX), y = fl32(u / s) clamped
    to +-FMAX, code = RNE cast; returns (code bytes, dequantized fp64 values, s)."""
    u32 = torch.as_tensor(np.asarray(u, np.float32))
    amax = u32.abs().max()
    s = (amax / torch.tensor(fmax, dtype=torch.float32)) if float(amax) > 0 else torch.tensor(1.0)
    y = (u32 / s).clamp(-fmax, fmax)
    c8 = y.to(torch.float8_e4m3fn)
    return c8.view(torch.uint8).numpy(), c8.to(torch.float64) * float(s), np.float32(s)


def forward_stage_errors(f, x, p, B, S, H, eps=1e-5):
    """{stage: relative error or code mismatch count} of the oracle's realized forward f."""
    T, d = x.shape
    dh = d // H
    t64 = lambda a: torch.as_tensor(np.asarray(a, np.float32)).to(torch.float64)
    W = {k: t64(p[k]) for k in ("Wqkv", "Wo", "Wg", "Wu", "Wd")}
    g1, g2 = t64(p["gain1"]), t64(p["gain2"])
    rel = lambda got, want: float(torch.linalg.norm(t64(got) - want) / torch.linalg.norm(want))
    rms = lambda v, g: g * v / torch.sqrt((v * v).mean(-1, keepdim=True) + eps)
    hs = lambda m: m.reshape(B, S, H, dh).permute(0, 2, 1, 3)
    err = {}

    def store(name, value, q):
        codes, deq, s = _torch_store(value)
        err[name + "_codes"] = int((codes != q.codes.reshape(codes.shape)).sum())
        err[name + "_scale"] = int(s != q.scale)
        return deq

    err["u1"] = rel(f["u1"], rms(t64(x), g1))
    u1q = store("u1", f["u1"], f["q1"])
    err["QKV"] = rel(f["QKV"], u1q @ W["Wqkv"])
    qkv16 = torch.as_tensor(f["QKV"]).to(torch.bfloat16).to(torch.float64)
    for i, n in enumerate("QKV"):
        err[n] = int((t64(f[n]) != hs(qkv16[:, i * d:(i + 1) * d])).sum())
    Q, K, V = (t64(f[n]) for n in "QKV")
    sc = (Q @ K.transpose(-1, -2)) / np.sqrt(dh)
    sc = sc.masked_fill(~torch.tril(torch.ones(S, S, dtype=torch.bool)), float("-inf"))
    err["O"] = rel(f["O"], torch.softmax(sc, -1) @ V)
    Oq = store("O", f["O"], f["qO"])
    err["h"] = rel(f["h"], t64(x) + Oq.permute(0, 2, 1, 3).reshape(T, d) @ W["Wo"])
    err["u2"] = rel(f["u2"], rms(t64(f["h"]), g2))
    u2q = store("u2", f["u2"], f["q2"])
    err["g"] = rel(f["g"], u2q @ W["Wg"])
    err["hh"] = rel(f["hh"], u2q @ W["Wu"])
    err["a"] = rel(f["a"], torch.nn.functional.silu(t64(f["g"])) * t64(f["hh"]))
    aq = store("a", f["a"], f["qa"])
    err["out"] = rel(f["out"], t64(f["h"]) + aq @ W["Wd"])
    return err


def forward_failures(err):
    return {k: v for k, v in err.items() if (v > FWD_TOL if isinstance(v, float) else v != 0)}


def _pin_case(seed=0):
    (x, p, dOut), (B, S, H) = small(seed=seed)
    pn = {k: v.float().numpy() for k, v in p.items()}
    g = torch.Generator().manual_seed(77 + seed)
    pn["gain1"] = (1 + 0.1 * torch.randn(x.shape[1], generator=g)).numpy()   # distinct gains: a swap shows
    pn["gain2"] = (1 + 0.1 * torch.randn(x.shape[1], generator=g)).numpy()
    return x.float().numpy(), pn, (B, S, H)


@pytest.mark.parametrize("seed", [0, 1])
def test_forward_matches_independent_torch_program(seed):
    x, pn, (B, S, H) = _pin_case(seed)
    f = decoder.forward(x, pn, B=B, S=S, H=H, seed=3)
    err = forward_stage_errors(f, x, pn, B, S, H)
    assert not forward_failures(err), forward_failures(err)


@pytest.mark.parametrize("plant", ["Wg<->Wu", "gain1<->gain2", "Wo transposed"])
def test_forward_pin_rejects_planted_formula_errors(plant):
    """A forward computed with a planted formula error (two weights or gains swapped, a weight
    transposed) must fail the pin against the intended parameters."""
    x, pn, (B, S, H) = _pin_case(0)
    bad = dict(pn)
    if plant == "Wg<->Wu":
        bad["Wg"], bad["Wu"] = pn["Wu"], pn["Wg"]
    elif plant == "gain1<->gain2":
        bad["gain1"], bad["gain2"] = pn["gain2"], pn["gain1"]
    else:
        bad["Wo"] = np.ascontiguousarray(pn["Wo"].T)
    f = decoder.forward(x, bad, B=B, S=S, H=H, seed=3)
    assert forward_failures(forward_stage_errors(f, x, pn, B, S, H)), plant


# ---------------------------------------------------------------------------------------------
# The letter applied at every use of every store together (decoder.all_uses)
# ---------------------------------------------------------------------------------------------
def _all_case(seed=2, B=1, S=12, d=64, H=1, F=96, fmt=fp8.E4M3):
    (x, p, dOut), _ = synth.decoder_inputs(B, S, d, H, F, stream=520 + seed)
    pn = {k: v.float().numpy() for k, v in p.items()}
    g = torch.Generator().manual_seed(90 + seed)
    pn["gain1"] = (1 + 0.1 * torch.randn(d, generator=g)).numpy()
    pn["gain2"] = (1 + 0.1 * torch.randn(d, generator=g)).numpy()
    f = decoder.forward(x.float().numpy(), pn, B=B, S=S, H=H, seed=7, fmt=fmt)
    r = decoder.reference_backward(f, pn, dOut.float().numpy())
    return x, pn, dOut, f, r, (B, S, H)


def test_all_uses_original_is_autograd_without_stores():
    """U at every use: the backward of the realized forward in which no store is seen by the
    backward (every use reads the original), by torch.autograd in fp64."""
    x, pn, dOut, f, r, (B, S, H) = _all_case()
    out = decoder.all_uses(f, pn, dOut.float().numpy(), r, K=3, seed=7, letters=("U",))
    t = lambda a: torch.tensor(np.asarray(a, np.float64), requires_grad=True)
    X = t(x.float().numpy())
    P = {k: t(v) for k, v in pn.items()}
    ste = lambda v, target: v + (torch.tensor(np.asarray(target, np.float64)) - v).detach()
    rms = lambda v, g: g * (v * ((v * v).mean(-1, keepdim=True) + 1e-5).rsqrt())
    T, d = X.shape
    u1 = rms(X, P["gain1"])
    qkv = ste(u1 @ P["Wqkv"], f["QKV"])
    hs = lambda m: m.reshape(B, S, H, d // H).permute(0, 2, 1, 3)
    Q, K, V = (ste(hs(qkv[:, i * d:(i + 1) * d]), f[n]) for i, n in enumerate("QKV"))
    sc = f["c"] * Q @ K.transpose(-1, -2)
    mask = torch.tril(torch.ones(S, S, dtype=torch.bool))
    O = ste(torch.softmax(sc.masked_fill(~mask, float("-inf")), -1) @ V, f["O"])
    h = ste(X + O.permute(0, 2, 1, 3).reshape(T, d) @ P["Wo"], f["h"])
    u2 = rms(h, P["gain2"])
    a = ste(torch.nn.functional.silu(ste(u2 @ P["Wg"], f["g"])) * ste(u2 @ P["Wu"], f["hh"]), f["a"])
    (((h + a @ P["Wd"]) * torch.tensor(dOut.double().numpy())).sum()).backward()
    rel = lambda a_, b_: np.linalg.norm(a_ - b_.detach().numpy()) / np.linalg.norm(b_.detach().numpy())
    for name, grad in (("dx", X.grad), ("dgain1", P["gain1"].grad), ("dWqkv", P["Wqkv"].grad), ("dWo", P["Wo"].grad),
                       ("dgain2", P["gain2"].grad), ("dWg", P["Wg"].grad), ("dWu", P["Wu"].grad),
                       ("dWd", P["Wd"].grad)):
        m, b, s = out["U"][name]
        assert rel(m, grad) < 2e-6, (name, rel(m, grad))
        assert np.all(s == 0)


def test_all_uses_agrees_with_the_per_use_checks_where_the_incoming_gradient_is_fixed():
    """The uses reached first by the backward (a's and u2's weight uses, u2's gain use) see the
    reference incoming gradient whatever the letter, and draw under the same (trial, use) keys as
    the per-use checks: their means equal the per-use oracles' exactly; R reads what the weight
    uses need (no bias)."""
    x, pn, dOut, f, r, (B, S, H) = _all_case(seed=3)
    K = 4
    al = decoder.all_uses(f, pn, dOut.float().numpy(), r, K=K, seed=7)
    pu = decoder.per_use_table(f, pn, r, K=K, seed=7)
    # (the per-use check of u2 takes its incoming gradient rounded to fp32, as the library holds it)
    rel = lambda a_, b_: np.linalg.norm(a_ - b_) / np.linalg.norm(b_)
    for l in ("U", "R", "N"):
        np.testing.assert_allclose(al[l]["dWd"][0], pu[("a", "weight", "dW", l)][0], rtol=1e-12, atol=1e-14)
        assert rel(al[l]["dgain2"][0], pu[("u2", "gain", "dgain", l)][0]) < 1e-6
        F = pn["Wg"].shape[1]
        dW2 = pu[("u2", "weight", "dW", l)][0]
        assert rel(al[l]["dWg"][0], dW2[:, :F]) < 1e-6 and rel(al[l]["dWu"][0], dW2[:, F:]) < 1e-6
    for name in ("dWd", "dWg", "dWu"):
        assert np.all(al["R"][name][1] == 0)
    # R's other gradients change through the normalization-input and D uses: biased, unlike the
    # per-use reading of the same weight gradient
    assert np.linalg.norm(al["R"]["dWo"][1]) > 0 and np.linalg.norm(al["R"]["dWqkv"][1]) > 0


def _n_against_u(f, pn, dOut, r, K, seed):
    al = decoder.all_uses(f, pn, dOut.float().numpy(), r, K=K, seed=seed, letters=("U", "N"))
    zmax = {}
    for name in decoder.GRADS:
        mN, _, se = al["N"][name]
        mU = al["U"][name][0]
        ok = se > 0
        assert np.all(mN[~ok] == mU[~ok]), name
        zmax[name] = float((np.abs(mN - mU)[ok] / se[ok]).max()) if ok.any() else 0.0
    return zmax


def test_all_uses_new_rounding_is_unbiased_to_first_order(monkeypatch):
    """N at every use, many trials: every use reads an independent unbiased rounding, so each
    gradient's mean is U's (every use reading the original) up to second-order terms (the
    normalization input's backward is quadratic in what it reads: a bias of order step^2, below
    this Monte Carlo's resolution): every entry within 5.5 se. A planted error that reads the
    forward's rounding of O at the D use instead of a new rounding fails it."""
    x, pn, dOut, f, r, (B, S, H) = _all_case(seed=4, S=8, d=64, F=64)
    z = _n_against_u(f, pn, dOut, r, 600, 11)
    assert max(z.values()) < 5.5, z
    reads = decoder.all_uses_reads

    def planted(f_, p_, letter, **kw):
        rd = reads(f_, p_, letter, **kw)
        if letter == "N":
            rd["O_D"] = f_["Oq"]
        return rd
    monkeypatch.setattr(decoder, "all_uses_reads", planted)
    z = _n_against_u(f, pn, dOut, r, 600, 11)
    assert z["dWqkv"] > 8 and z["dx"] > 8, z
