"""Pins of the P-store oracle (oracle/pstore.py).

The row functions are checked by exact enumeration, in rational arithmetic, of every rounding
outcome in the paper's cells A and B (App. B.3) under its two rounding laws, against the
closed forms of Table app-theory-errors, Eq. app-replay-error and App. B.4. The backward of each
policy is formed from its operands by the oracle; the expected averages are written from the
closed forms only. The attention-level reference is pinned to torch.autograd in fp64.
"""
from fractions import Fraction as Fr
import itertools

import numpy as np
import pytest
import torch

from oracle import fp8, pstore, qround

CELLS = {
    "A": ([Fr(2, 5), Fr(1, 4), Fr(1, 5), Fr(3, 20)], [[1, 0, 2], [0, 1, -1], [2, -1, 1], [3, 1, 0]], Fr(1, 8)),
    "B": ([Fr(1, 2), Fr(3, 10), Fr(1, 5)], [[1, 1], [2, -1], [0, 3]], Fr(1, 6)),
}


def law_sr(p, step):
    """Per entry: [(value of r, probability)] of stochastic rounding to a grid of spacing step."""
    out = []
    for x in p:
        lo = (x // step) * step
        up = (x - lo) / step
        out.append([(Fr(0), Fr(1))] if up == 0 else [(lo - x, 1 - up), (lo + step - x, up)])
    return out


def law_sym(p, half=Fr(1, 8)):
    return [[(-half, Fr(1, 2)), (half, Fr(1, 2))] for _ in p]


def law_zero(p):
    return [[(Fr(0), Fr(1))] for _ in p]


def outcomes(law):
    """All joint outcomes (r vector as an object array, probability) of independent entries."""
    for combo in itertools.product(*law):
        pr = Fr(1)
        for _, q in combo:
            pr *= q
        yield np.array([v for v, _ in combo], dtype=object), pr


def moments(law):
    s2 = np.array([sum(q * v * v for v, q in e) for e in law], dtype=object)
    m3 = np.array([sum(q * v * v * v for v, q in e) for e in law], dtype=object)
    assert all(sum(q * v for v, q in e) == 0 for e in law)      # right on average
    return s2, m3


def enumerate_policy(code, p, V, law):
    """E[Delta_s | F], E[Delta_V | F] and the per-draw zero flags, with L = |o|^2 / 2."""
    n, d = V.shape
    Es = np.array([Fr(0)] * n, dtype=object)
    EV = np.array([[Fr(0)] * d for _ in range(n)], dtype=object)
    cond_zero = True          # E[Delta_s | F, r] = 0 for every forward rounding r
    zs, zv = True, True       # Delta_s / Delta_V zero in every draw
    nd = pstore.draws(code)
    for r, pr in outcomes(law):
        pq = p + r
        h = V.T @ pq                                  # o = V^T p_q, h = dL/do = o
        dp = V @ h
        ds_ref = pstore.J_apply(p, dp)
        Es_r = np.array([Fr(0)] * n, dtype=object)
        for ra, pa in (outcomes(law) if nd >= 1 else [(None, Fr(1))]):
            for rb, pb in (outcomes(law) if nd >= 2 else [(None, Fr(1))]):
                a = p + ra if ra is not None else None
                b = p + rb if rb is not None else None
                dV, ds = pstore.row_uses(code, p, pq, a, b, V, h)
                dS = ds - ds_ref
                dVe = dV - np.outer(pq, h)
                w = pr * pa * pb
                Es = Es + w * dS
                EV = EV + w * dVe
                Es_r = Es_r + pa * pb * dS
                zs = zs and all(x == 0 for x in dS)
                zv = zv and all(x == 0 for x in dVe.ravel())
        cond_zero = cond_zero and all(x == 0 for x in Es_r)
    return Es, EV, cond_zero, zs, zv


def closed_forms(p, V, law):
    s2, m3 = moments(law)
    G = V @ V.T
    g = np.array([G[j, j] for j in range(len(p))], dtype=object)
    tau = sum(g * s2)
    Sig_Gp = s2 * (G @ p)
    delta = g * s2 - tau * p - 2 * Sig_Gp - g * m3            # Eq. app-replay-error
    dv = -np.array([[s2[j] * V[j, c] for c in range(V.shape[1])] for j in range(len(p))], dtype=object)
    zero_s = np.array([Fr(0)] * len(p), dtype=object)
    zero_v = np.zeros_like(dv) * Fr(0)
    return {   # (E[Delta_s | F], E[Delta_V | F]) per policy (Table app-theory-errors, App. B.4)
        "U/R": (zero_s, zero_v),
        "R/R": (delta, zero_v),
        "U/U": (zero_s, dv),
        "N/N": (-Sig_Gp, dv),
        "R/U": (delta, dv),
        "K/R": (zero_s, zero_v),
        "J2/R": (zero_s, zero_v),
        "Q2/R": ((g * s2 - tau * p - Sig_Gp) / 2, zero_v),
    }, s2, m3


def cell(name):
    p, V, step = CELLS[name]
    return np.array(p, dtype=object), np.array([[Fr(x) for x in row] for row in V], dtype=object), step


@pytest.mark.parametrize("name", ["A", "B"])
@pytest.mark.parametrize("lawname", ["sr", "sym"])
def test_policy_errors_match_closed_forms(name, lawname):
    p, V, step = cell(name)
    assert sum(p) == 1
    law = law_sr(p, step) if lawname == "sr" else law_sym(p)
    exp, s2, m3 = closed_forms(p, V, law)
    if lawname == "sr":
        assert sum(1 for x in s2 if x == 0) == 1             # one entry on the grid, never rounded
        assert any(x != 0 for x in m3)                       # the third-moment term is exercised
    else:
        assert all(x == 0 for x in m3)
    for code, (es, ev) in exp.items():
        Es, EV, cond_zero, zs, zv = enumerate_policy(code, p, V, law)
        assert list(Es) == list(es), code
        assert [list(r) for r in EV] == [list(r) for r in ev], code
        # zeros that hold in every draw (marked * in the table)
        if code in ("U/R", "U/U"):
            assert zs, code
        if code in ("U/R", "R/R", "K/R", "J2/R", "Q2/R"):
            assert zv, code
        # the substitutes of App. B.4 are right on average with the forward held fixed
        if code in ("K/R", "J2/R"):
            assert cond_zero, code


@pytest.mark.parametrize("name", ["A", "B"])
def test_false_statement_refuted_and_zero_rounding_control(name):
    p, V, step = cell(name)
    Es, EV, _, _, _ = enumerate_policy("N/N", p, V, law_sr(p, step))
    assert any(x != 0 for x in Es) and any(x != 0 for x in EV.ravel())    # N/N is not error-free
    for code in ("R/R", "U/U", "N/N", "R/U", "K/R", "J2/R", "Q2/R"):
        Es, EV, _, zs, zv = enumerate_policy(code, p, V, law_zero(p))
        assert zs and zv, code


@pytest.mark.parametrize("name", ["A", "B"])
def test_one_copy_operator_rows_sum_to_zero_in_every_draw(name):
    p, V, step = cell(name)
    ones = np.array([Fr(1)] * len(p), dtype=object)
    for r, _ in outcomes(law_sr(p, step)):
        a = p + r
        assert all(x == 0 for x in pstore.K_apply(a, ones))
        assert all(x == 0 for x in pstore.J_apply(p, ones))


def test_attention_reference_matches_autograd():
    g = torch.Generator().manual_seed(3)
    B, H, S, dh = 1, 2, 37, 8
    Q, Kt, V, dO = (torch.randn(B, H, S, dh, generator=g).double() for _ in range(4))   # fp32 values
    c = 0.3
    out = pstore.check(Q.numpy(), Kt.numpy(), V.numpy(), dO.numpy(), causal=True, c=c, fmt=fp8.E4M3,
                       fwd_mode=qround.RNE, policies=("U/R",), K=1)
    # the program o = (softmax(c Q K^T) + r) V with the rounding r = p_q - p held fixed
    pq = torch.from_numpy(qround.dequant(out["codes"], out["scale"], fp8.E4M3))
    Qr, Kr, Vr = (x.clone().requires_grad_(True) for x in (Q, Kt, V))
    s = c * Qr @ Kr.transpose(-1, -2)
    s = s.masked_fill(~torch.tril(torch.ones(S, S, dtype=torch.bool)), float("-inf"))
    p = torch.softmax(s, dim=-1)
    o = (p + (pq - p).detach()) @ Vr
    (o * dO).sum().backward()
    # the oracle stores and differentiates at the fp32 rounding of P (the realized forward):
    # differences from the fp64 program are of the order of 2^-24 relative
    for name, t in (("dQ", Qr), ("dK", Kr), ("dV", Vr)):
        ref = t.grad[0].numpy()
        assert np.abs(out[name + "_ref"] - ref).max() <= 1e-6 * max(1.0, np.abs(ref).max()), name
    np.testing.assert_allclose(out["O"], (pq @ V).numpy(), rtol=0, atol=0)


def test_attention_policy_zeros_and_draw_counts():
    g = torch.Generator().manual_seed(4)
    B, H, S, dh = 1, 1, 21, 8
    Q, Kt, V, dO = (torch.randn(B, H, S, dh, generator=g, dtype=torch.float64).numpy() for _ in range(4))
    out = pstore.check(Q, Kt, V, dO, causal=True, K=4, seed=9)
    assert np.all(out["U/R"]["dQ"][1] == 0) and np.all(out["U/R"]["dV"][1] == 0)
    assert np.all(out["R/R"]["dV"][1] == 0) and np.all(out["K/R"]["dV"][1] == 0)
    assert np.all(out["U/U"]["dQ"][1] == 0) and np.all(out["U/U"]["dK"][1] == 0)
    assert np.any(out["R/R"]["dQ"][1] != 0) and np.any(out["N/N"]["dV"][1] != 0)
    for code in ("U/R", "R/R", "U/U", "R/U"):
        assert np.all(out[code]["dQ"][2] == 0)                  # no new rounding: se = 0
    assert np.any(out["N/N"]["dQ"][2] > 0) and np.any(out["J2/R"]["dK"][2] > 0)
    # the store: codes above the causal diagonal are zero, p_q = s val(codes) reproduces O
    assert np.all(out["codes"][0, 0][np.triu_indices(S, 1)] == 0)


@pytest.mark.parametrize("name,lawname,printed", [("A", "sr", "0.4808"), ("A", "sym", "0.5598"),
                                                  ("B", "sr", "0.4222"), ("B", "sym", "0.4254")])
def test_new_rounding_over_reuse_ratio_printed_in_app_b3(name, lawname, printed):
    """App. B.3 prints, to four places, the L1 norm of N/N's average error at the softmax's
    backward as a fraction of R/R's, in cells A and B under both laws; the oracle's enumerated
    averages must give the same four digits."""
    p, V, step = cell(name)
    law = law_sr(p, step) if lawname == "sr" else law_sym(p)
    es_n = enumerate_policy("N/N", p, V, law)[0]
    es_r = enumerate_policy("R/R", p, V, law)[0]
    ratio = sum(abs(x) for x in es_n) / sum(abs(x) for x in es_r)
    assert f"{float(ratio):.4f}" == printed, (name, lawname, float(ratio))
