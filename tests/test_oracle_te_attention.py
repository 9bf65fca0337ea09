"""Pins of the FP8 attention backward emulation oracle (oracle/te_attention.py).

* the pre-cast dS with D from P is the softmax backward of the program with incoming gradient
  dO_q (torch.autograd, fp64); D from P equals rowsum(dO_q * P V);
* the casts are the codec at a given scale (E5M2 / E4M3 RNE, clamped and counted);
* the repair reads D from P exactly on the rows whose largest probability reaches the threshold
  and the R copy elsewhere; the gradients are the casts of c dS_q K, c dS_q^T Q and P_q^T dO_q.
"""
import numpy as np
import torch

from oracle import attention, fp8, qround, te_attention as te


def setup(S=24, dh=8, seed=0, sharp=1.0):
    g = torch.Generator().manual_seed(seed)
    Q, K, V, dO = (torch.randn(1, 1, S, dh, generator=g).double() for _ in range(4))   # fp32 values
    Q = (Q * sharp).float().double()
    c = 0.5
    O64, P, _, _ = attention.forward(Q.numpy(), K.numpy(), V.numpy(), True, c)
    P32 = P.astype(np.float32)
    O32 = (P32.astype(np.float64) @ V.numpy()).astype(np.float32)
    q = qround.qround(O32, fp8.E4M3, qround.SR, 3, 0, 0)
    return Q, K, V, dO, c, P32, O32, q


def test_pre_cast_ds_is_the_softmax_backward_and_d_identity():
    Q, K, V, dO, c, P32, O32, q = setup()
    scales = (np.float32(1 / 448), np.float32(0.01), np.float32(1e-3), np.float32(1e-2))
    out = te.check(Q.numpy(), K.numpy(), V.numpy(), dO.numpy(), P=P32, O=O32, O_codes=q.codes, O_scale=q.scale,
                   c=c, scales=scales, source="P")
    dOq, _, _ = te.cast(dO.numpy(), scales[1], fp8.E5M2)
    s = torch.from_numpy(np.log(np.maximum(P32.astype(np.float64), 1e-300))).requires_grad_(True)
    Pt = torch.softmax(s.masked_fill(torch.from_numpy(P32 == 0), float("-inf")), dim=-1)
    ((Pt @ V) * torch.from_numpy(dOq)).sum().backward()
    # autograd renormalizes the fp32 probabilities (their rows sum to 1 within 2^-24)
    ref = s.grad[0, 0].numpy()
    np.testing.assert_allclose(out["dS"][0], ref, rtol=0, atol=1e-6 * np.abs(ref).max())
    D_pv = (dOq[0, 0] * (P32[0, 0].astype(np.float64) @ V[0, 0].numpy())).sum(-1)
    np.testing.assert_allclose(out["D"][0], D_pv, rtol=1e-12, atol=1e-12)


def test_casts_and_gradients():
    Q, K, V, dO, c, P32, O32, q = setup(seed=1)
    scales = (np.float32(P32.max() / 448), np.float32(np.abs(dO.numpy()).max() / 57344), np.float32(2e-4),
              np.float32(5e-5))
    out = te.check(Q.numpy(), K.numpy(), V.numpy(), dO.numpy(), P=P32, O=O32, O_codes=q.codes, O_scale=q.scale,
                   c=c, scales=scales, source="R")
    Pq = qround.dequant(qround.round_scaled(qround.scaled(P32, scales[0]), fp8.E4M3, qround.RNE)[0], scales[0],
                        fp8.E4M3)
    dOq = qround.dequant(qround.round_scaled(qround.scaled(dO.numpy().astype(np.float32), scales[1]), fp8.E5M2,
                                             qround.RNE)[0], scales[1], fp8.E5M2)
    np.testing.assert_array_equal(out["dV_pre"][0], Pq[0, 0].T @ dOq[0, 0])
    dsq = qround.dequant(out["dS_codes"][0], scales[2], fp8.E5M2)
    np.testing.assert_allclose(out["dQ_pre"][0], c * dsq @ K[0, 0].numpy(), rtol=1e-15)
    for name in ("dQ", "dK", "dV"):
        vals = out[name][0] / np.float64(scales[3])
        assert np.all(np.isin(np.abs(vals), fp8.decode(np.arange(128, dtype=np.uint8), fp8.E5M2)))
    # the R copy: D reads the E4M3 store of O
    Or = qround.dequant(q.codes, q.scale, fp8.E4M3)
    np.testing.assert_allclose(out["D"][0], (dOq[0, 0] * Or[0, 0]).sum(-1), rtol=1e-14)


def test_repair_selects_saturated_rows():
    Q, K, V, dO, c, P32, O32, q = setup(seed=2, sharp=4.0)
    scales = (np.float32(1 / 448), np.float32(1e-3), np.float32(1e-3), np.float32(1e-3))
    kw = dict(P=P32, O=O32, O_codes=q.codes, O_scale=q.scale, c=c, scales=scales)
    rep = te.check(Q.numpy(), K.numpy(), V.numpy(), dO.numpy(), source="repair", thr=0.9, **kw)
    fromP = te.check(Q.numpy(), K.numpy(), V.numpy(), dO.numpy(), source="P", **kw)
    fromR = te.check(Q.numpy(), K.numpy(), V.numpy(), dO.numpy(), source="R", **kw)
    sat = P32[0, 0].max(-1) >= 0.9
    assert 0 < sat.sum() < len(sat) and rep["sat_rows"][0] == sat.sum()
    np.testing.assert_array_equal(rep["D"][0][sat], fromP["D"][0][sat])
    np.testing.assert_array_equal(rep["D"][0][~sat], fromR["D"][0][~sat])


def test_delayed_scales_are_the_window_maximum():
    """The ring history gives, at every step, the largest amax of the last `len` steps over FMAX,
    and keeps the old scale while that window holds only zeros (or a non-finite value)."""
    rng = np.random.default_rng(3)
    L, T = 4, 23
    seq = rng.uniform(0.1, 10.0, size=(T, 4)).astype(np.float32)
    seq[6:12, 1] = 0.0                     # a window of zeros for dO: its scale must hold
    seq[15, 2] = np.inf                    # a non-finite amax blocks dS's updates for L steps
    hist, scales = np.zeros((4, L), np.float32), np.ones(4, np.float32)
    prev = scales
    for t in range(T):
        hist, scales = te.delayed_scales(hist, seq[t], t, scales)
        for i in range(4):
            win = seq[max(0, t - L + 1):t + 1, i]
            m = win.max()
            if np.isfinite(m) and m > 0:
                assert scales[i] == np.float32(m / np.float32(te.FMAX[i]))
            else:
                assert scales[i] == prev[i]
        prev = scales
    assert te.FMAX[0] == fp8.E4M3.fmax and te.FMAX[1] == fp8.E5M2.fmax
