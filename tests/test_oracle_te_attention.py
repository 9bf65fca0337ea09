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
    # returned in BF16 (App. D.2): torch's own E5M2 cast of fl32(pre / s_g), its fp32 dequantization,
    # then torch's bf16 cast
    sg = torch.tensor(scales[3])
    for name in ("dQ", "dK", "dV"):
        y = (torch.from_numpy(out[name + "_pre"][0]).to(torch.float32).double() / sg.double()).float()
        c8 = y.clamp(-57344.0, 57344.0).to(torch.float8_e5m2)
        want = (c8.to(torch.float32) * sg).to(torch.bfloat16).double().numpy()
        np.testing.assert_array_equal(out[name][0], want)
    f32 = te.check(Q.numpy(), K.numpy(), V.numpy(), dO.numpy(), P=P32, O=O32, O_codes=q.codes, O_scale=q.scale,
                   c=c, scales=scales, source="R", grad_dtype="f32")
    for name in ("dQ", "dK", "dV"):
        y = (torch.from_numpy(out[name + "_pre"][0]).double() / sg.double()).float()
        want = (y.clamp(-57344.0, 57344.0).to(torch.float8_e5m2).to(torch.float32) * sg).double().numpy()
        np.testing.assert_array_equal(f32[name][0], want)
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


def test_fp8_operands_are_the_dequantized_codes():
    """With Q, K and V stored in E4M3 at their scales, the backward reads their dequantized values
    (App. D.2): dS with D from P is autograd's softmax backward of the program built on torch's own
    dequantization of the codes, and the pre-cast gradients are c dS_q K_deq, c dS_q^T Q_deq,
    P_q^T dO_q."""
    g = torch.Generator().manual_seed(4)
    S, dh, c = 24, 8, 0.5
    x = [torch.randn(1, 1, S, dh, generator=g) * 2 for _ in range(4)]
    sc = [torch.tensor(float(t.abs().max()) / 448 * f, dtype=torch.float32) for t, f in zip(x[:3], (1.0, 0.5, 1.0))]
    codes = [(t / s).clamp(-448, 448).to(torch.float8_e4m3fn) for t, s in zip(x[:3], sc)]
    deq = [(cd.to(torch.float32) * s).double() for cd, s in zip(codes, sc)]       # torch's dequantization
    dO = x[3]
    Qd, Kd, Vd = deq
    mask = torch.tril(torch.ones(S, S, dtype=torch.bool))
    P32 = torch.softmax((c * Qd @ Kd.transpose(-1, -2)).masked_fill(~mask, float("-inf")), -1).float()
    O32 = (P32.double() @ Vd).float().numpy()
    q = qround.qround(O32, fp8.E4M3, qround.SR, 3, 0, 0)
    scales = (np.float32(1 / 448), np.float32(float(dO.abs().max()) / 57344), np.float32(1e-3), np.float32(1e-2))
    u8 = [cd.view(torch.uint8).numpy() for cd in codes]
    out = te.check(*u8, dO.numpy(), P=P32.numpy(), O=O32, O_codes=q.codes, O_scale=q.scale, c=c, scales=scales,
                   source="P", qkv_scales=tuple(float(s) for s in sc))
    dOq, _, _ = te.cast(dO.numpy(), scales[1], fp8.E5M2)
    s_ = torch.from_numpy(np.log(np.maximum(P32.double().numpy(), 1e-300))).requires_grad_(True)
    Pt = torch.softmax(s_.masked_fill(P32 == 0, float("-inf")), dim=-1)
    ((Pt @ Vd) * torch.from_numpy(dOq)).sum().backward()
    ref = s_.grad[0, 0].numpy()
    np.testing.assert_allclose(out["dS"][0], ref, rtol=0, atol=1e-6 * np.abs(ref).max())
    dsq = qround.dequant(out["dS_codes"][0], scales[2], fp8.E5M2)
    np.testing.assert_allclose(out["dQ_pre"][0], c * dsq @ Kd[0, 0].numpy(), rtol=1e-13, atol=0)
    np.testing.assert_allclose(out["dK_pre"][0], c * dsq.T @ Qd[0, 0].numpy(), rtol=1e-13, atol=0)
    # bf16 operands instead of the codes change the result: the option is not a no-op
    plain = te.check(*(t.numpy() for t in x[:3]), dO.numpy(), P=P32.numpy(), O=O32, O_codes=q.codes,
                     O_scale=q.scale, c=c, scales=scales, source="P")
    assert not np.allclose(plain["dQ_pre"], out["dQ_pre"], rtol=1e-3)
