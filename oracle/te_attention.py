"""An emulation of an FP8 attention backward with delayed scaling (App. D.2; App. E.3).

Test infrastructure (see ``oracle/__init__``).

The forks' backward (App. D.2) is a dense emulation of TE's FP8 attention backward, whose
correction term D is computed from the saved output:

  * the operands Q, K and V are the forward's FP8 tensors: E4M3 codes at their scales, read as
    their fp32 dequantization fl32(val(C) s) (App. D.2 recomputes the output in fp32 from the
    dequantized FP8 Q, K and V); bf16 Q, K, V are accepted as well (qkv_scales None);
  * dO is cast to E5M2 at its delayed scale s_dO: dO_q = Q8(dO);
  * P is recomputed; dV = P_q^T dO_q with P_q the E4M3 store of P at the forward's scale s_P;
  * dP = dO_q V^T; D is taken from the assigned output copy, rowsum(dO_q * O_copy), or from P,
    rowsum(P * dP); dS = P * (dP - D);
  * dS is cast to E5M2 at its delayed scale s_dS; dQ = c dS_q K and dK = c dS_q^T Q;
  * dQ, dK and dV are cast to E5M2 at the gradients' delayed scale s_g, then return in BF16:
    bf16(fl32(val(C) s_g)), the fp32 dequantization rounded to nearest even (fp32 on request).

The delayed scales (P's from the forward; dO, dS, the gradients) come from histories of past
amaxes (TE keeps the largest of 1024, margin 0, App. D.1): they are inputs of the backward,
which reports the amaxes it saw (P, dO, the pre-cast dS and gradients) for the histories;
``delayed_scales`` is one step of that recipe. Every cast rounds to
nearest even, clamps |x/s| > FMAX to FMAX and counts it (the store of reading 1 at a given
scale).

D sources: "P" computes D from P (rowsum(P * dP), equal to rowsum(dO_q * P V)); "U" reads the
original fp32 output O; "R" the forward's E4M3 store of O (TE's saved output); "N" a new
stochastic rounding of O at the same scale; "repair" computes D from P on saturated rows (the
largest probability at least a threshold, 0.9 in App. E.3) and reads R elsewhere.

Casts decide integers, so both sides take the decisions of dS on the same fp32 values: the
GPU's realized pre-cast dS is handed in (as the realized P is), the oracle checks it against
its own fp64 dS and quantizes the handed values. The final casts of the gradients are taken
on the oracle's fp64 pre-cast values; the GPU's fp32 accumulation can only change a decision
within an fp32 rounding of a tie, which the parity test allows and counts.

Parity: the casts are the codec of ``oracle.qround`` at a given scale (pinned there); the
backward pieces are those of ``oracle.attention`` (pinned to torch.autograd); D from P equals
D from P V (identity, tested); the repair selects exactly the rows whose largest probability
reaches the threshold (tests/test_oracle_te_attention.py).
"""
import numpy as np

from . import fp8, qround
from .norm_store import fresh_values

D_SOURCES = ("P", "U", "R", "N", "repair")
FMAX = (448.0, 57344.0, 57344.0, 57344.0)  # P in E4M3; dO, dS and the gradients in E5M2


def delayed_scales(history, amax, step, scales):
    """One step of delayed scaling (App. D.1: history of past amaxes, their maximum, margin 0).

    history [4, len] fp32, amax [4] (P, dO, dS, gradients), scales [4] fp32. The step's amax is
    recorded at slot step % len; a tensor's new scale is fl32(largest |amax| in its history /
    FMAX), or its old scale when that largest amax is zero or not finite. Returns the new
    (history, scales)."""
    h = np.array(history, dtype=np.float32, copy=True)
    h[:, step % h.shape[1]] = np.asarray(amax, dtype=np.float32)
    new = np.array(scales, dtype=np.float32, copy=True)
    for i in range(h.shape[0]):
        m = np.float32(np.max(np.abs(h[i])))
        if np.isfinite(m) and m > 0:
            new[i] = np.float32(m / np.float32(FMAX[i]))
    return h, new


def cast(x, s, fmt):
    """Q8 at a given scale: (dequantized values, codes, clamp count), round to nearest even."""
    y = qround.scaled(np.asarray(x, dtype=np.float32), s)
    codes, nsat = qround.round_scaled(y, fmt, qround.RNE)
    return qround.dequant(codes, s, fmt), codes, nsat


def cast64(x, s, fmt):
    """The same cast of fp64 values: y = x / s rounded to fp32 once, then to nearest even."""
    y = (np.asarray(x, dtype=np.float64) / np.float64(s)).astype(np.float32)
    codes, nsat = qround.round_scaled(y, fmt, qround.RNE)
    return qround.dequant(codes, s, fmt), codes, nsat


def bf16(x):
    """Round fp32 values to nearest even into bfloat16 (returned as fp64 values)."""
    b = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (b >> np.uint64(16)) & np.uint64(1)
    r = ((b + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def returned(codes, s, fmt, grad_dtype="bf16"):
    """A gradient as it returns after its FP8 cast: the fp32 dequantization fl32(val(C) s), in
    BF16 (rounded to nearest even; App. D.2) or left in fp32."""
    v = (fp8.decode(codes, fmt).astype(np.float32) * np.float32(s)).astype(np.float32)
    return bf16(v) if grad_dtype == "bf16" else v.astype(np.float64)


def operands(Q, Kt, V, qkv_scales):
    """The operands of the backward: bf16 inputs as they are, or E4M3 codes read as their fp32
    dequantization fl32(val(C) s) (the emulation's dense fp32 arithmetic, App. D.2)."""
    if qkv_scales is None:
        return tuple(np.asarray(a, dtype=np.float32).astype(np.float64) for a in (Q, Kt, V))
    return tuple((fp8.decode(np.asarray(a, dtype=np.uint8), fp8.E4M3).astype(np.float32) * np.float32(sc))
                 .astype(np.float32).astype(np.float64) for a, sc in zip((Q, Kt, V), qkv_scales))


def d_term(source, P, dP, dOq, O, Or, On, thr):
    """The correction term D per row for a D source."""
    fromP = (P * dP).sum(axis=-1)
    if source == "P":
        return fromP
    if source == "U":
        return (dOq * O).sum(axis=-1)
    if source == "R":
        return (dOq * Or).sum(axis=-1)
    if source == "N":
        return (dOq * On).sum(axis=-1)
    if source == "repair":
        sat = P.max(axis=-1) >= thr
        return np.where(sat, fromP, (dOq * Or).sum(axis=-1))
    raise ValueError(source)


def check(Q, Kt, V, dO, *, P, dS=None, O, O_codes, O_scale, causal=True, c=None, scales, source="R", thr=0.9,
          seed=0, store_id=0, trial=1, heads=None, qkv_scales=None, grad_dtype="bf16"):
    """The emulated backward per head.

    Q, Kt, V [B, H, S, dh]: bf16 values, or E4M3 codes at qkv_scales = (s_Q, s_K, s_V); dO
    [B, H, S, dh]; P: the realized fp32 probabilities [B, H, S, S]; dS: the realized fp32 pre-cast
    dS (None: cast the oracle's own); O: the original fp32 output; O_codes, O_scale: its E4M3 store
    (the R copy); scales: (s_P, s_dO, s_dS, s_g) as fp32; grad_dtype: "bf16" (App. D.2) or "f32",
    the format the cast gradients return in. Besides the values, the clamp counts of dO, dS and
    the three gradients and the rows at or over the threshold are reported.
    """
    Q, Kt, V = operands(Q, Kt, V, qkv_scales)
    dO = np.asarray(dO, dtype=np.float32).astype(np.float64)
    B, H, S, dh = Q.shape
    c = 1.0 / np.sqrt(dh) if c is None else c
    sP, sdO, sdS, sg = (np.float32(x) for x in scales)
    P = np.asarray(P, dtype=np.float32)
    O = np.asarray(O, dtype=np.float32)
    Or = qround.dequant(O_codes, O_scale, fp8.E4M3)
    yO = qround.scaled(O, O_scale)
    elem = np.arange(O.size, dtype=np.uint64).reshape(O.shape)
    Pq, Pcodes, _ = cast(P, sP, fp8.E4M3)
    dOq, _, sat_dO = cast(dO, sdO, fp8.E5M2)
    heads = [(b, h) for b in range(B) for h in range(H)] if heads is None else list(heads)
    out = {"heads": heads, "P_codes": Pcodes, "amax_dO": float(np.abs(dO).max()), "sat_dO": sat_dO,
           "dS": [], "D": [], "dQ_pre": [], "dK_pre": [], "dV_pre": [], "dQ": [], "dK": [], "dV": [],
           "dS_codes": [], "sat_rows": [], "sat_dS": 0, "sat_grad": 0}
    for (b, h) in heads:
        p = P[b, h].astype(np.float64)
        dP = dOq[b, h] @ V[b, h].T
        On = (fresh_values(yO[b, h], elem[b, h], fp8.E4M3, O_scale, seed, trial, store_id * 256 + 1)
              if source == "N" else None)
        D = d_term(source, p, dP, dOq[b, h], O[b, h].astype(np.float64), Or[b, h], On, thr)
        ds = p * (dP - D[:, None])
        if causal:
            ds = np.where(np.tril(np.ones((S, S), dtype=bool)), ds, 0.0)
        dsq, dscodes, nsat = cast(ds if dS is None else dS[b, h], sdS, fp8.E5M2)
        out["sat_dS"] += nsat
        dQp = c * dsq @ Kt[b, h]
        dKp = c * dsq.T @ Q[b, h]
        dVp = Pq[b, h].T @ dOq[b, h]
        for name, v in (("dS", ds), ("D", D), ("dQ_pre", dQp), ("dK_pre", dKp), ("dV_pre", dVp),
                        ("dS_codes", dscodes)):
            out[name].append(v)
        for name, v in (("dQ", dQp), ("dK", dKp), ("dV", dVp)):
            _, codes, nsat = cast64(v, sg, fp8.E5M2)
            out[name].append(returned(codes, sg, fp8.E5M2, grad_dtype))
            out["sat_grad"] += nsat
        out["sat_rows"].append(int((p.max(axis=-1) >= thr).sum()))
    for name in ("dS", "D", "dQ_pre", "dK_pre", "dV_pre", "dQ", "dK", "dV", "dS_codes"):
        out[name] = np.stack(out[name])
    out["amax_P"] = float(np.max([P[b, h].max() for b, h in heads]))
    out["amax_dS"] = float(np.abs(out["dS"] if dS is None else np.asarray(dS)[[b for b, _ in heads], [h for _, h in heads]]).max())
    out["amax_grad"] = float(max(np.abs(out[k]).max() for k in ("dQ_pre", "dK_pre", "dV_pre")))
    return out
