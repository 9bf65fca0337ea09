"""One pre-norm decoder layer with four FP8 stores, and the per-use check of every store.

Test infrastructure (see ``oracle/__init__``).

The layer is the block of the paper's model (App. D.1: pre-norm, root-mean-square
normalization, SwiGLU MLP, no biases; Table "Training recipes"), without rotary embeddings
and with multi-head attention (the configured 16 heads of 64):

  u1 = gain1 * RMSNorm(x)            store 0 (u1)   QKV = deq(C_u1) Wqkv
  Q, K, V = bf16(QKV) per head       O = softmax(c Q K^T, causal) V
                                     store 1 (O)    h = x + deq(C_O) Wo
  u2 = gain2 * RMSNorm(h)            store 2 (u2)   g = deq(C_u2) Wg, hh = deq(C_u2) Wu
  a = silu(g) * hh                   store 3 (a)    out = h + deq(C_a) Wd

Every store is the FP8 store of ``oracle.qround`` with the forward's rounding at trial 0 and
use id store*256. Values the model keeps in bf16 (Q, K, V) or fp32 (h, g, hh, a, O) are
rounded to those formats; the backward passes gradients through every rounding unchanged
(the straight-through reference, Sec. 1, App. B.2).

Per-use check (Sec. 4.1): each use of each store is evaluated at its own operator with the
incoming gradient the reference backward delivers there, under each letter U / R / N (and, in
``all_uses``, each letter applied at every use of every store at once, the backward carrying the
changed incoming gradients on to the earlier uses):

  store u1: gain use, weight use (dWqkv), normalization-input use  -- oracle.norm_store
  store O:  D use (dQ, dK of the attention backward)               -- oracle.attention
            weight use (dWo)                                        -- weight_use below
  store u2: gain use, weight use (dWg, dWu), normalization-input use -- oracle.norm_store
  store a:  weight use (dWd)                                        -- weight_use below

New roundings at a weight use of O or a use id store*256 + 2 and index the store's
elements token-major ([T, width], row t = b*S + s); the D use of O uses id store*256 + 1 and
the head-major layout of the attention store; the normalization stores follow
oracle.norm_store.

Parity: the reference gradients are pinned to torch.autograd in fp64 of the straight-through
program; the weight-use biases to the closed form (U adds -r^T dY, R adds nothing); the
per-use checks reuse the pinned single-operator oracles (tests/test_oracle_decoder.py).
"""
import numpy as np

from . import fp8, policy, qround, norm_store, attention
from .norm_store import rmsnorm_fp32, norm_backward, fresh_values
from .stats import trial_stats

STORES = ("u1", "O", "u2", "a")


def bf16(x):
    """Round to nearest even into bfloat16, returned as fp32 values."""
    b = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (b >> np.uint64(16)) & np.uint64(1)
    r = ((b + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    return r.astype(np.uint32).view(np.float32)


def heads(x, B, S, H):
    """[B*S, H*dh] -> [B, H, S, dh]."""
    T, w = x.shape
    return np.ascontiguousarray(x.reshape(B, S, H, w // H).transpose(0, 2, 1, 3))


def tokens(x):
    """[B, H, S, dh] -> [B*S, H*dh]."""
    B, H, S, dh = x.shape
    return np.ascontiguousarray(x.transpose(0, 2, 1, 3).reshape(B * S, H * dh))


def silu(g):
    return g / (1.0 + np.exp(-g))


def forward(x, p, *, B, S, H, eps=1e-5, fmt=fp8.E4M3, fwd_mode=qround.RNE, seed=0):
    """The realized forward: stores, their inputs and the fp32 / bf16 intermediates."""
    x32 = np.asarray(x, dtype=np.float32)
    T, d = x32.shape
    dh = d // H
    c = 1.0 / np.sqrt(dh)
    f = {}
    z1, u1, r1 = rmsnorm_fp32(x32, p["gain1"], eps)
    q1 = qround.qround(u1, fmt, fwd_mode, seed, 0, 0 * 256)
    u1q = qround.dequant(q1.codes, q1.scale, fmt)
    QKV = (u1q @ p["Wqkv"].astype(np.float64)).astype(np.float32)
    Qh, Kh, Vh = (bf16(heads(QKV[:, i * d:(i + 1) * d], B, S, H)) for i in range(3))
    O64, P, _, _ = attention.forward(Qh, Kh, Vh, True, c)
    O32 = O64.astype(np.float32)
    qO = qround.qround(O32, fmt, fwd_mode, seed, 0, 1 * 256)
    Oq = qround.dequant(qO.codes, qO.scale, fmt)
    h = (x32.astype(np.float64) + tokens(Oq) @ p["Wo"].astype(np.float64)).astype(np.float32)
    z2, u2, r2 = rmsnorm_fp32(h, p["gain2"], eps)
    q2 = qround.qround(u2, fmt, fwd_mode, seed, 0, 2 * 256)
    u2q = qround.dequant(q2.codes, q2.scale, fmt)
    g = (u2q @ p["Wg"].astype(np.float64)).astype(np.float32)
    hh = (u2q @ p["Wu"].astype(np.float64)).astype(np.float32)
    a = (silu(g.astype(np.float64)) * hh.astype(np.float64)).astype(np.float32)
    qa = qround.qround(a, fmt, fwd_mode, seed, 0, 3 * 256)
    aq = qround.dequant(qa.codes, qa.scale, fmt)
    f.update(x=x32, z1=z1, u1=u1, r1=r1, q1=q1, u1q=u1q, QKV=QKV, Q=Qh, K=Kh, V=Vh, P=P, O=O32, qO=qO, Oq=Oq, h=h,
             z2=z2, u2=u2, r2=r2, q2=q2, u2q=u2q, g=g, hh=hh, a=a, qa=qa, aq=aq, c=c, B=B, S=S, H=H, eps=eps,
             fwd_mode=fwd_mode)
    f["out"] = h.astype(np.float64) + aq @ p["Wd"].astype(np.float64)
    return f


def reference_reads(f):
    """What each use reads in the straight-through reference: the rounded value at the weight uses,
    the original at the gain, normalization-input and D uses (Eq. norm-uses; Eq. dterm)."""
    return {"a_W": f["aq"], "u2_g": f["z2"], "u2_W": f["u2q"], "u2_x": f["z2"], "O_W": tokens(f["Oq"]),
            "O_D": f["O"], "u1_g": f["z1"], "u1_W": f["u1q"], "u1_x": f["z1"]}


def layer_backward(f, p, dOut, reads):
    """The layer's backward (fp64) with the value each use reads given in `reads`: a_W (weight use
    of Wd), u2_g / u1_g (gain uses, the normalized value z), u2_W / u1_W (weight uses of [Wg | Wu]
    and Wqkv), u2_x / u1_x (normalization-input uses, z), O_W (weight use of Wo, token-major), O_D
    (the D use, head-major). Returns the gradients and the incoming gradient at every use."""
    dOut = np.asarray(dOut, dtype=np.float32).astype(np.float64)
    W = {k: p[k].astype(np.float64) for k in ("Wqkv", "Wo", "Wg", "Wu", "Wd")}
    B, S, H = f["B"], f["S"], f["H"]
    rd = {k: np.asarray(v, dtype=np.float64) for k, v in reads.items()}
    r = {"dOut": dOut}
    r["dWd"] = rd["a_W"].T @ dOut
    da = dOut @ W["Wd"].T
    g = f["g"].astype(np.float64)
    sg = 1.0 / (1.0 + np.exp(-g))
    r["dg"] = da * f["hh"].astype(np.float64) * sg * (1.0 + g * (1.0 - sg))
    r["dhh"] = da * g * sg
    du2 = r["dg"] @ W["Wg"].T + r["dhh"] @ W["Wu"].T
    r["dWg"] = rd["u2_W"].T @ r["dg"]
    r["dWu"] = rd["u2_W"].T @ r["dhh"]
    r["dgain2"] = (rd["u2_g"] * du2).sum(0)
    r["dh"] = dOut + norm_backward(rd["u2_x"], f["r2"], p["gain2"].astype(np.float64) * du2)
    r["dO_tok"] = r["dh"] @ W["Wo"].T
    r["dWo"] = rd["O_W"].T @ r["dh"]
    dO = heads(r["dO_tok"], B, S, H)
    D = attention.d_from_copy(dO, rd["O_D"])
    dQ, dK, dV = attention.backward(f["Q"], f["K"], f["V"], dO, f["P"], D, f["c"])
    r["dQKV"] = np.concatenate([tokens(dQ), tokens(dK), tokens(dV)], axis=1)
    du1 = r["dQKV"] @ W["Wqkv"].T
    r["dWqkv"] = rd["u1_W"].T @ r["dQKV"]
    r["dgain1"] = (rd["u1_g"] * du1).sum(0)
    r["dx"] = r["dh"] + norm_backward(rd["u1_x"], f["r1"], p["gain1"].astype(np.float64) * du1)
    return r


def reference_backward(f, p, dOut):
    """Straight-through reference gradients and the incoming gradient at every use (fp64)."""
    return layer_backward(f, p, dOut, reference_reads(f))


GRADS = ("dx", "dgain1", "dWqkv", "dWo", "dgain2", "dWg", "dWu", "dWd")


def all_uses_reads(f, p, letter, *, seed, trial, fmt=fp8.E4M3):
    """What every use reads when the letter is applied at all uses together: the original (U), the
    forward's rounding (R) or, per use, a new stochastic rounding at the store's scale (N: trial
    `trial`; use id store*256 + 1 at a gain use and the D use, + 2 at a weight use, + 3 at a
    normalization-input use; the store's elements in its own layout, token-major except the D use's
    head-major O)."""
    if letter == "U":
        return {"a_W": f["a"], "u2_g": f["z2"], "u2_W": f["u2"], "u2_x": f["z2"], "O_W": tokens(f["O"]),
                "O_D": f["O"], "u1_g": f["z1"], "u1_W": f["u1"], "u1_x": f["z1"]}
    g1, g2 = (np.asarray(p[k], np.float32).astype(np.float64) for k in ("gain1", "gain2"))
    if letter == "R":
        return {"a_W": f["aq"], "u2_g": f["u2q"] / g2, "u2_W": f["u2q"], "u2_x": f["u2q"] / g2,
                "O_W": tokens(f["Oq"]), "O_D": f["Oq"], "u1_g": f["u1q"] / g1, "u1_W": f["u1q"],
                "u1_x": f["u1q"] / g1}
    assert letter == "N", letter

    def fresh(x, q, store, j):
        x = np.asarray(x, dtype=np.float32)
        y = qround.scaled(x, q.scale)
        el = np.arange(x.size, dtype=np.uint64).reshape(x.shape)
        return fresh_values(y, el, fmt, q.scale, seed, trial, STORES.index(store) * 256 + j)
    return {"a_W": fresh(f["a"], f["qa"], "a", 2),
            "u2_g": fresh(f["u2"], f["q2"], "u2", 1) / g2, "u2_W": fresh(f["u2"], f["q2"], "u2", 2),
            "u2_x": fresh(f["u2"], f["q2"], "u2", 3) / g2,
            "O_W": fresh(tokens(f["O"]), f["qO"], "O", 2), "O_D": fresh(f["O"], f["qO"], "O", 1),
            "u1_g": fresh(f["u1"], f["q1"], "u1", 1) / g1, "u1_W": fresh(f["u1"], f["q1"], "u1", 2),
            "u1_x": fresh(f["u1"], f["q1"], "u1", 3) / g1}


def all_uses(f, p, dOut, r, *, K, seed, fmt=fp8.E4M3, letters=("U", "R", "N")):
    """The letter applied at every use of every store in one backward (the policy applied to
    every stored rounded tensor), K trials with the forward held fixed (one pass for U and R, which
    draw nothing): {letter: {gradient: (mean, bias, se)}} against the reference gradients r."""
    out = {}
    for letter in letters:
        ntr = K if letter == "N" else 1
        tr = {gname: [] for gname in GRADS}
        for k in range(1, ntr + 1):
            g = layer_backward(f, p, dOut, all_uses_reads(f, p, letter, seed=seed, trial=k, fmt=fmt))
            for gname in GRADS:
                tr[gname].append(g[gname])
        out[letter] = {gname: trial_stats(np.stack(tr[gname] * (K if ntr == 1 else 1)), r[gname])
                       for gname in GRADS}
    return out


def weight_use(Xs, q, dY, fmt, letter, K, seed, use):
    """dW = X_read^T dY for a stored tensor Xs [T, k] (fp32) with forward codes q; returns
    (ref, mean, bias, se) over K trials (new roundings: trials 1..K, use id ``use``)."""
    Xs = np.asarray(Xs, dtype=np.float32)
    dY = np.asarray(dY, dtype=np.float64)
    Xq = qround.dequant(q.codes, q.scale, fmt)
    ref = Xq.T @ dY
    y = qround.scaled(Xs, q.scale)
    elems = np.arange(Xs.size, dtype=np.uint64).reshape(Xs.shape)
    ntr = K if letter == "N" else 1
    tr = []
    for k in range(1, ntr + 1):
        fresh = fresh_values(y, elems, fmt, q.scale, seed, k, use) if letter == "N" else None
        tr.append(policy.read(letter, Xs.astype(np.float64), Xq, fresh).T @ dY)
    g = np.stack(tr * (K if ntr == 1 else 1))
    mean, bias, se = trial_stats(g, ref)
    return ref, mean, bias, se


def per_use_table(f, p, r, *, K, seed, fmt=fp8.E4M3, letters=("U", "R", "N")):
    """{(store, use, gradient, letter): (mean, bias, se, ref)} for every use of every store."""
    out = {}
    # store u1: the normalization store with W = Wqkv and dY = dQKV
    n1 = norm_store.check(f["x"], p["gain1"], p["Wqkv"], r["dQKV"], eps=f["eps"], fmt=fmt, fwd_mode=f["fwd_mode"],
                          policies=tuple(f"{l}/{l}" for l in letters), K=K, seed=seed, store_id=0)
    n1r = norm_store.check(f["x"], p["gain1"], p["Wqkv"], r["dQKV"], eps=f["eps"], fmt=fmt, fwd_mode=f["fwd_mode"],
                           policies=("U/R",), K=K, seed=seed, store_id=0, norm_input="R")
    gu = np.concatenate([p["Wg"], p["Wu"]], axis=1)
    dgu = np.concatenate([r["dg"], r["dhh"]], axis=1)
    n2 = norm_store.check(f["h"], p["gain2"], gu, dgu, eps=f["eps"], fmt=fmt, fwd_mode=f["fwd_mode"],
                          policies=tuple(f"{l}/{l}" for l in letters), K=K, seed=seed, store_id=2)
    n2r = norm_store.check(f["h"], p["gain2"], gu, dgu, eps=f["eps"], fmt=fmt, fwd_mode=f["fwd_mode"],
                           policies=("U/R",), K=K, seed=seed, store_id=2, norm_input="R")
    for store, n, nr in (("u1", n1, n1r), ("u2", n2, n2r)):
        for l in letters:
            m, b, s = n[f"{l}/{l}"]["dgamma"]
            out[(store, "gain", "dgain", l)] = (m, b, s, n["dgamma_ref"])
            m, b, s = n[f"{l}/{l}"]["dW"]
            out[(store, "weight", "dW", l)] = (m, b, s, n["dW_ref"])
        ref = n["dX_ref"]
        for l in ("U", "R"):
            m, b, s = (n if l == "U" else nr)["U/U" if l == "U" else "U/R"]["dX"]
            out[(store, "norm_input", "dX", l)] = (m, b, s, ref)
    # store O: D use through the attention backward, weight use of Wo
    dO = heads(r["dO_tok"], f["B"], f["S"], f["H"])
    at = attention.check(f["Q"], f["K"], f["V"], dO, causal=True, c=f["c"], fmt=fmt, fwd_mode=f["fwd_mode"],
                         policies=letters, K=K, seed=seed, store_id=1, O=f["O"])
    for l in letters:
        for gname in ("dQ", "dK"):
            m, b, s = at[l][gname]
            out[("O", "D", gname, l)] = (m, b, s, at[gname + "_ref"])
    for store, Xs, q, dY in (("O", tokens(f["O"]), _tokens_q(f["qO"]), r["dh"]), ("a", f["a"], f["qa"], r["dOut"])):
        sid = STORES.index(store)
        for l in letters:
            ref, m, b, s = weight_use(Xs, q, dY, fmt, l, K, seed, sid * 256 + 2)
            out[(store, "weight", "dW", l)] = (m, b, s, ref)
    return out


def _tokens_q(q):
    """The store of O with its codes in token-major layout (the weight use's element order)."""
    return qround.QResult(tokens(q.codes), q.scale, q.amax, q.n_saturated, q.nonfinite)


def table(entries):
    """||bias|| / ||ref|| and R = ||bias||^2 / sum se^2 for every (store, use, gradient, letter)."""
    rows = {}
    for key, (m, b, s, ref) in entries.items():
        b2 = float(np.sum(np.asarray(b) ** 2))
        s2 = float(np.sum(np.asarray(s) ** 2))
        rows[key] = {"rel_bias": np.sqrt(b2) / max(float(np.linalg.norm(ref)), 1e-300),
                     "R": b2 / s2 if s2 > 0 else float("nan")}
    return rows
