"""GPU parity of the decoder layer at its configured size (B8 x S2048, d 1024, 16 heads of 64,
SwiGLU F 4096, E4M3 RNE stores, K = 16), the benchmark's launch with every use at once.

The oracle's realized forward (fp64, rounded to the model's fp32 / bf16) is handed to the library.
Checked on full tensors: the four stores bit for bit; the eight reference gradients against the
oracle's fp64 straight-through backward; the per-use table's weight and gain rows under U and R,
whose biases have closed forms in the reference incoming gradients (U: the residual times the
incoming gradient; R: zero at a weight use, the residual column sums at a gain use); and the
every-use-at-once U biases of dWo and dWqkv (the same closed forms: U moves no incoming gradient)
and R's dWo (O_q^T times the move of dh at u2's normalization input). Checked on sampled rows
under N: dWd and dWo of the every-use-at-once check against plain K-trial passes over those rows.
"""
import numpy as np
import pytest
import torch

from oracle import decoder, fp8, qround
from oracle.norm_store import fresh_values, norm_backward
from paper_2609_39813_amd import synth
from tests.parity import assert_rel, to_np
from tests.test_gpu_decoder import TOL, check_sumsq, fixed_of

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def say(msg):
    print(f"[layer full size] {msg}", flush=True)


@pytest.fixture(scope="module")
def full(lib):
    cfg = synth.WORKLOADS["decoder_layer_b8_s2048_d1024_h16_f4096"]
    B, S, d, H, F, K, seed = cfg["B"], cfg["S"], cfg["d"], cfg["H"], cfg["F"], cfg["K"], cfg["seed"]
    (x, p, dOut), _ = synth.decoder_inputs(B, S, d, H, F, stream=5)
    pn = {k: v.float().numpy() for k, v in p.items()}
    say("oracle forward")
    f = decoder.forward(x.float().numpy(), pn, B=B, S=S, H=H, seed=seed)
    say("library call (realized forward handed in, every use at once)")
    out = lib.decoder_layer_policy(x.cuda(), {k: v.cuda() for k, v in p.items()}, dOut.cuda(), B=B, S=S, H=H,
                                   fmt="e4m3", fwd_mode="rne", K=K, seed=seed, fixed=fixed_of(f), all_uses=True)
    torch.cuda.synchronize()
    host = {k: v for k, v in out.items() if not isinstance(v, dict)}
    host = {k: to_np(v) for k, v in host.items()}
    host["all_bias"] = {l: {g: to_np(t) for g, t in m.items()} for l, m in out["all_bias"].items()}
    del out
    torch.cuda.empty_cache()
    say("oracle reference backward")
    r = decoder.reference_backward(f, pn, dOut.float().numpy())
    return dict(f=f, r=r, out=host, pn=pn, cfg=cfg, dOut=dOut.float().numpy())


def test_stores_and_reference_gradients(full):
    f, r, out = full["f"], full["r"], full["out"]
    for name, q in (("u1", f["q1"]), ("O", f["qO"]), ("u2", f["q2"]), ("a", f["qa"])):
        assert np.array_equal(out["codes_" + name].reshape(q.codes.shape), q.codes), name
    assert np.array_equal(out["scales"], np.array([f[k].scale for k in ("q1", "qO", "q2", "qa")], np.float32))
    for name in decoder.GRADS:
        say(f"reference {name}")
        assert_rel(out[name], r[name], TOL, name)


def test_per_use_weight_and_gain_rows_under_u_and_r(full, lib):
    """Closed forms of the per-use biases where no new rounding is drawn (Eq. norm-uses)."""
    f, r, out, pn = full["f"], full["r"], full["out"], full["pn"]
    tab = lib.layer_table(out["table_raw"])
    W = {k: pn[k].astype(np.float64) for k in ("Wqkv", "Wg", "Wu")}
    cases = (("u1", f["u1"], f["u1q"], r["dQKV"], "gain1", r["dQKV"] @ W["Wqkv"].T, f["z1"]),
             ("u2", f["u2"], f["u2q"], np.concatenate([r["dg"], r["dhh"]], axis=1), "gain2",
              r["dg"] @ W["Wg"].T + r["dhh"] @ W["Wu"].T, f["z2"]))
    for store, u, uq, dY, gname, du, z in cases:
        say(f"per-use rows of {store}")
        res = u.astype(np.float64) - uq
        check_sumsq(tab[(store, "weight", "dW", "U")][0], float(np.sum((res.T @ dY) ** 2)), (store, "weight U"))
        assert tab[(store, "weight", "dW", "R")][0] == 0.0
        g = pn[gname].astype(np.float64)
        br = ((uq / g - z.astype(np.float64)) * du).sum(0)
        check_sumsq(tab[(store, "gain", "dgain", "R")][0], float(np.sum(br ** 2)), (store, "gain R"))
        assert tab[(store, "gain", "dgain", "U")][0] == 0.0
    say("per-use rows of O and a")
    Ot, Oqt = decoder.tokens(f["O"]).astype(np.float64), decoder.tokens(f["Oq"])
    check_sumsq(tab[("O", "weight", "dW", "U")][0], float(np.sum(((Ot - Oqt).T @ r["dh"]) ** 2)), "O weight U")
    check_sumsq(tab[("a", "weight", "dW", "U")][0], float(np.sum(((f["a"] - f["aq"]).T @ r["dOut"]) ** 2)),
                "a weight U")


def test_every_use_at_once_u_and_r(full):
    f, r, out, pn = full["f"], full["r"], full["out"], full["pn"]
    ab = out["all_bias"]
    say("every use at once: U's dWo and dWqkv, R's dWo")
    Ot, Oqt = decoder.tokens(f["O"]).astype(np.float64), decoder.tokens(f["Oq"])
    assert_rel(ab["U"]["dWo"], (Ot - Oqt).T @ r["dh"], TOL, "U dWo")
    assert_rel(ab["U"]["dWqkv"], (f["u1"].astype(np.float64) - f["u1q"]).T @ r["dQKV"], TOL, "U dWqkv")
    for g in ("dx", "dgain1", "dgain2"):
        assert np.all(ab["U"][g] == 0), g
    W = {k: pn[k].astype(np.float64) for k in ("Wg", "Wu")}
    du2 = r["dg"] @ W["Wg"].T + r["dhh"] @ W["Wu"].T
    g2 = pn["gain2"].astype(np.float64)
    dz = g2 * du2
    move = norm_backward(f["u2q"] / g2, f["r2"], dz) - norm_backward(f["z2"], f["r2"], dz)
    assert_rel(ab["R"]["dWo"], Oqt.T @ move, TOL, "R dWo")


def test_every_use_at_once_new_roundings_sampled_rows(full):
    """N's dWd and dWo on sampled rows: K plain trials of the reads of those rows (dWo's incoming
    gradient dh moves in every trial through u2's normalization input, drawn over all tokens)."""
    f, r, out, pn, cfg = full["f"], full["r"], full["out"], full["pn"], full["cfg"]
    K, seed = cfg["K"], cfg["seed"]
    ab = out["all_bias"]
    rng = np.random.default_rng(5)
    rows_a = np.sort(rng.choice(cfg["F"], 6, replace=False))
    rows_o = np.sort(rng.choice(cfg["d"], 6, replace=False))
    W = {k: pn[k].astype(np.float64) for k in ("Wg", "Wu")}
    du2 = r["dg"] @ W["Wg"].T + r["dhh"] @ W["Wu"].T
    g2 = pn["gain2"].astype(np.float64)
    T = f["a"].shape[0]
    Ot = decoder.tokens(f["O"]).astype(np.float32)
    ya = qround.scaled(f["a"][:, rows_a], f["qa"].scale)
    yo = qround.scaled(Ot[:, rows_o], f["qO"].scale)
    yu2 = qround.scaled(f["u2"], f["q2"].scale)
    el_all = np.arange(f["u2"].size, dtype=np.uint64).reshape(f["u2"].shape)
    tidx = np.arange(T, dtype=np.uint64)[:, None]
    wd, wo = [], []
    for k in range(1, K + 1):
        say(f"N trial {k}")
        aw = fresh_values(ya, tidx * np.uint64(cfg["F"]) + rows_a.astype(np.uint64), fp8.E4M3, f["qa"].scale, seed, k,
                          3 * 256 + 2)
        wd.append(aw.T @ r["dOut"])
        zx = fresh_values(yu2, el_all, fp8.E4M3, f["q2"].scale, seed, k, 2 * 256 + 3) / g2
        dh = r["dOut"] + norm_backward(zx, f["r2"], g2 * du2)
        ow = fresh_values(yo, tidx * np.uint64(cfg["d"]) + rows_o.astype(np.uint64), fp8.E4M3, f["qO"].scale, seed, k,
                          1 * 256 + 2)
        wo.append(ow.T @ dh)
    bd = np.mean(wd, axis=0) - r["dWd"][rows_a]
    bo = np.mean(wo, axis=0) - r["dWo"][rows_o]
    assert_rel(ab["N"]["dWd"][rows_a], bd, TOL, "N dWd rows")
    assert_rel(ab["N"]["dWo"][rows_o], bo, TOL, "N dWo rows")
