"""GPU parity: bs_te_attn_bwd against the oracle (oracle/te_attention.py).

The forward's fp32 output O and its E4M3 store come from the oracle; the delayed scales from
the oracle's own fp64 pass (the amaxes a previous step would have seen), scaled to provoke
clamps or flushes. Q, K and V are bf16, or the forward's E4M3 stores at their scales (App. D.2).
The library's realized P and pre-cast dS are handed to the oracle, which casts them: the P and
dS codes agree bit for bit, P matches the fp64 softmax, dS and the pre-cast gradients match the
oracle's fp64 values within 1e-5. The returned gradients (BF16, or fp32, values of code times
s_g) are those of the E5M2 casts of the library's own pre-cast values bit for bit; against the
oracle's casts of its fp64 values the codes may differ only where a rounding boundary lies
between the two pre-cast values (rare). amaxes and counts match.
"""
import numpy as np
import pytest
import torch

from oracle import attention, fp8, pstore, qround as oq, te_attention as te
from paper_2609_39813_amd import synth
from tests.parity import assert_rel, to_np

pytestmark = pytest.mark.gpu
TOL = 1e-5
F32 = np.float32


def inputs(B, H, S, seed, sharp=1):
    Q, K, V, dO = synth.attention_inputs(B, H, S, 64, torch.float32, stream=500 + seed)
    return [t.to(torch.bfloat16) for t in (Q * sharp, K, V, dO)]


def fp8_operands(Q, K, V, factors=(1.0, 1.0, 1.0)):
    """The forward's E4M3 stores of Q, K, V at scales amax / 448 times a factor (a stale delayed
    scale clamps): (codes, scales, fp32 dequantized values)."""
    codes, scales, deq = [], [], []
    for t, f in zip((Q, K, V), factors):
        x = t.float().numpy()
        s = F32(oq.scale_of(np.abs(x).max(), fp8.E4M3) * F32(f))
        q = oq.qround(x, fp8.E4M3, oq.RNE, scale=s)
        codes.append(q.codes)
        scales.append(s)
        deq.append((fp8.decode(q.codes, fp8.E4M3).astype(F32) * s).astype(F32))
    return codes, scales, deq


def forward_store(Q, K, V, causal, c, seed, store_id):
    """The forward's fp32 output and its E4M3 stochastic store (oracle only)."""
    O64, P64, _, _ = attention.forward(Q.float().numpy(), K.float().numpy(), V.float().numpy(), causal, c)
    O32 = O64.astype(np.float32)
    q = oq.qround(O32, fp8.E4M3, oq.SR, seed, 0, store_id * 256)
    return O32, P64.astype(np.float32), q


def delayed_scales(Q, K, V, dO, P32, O32, q, causal, c, factors):
    """Scales from the amaxes of the oracle's own pass, each times its factor."""
    probe = (F32(1 / 448), F32(np.abs(dO.float().numpy()).max() / 57344), F32(1.0), F32(1.0))
    ref = te.check(Q.float().numpy(), K.float().numpy(), V.float().numpy(), dO.float().numpy(), P=P32, O=O32,
                   O_codes=q.codes, O_scale=q.scale, causal=causal, c=c, scales=probe, source="P")
    am = (1.0 / 448, ref["amax_dO"] / 57344, ref["amax_dS"] / 57344, ref["amax_grad"] / 57344)
    return tuple(F32(a * f) for a, f in zip(am, factors))


def run_case(lib, B, H, S, *, causal=True, source="R", factors=(1, 1, 1, 1), sharp=1, thr=0.9, seed=1, store_id=4,
             trial=3, fp8_qkv=None, grad_dtype="bf16"):
    """fp8_qkv: None (bf16 Q, K, V) or the factors of the E4M3 stores' scales of Q, K, V."""
    c = 0.125
    Q, K, V, dO = inputs(B, H, S, seed, sharp)
    qkv_sc = None
    if fp8_qkv is not None:
        codes, qkv_sc, deq = fp8_operands(Q, K, V, fp8_qkv)
        ops = [torch.from_numpy(d) for d in deq]          # the operands the forward used
        args = [torch.from_numpy(cd) for cd in codes]
        ref_ops = codes
    else:
        ops = [Q, K, V]
        args = [Q, K, V]
        ref_ops = [t.float().numpy() for t in (Q, K, V)]
    O32, P32, q = forward_store(*ops, causal, c, seed, store_id)
    sc = delayed_scales(*ops, dO, P32, O32, q, causal, c, factors)
    print(f"[te] B={B} H={H} S={S} causal={causal} source={source} factors={factors} sharp={sharp} scales={sc} "
          f"fp8_qkv={fp8_qkv} grad={grad_dtype}", flush=True)
    dev = torch.device("cuda")
    out = lib.te_attn_bwd(*(t.to(dev) for t in args), dO.to(dev), torch.tensor(sc, device=dev),
                          qkv_scales=None if qkv_sc is None else torch.tensor(qkv_sc, device=dev),
                          O=torch.from_numpy(O32).to(dev), O_codes=torch.from_numpy(q.codes).to(dev),
                          O_scale=torch.tensor([q.scale], dtype=torch.float32, device=dev), source=source,
                          threshold=thr, causal=causal, scale=c, seed=seed, store_id=store_id, trial=trial,
                          grad_dtype=grad_dtype, want_p=True, want_ds=True, want_codes=True, want_pre=True)
    torch.cuda.synchronize()
    ref = te.check(*ref_ops, dO.float().numpy(), P=out["P"].cpu().numpy(), dS=out["dS"].cpu().numpy(), O=O32,
                   O_codes=q.codes, O_scale=q.scale, causal=causal, c=c, scales=sc, source=source, thr=F32(thr),
                   seed=seed, store_id=store_id, trial=trial, qkv_scales=qkv_sc, grad_dtype=grad_dtype)
    compare(out, ref, ops[0], ops[1], causal, c, sc, grad_dtype=grad_dtype)
    ref.update(O32=O32, Oc=q.codes, Os=q.scale, sc=sc)
    return out, ref


def fl32(x):
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def compare(out, ref, Q, K, causal, c, sc, totals=True, grad_dtype="bf16"):
    B, H, S, dh = out["dQ"].shape
    flat = lambda t: to_np(t).reshape(B * H, *t.shape[2:])
    assert_rel(to_np(out["P"]), pstore.probabilities(Q.float().numpy(), K.float().numpy(), causal, c), TOL,
               "P against the fp64 softmax")
    assert np.array_equal(out["P_codes"].cpu().numpy(), ref["P_codes"])
    assert np.array_equal(out["dS_codes"].cpu().numpy().reshape(B * H, S, S), ref["dS_codes"])
    assert_rel(flat(out["dS"]), ref["dS"], TOL, "dS")
    pre = out["pre"].cpu().numpy().astype(np.float64)
    n_miss, n_sat, n_edge = 0, 0, 0
    want_dt = torch.bfloat16 if grad_dtype == "bf16" else torch.float32
    for i, name in enumerate(("dQ", "dK", "dV")):
        assert out[name].dtype == want_dt, (name, out[name].dtype)
        p = pre[i].reshape(B * H, S, dh)
        assert_rel(p, ref[name + "_pre"], TOL, name + " pre-cast")
        _, gcodes, ns = te.cast64(p, sc[3], fp8.E5M2)
        n_sat += ns
        got = flat(out[name])                     # BF16 (or fp32) values of fl32(code value * s_g)
        assert np.array_equal(got, te.returned(gcodes, sc[3], fp8.E5M2, grad_dtype)), \
            f"{name}: the returned values are not the cast of the pre-cast values"
        assert np.array_equal(fl32(ref[name]), te.returned(te.cast64(ref[name + "_pre"], sc[3], fp8.E5M2)[1], sc[3],
                                                           fp8.E5M2, grad_dtype))
        _, ocodes, _ = te.cast64(ref[name + "_pre"], sc[3], fp8.E5M2)
        n_edge += int((np.abs(np.abs(ref[name + "_pre"]) / np.float64(sc[3]) - 57344.0) <= 1e-4 * 57344.0).sum())
        miss = gcodes != ocodes
        n_miss += int(miss.sum())
        if miss.any():
            # the cast is monotone, so two codes differ only where the rounding boundary (the midpoint
            # of their values, up to the rounding of x / s_g) lies between the two pre-cast values
            mid = 0.5 * (oq.dequant(gcodes[miss], sc[3], fp8.E5M2) + oq.dequant(ocodes[miss], sc[3], fp8.E5M2))
            dist = np.abs(ref[name + "_pre"][miss] - mid)
            gap = np.abs(ref[name + "_pre"][miss] - p[miss])
            assert np.all(dist <= gap + 1e-7 * np.abs(mid)), f"{name}: a cast differs away from a rounding midpoint"
            assert np.all(gap <= TOL * np.abs(ref[name + "_pre"]).max())
    assert n_miss <= max(2, 1e-4 * 3 * pre[0].size), f"{n_miss} near-tie cast differences"
    if not totals:
        return
    amax = out["amax"].cpu().numpy()
    assert amax[0] == F32(ref["amax_P"]) and amax[1] == F32(ref["amax_dO"]) and amax[2] == F32(ref["amax_dS"])
    assert abs(amax[3] - ref["amax_grad"]) <= TOL * ref["amax_grad"]
    counts = out["counts"].cpu().numpy()
    assert counts[0] == sum(ref["sat_rows"])
    assert counts[1] == ref["sat_dO"] and counts[2] == ref["sat_dS"]
    # the clamp count may differ only at entries within 1e-4 of FMAX (same returned value)
    assert counts[3] == n_sat and abs(int(counts[3]) - ref["sat_grad"]) <= n_edge


@pytest.mark.parametrize("source", ["R", "P", "U", "N"])
def test_causal_ragged_sources(lib, source):
    run_case(lib, 1, 2, 200, source=source, seed=2)


@pytest.mark.parametrize("source", ["P", "R", "repair"])
def test_fp8_operands_and_bf16_return(lib, source):
    """App. D.2's emulation: Q, K, V are the forward's E4M3 stores, the gradients return in BF16."""
    run_case(lib, 1, 2, 200, source=source, seed=13, fp8_qkv=(1.0, 1.0, 1.0), sharp=2 if source == "repair" else 1)


def test_fp8_operands_stale_scales_fp32_return(lib):
    """E4M3 stores of Q and V at half their amax scale (clamped entries), non-causal, fp32 return."""
    run_case(lib, 2, 1, 128, causal=False, source="N", seed=14, fp8_qkv=(0.5, 1.0, 0.5), grad_dtype="f32")


def test_clamped_scales_noncausal(lib):
    """Stale delayed scales: dO, dS and the gradients clamp at their largest entries."""
    out, ref = run_case(lib, 2, 1, 128, causal=False, source="R", factors=(1, 0.5, 0.25, 0.5), seed=3)
    c = out["counts"].cpu().numpy()
    assert c[1] > 0 and c[2] > 0 and c[3] > 0


def test_coarse_scales_subnormal_and_zero_codes(lib):
    """Scales far above the amaxes: most dS entries land on E5M2 subnormals or zero."""
    out, _ = run_case(lib, 1, 2, 64, source="P", factors=(1, 2 ** 8, 2 ** 24, 2 ** 16), seed=4)
    mag = out["dS_codes"].cpu().numpy()[..., np.tril(np.ones((64, 64), dtype=bool))] & 0x7F
    assert (mag == 0).mean() > 0.05 and (mag < 4).mean() > 0.3


def test_repair_selects_saturated_rows(lib):
    out, ref = run_case(lib, 1, 2, 136, source="repair", sharp=4, seed=5)
    n = int(out["counts"].cpu()[0])
    assert 0 < n < 2 * 136 and n == sum(ref["sat_rows"])


@pytest.mark.parametrize("thr", [0.0, 1.5])
def test_repair_threshold_extremes(lib, thr):
    """Threshold 0: every row reads D from P (the same D as the P source); above 1: no row does
    (the same D as the R source). Checked through dS against the oracle of the plain source."""
    out, ref = run_case(lib, 1, 2, 72, source="repair", thr=thr, seed=12, causal=False)
    n = int(out["counts"].cpu()[0])
    assert n == (2 * 72 if thr == 0.0 else 0)
    plain = te.check(*(t.float().numpy() for t in inputs(1, 2, 72, 12)), P=out["P"].cpu().numpy(),
                     dS=out["dS"].cpu().numpy(), O=ref["O32"], O_codes=ref["Oc"], O_scale=ref["Os"], causal=False,
                     c=0.125, scales=ref["sc"], source="P" if thr == 0.0 else "R", seed=12, store_id=4, trial=3)
    np.testing.assert_array_equal(plain["D"], ref["D"])


@pytest.mark.parametrize("S", [4, 64])
def test_small_and_single_tile(lib, S):
    run_case(lib, 1, 1, S, source="R", seed=6 + S)


def test_delayed_scale_steps(lib):
    """bs_te_delayed_scales against the oracle's step over a sequence with zeros, an infinity and
    a NaN, bit for bit (history and scales)."""
    rng = np.random.default_rng(8)
    L, T = 5, 14
    seq = rng.uniform(1e-3, 50.0, size=(T, 4)).astype(np.float32)
    seq[3:9, 0] = 0.0
    seq[7, 2] = np.inf
    seq[9, 3] = np.nan
    dev = torch.device("cuda")
    hist_g, sc_g = torch.zeros(4, L, device=dev), torch.ones(4, device=dev)
    hist_o, sc_o = np.zeros((4, L), np.float32), np.ones(4, np.float32)
    for t in range(T):
        lib.te_delayed_scales(torch.from_numpy(seq[t]).to(dev), hist_g, t, sc_g)
        hist_o, sc_o = te.delayed_scales(hist_o, seq[t], t, sc_o)
        assert np.array_equal(sc_g.cpu().numpy(), sc_o), t
        assert np.array_equal(hist_g.cpu().numpy(), hist_o, equal_nan=True), t


def test_delayed_scaling_loop(lib):
    """Three backward steps whose scales come from the amax history of the steps before (the
    first from a warm-up amax): each step against the oracle, the library's scales against the
    oracle's history of its own amaxes (P, dO, dS bit for bit; the gradients' within 1e-5)."""
    B, H, S, c, store_id, L = 1, 2, 136, 0.125, 4, 16
    dev = torch.device("cuda")
    hist_g, hist_o = torch.zeros(4, L, device=dev), np.zeros((4, L), np.float32)
    sc_o = np.ones(4, np.float32)
    warm = np.array([1.0, 3.0, 5e-3, 1.0], np.float32)
    hist_o, sc_o = te.delayed_scales(hist_o, warm, 0, sc_o)
    sc_g = torch.ones(4, device=dev)
    lib.te_delayed_scales(torch.from_numpy(warm).to(dev), hist_g, 0, sc_g)
    for step in range(1, 4):
        Q, K, V, dO = inputs(B, H, S, 20 + step)
        O32, _, q = forward_store(Q, K, V, True, c, step, store_id)
        sc = tuple(np.float32(x) for x in sc_g.cpu().numpy())
        assert sc[:3] == tuple(sc_o[:3]) and abs(sc[3] - sc_o[3]) <= 1e-5 * sc_o[3]
        print(f"[te] delayed-scaling step {step} scales={sc}", flush=True)
        out = lib.te_attn_bwd(Q.to(dev), K.to(dev), V.to(dev), dO.to(dev), sc_g.clone(),
                              O=torch.from_numpy(O32).to(dev), O_codes=torch.from_numpy(q.codes).to(dev),
                              O_scale=torch.tensor([q.scale], dtype=torch.float32, device=dev), source="R",
                              causal=True, scale=c, seed=step, store_id=store_id, want_p=True, want_ds=True,
                              want_codes=True, want_pre=True)
        torch.cuda.synchronize()
        ref = te.check(Q.float().numpy(), K.float().numpy(), V.float().numpy(), dO.float().numpy(),
                       P=out["P"].cpu().numpy(), dS=out["dS"].cpu().numpy(), O=O32, O_codes=q.codes,
                       O_scale=q.scale, causal=True, c=c, scales=sc, source="R", thr=F32(0.9), seed=step,
                       store_id=store_id)
        compare(out, ref, Q, K, True, c, sc)
        lib.te_delayed_scales(out["amax"], hist_g, step, sc_g)
        hist_o, sc_o = te.delayed_scales(hist_o, [ref["amax_P"], ref["amax_dO"], ref["amax_dS"], ref["amax_grad"]],
                                         step, sc_o)


def test_errors(lib):
    dev = torch.device("cuda")
    Q, K, V, dO = (t.to(dev) for t in inputs(1, 1, 64, 9))
    sc = torch.ones(4, device=dev)
    with pytest.raises(TypeError):
        lib.te_attn_bwd(Q, K, V, dO, sc, source="P", qkv_scales=torch.ones(3, device=dev))   # bf16, not codes
    with pytest.raises(lib.BspError):
        lib.te_attn_bwd(Q, K, V, dO, sc, source="R")                     # no O store
    with pytest.raises(lib.BspError):
        lib.te_attn_bwd(Q, K, V, dO, sc, source="U")                     # no O
    Q6 = torch.zeros(1, 1, 66, 64, dtype=torch.bfloat16, device=dev)
    with pytest.raises(lib.BspError):
        lib.te_attn_bwd(Q6, Q6, Q6, Q6, sc, source="P", ws=torch.empty(1 << 20, dtype=torch.uint8, device=dev))


@pytest.mark.slow
def test_full_size_sampled_heads(lib):
    """B 4, H 16, S 1024, causal, D from the repair (the benchmark's launch): every output of two
    sampled heads against the oracle; the amaxes and counts over the whole call."""
    B, H, S, c, thr, store_id = 4, 16, 1024, 0.125, 0.9, 4
    Q, K, V, dO = inputs(B, H, S, 11)
    heads = [(0, 3), (3, 14)]
    O32 = np.empty((B, H, S, 64), dtype=np.float32)
    for b in range(B):                      # the forward's output, head batch by head batch
        O32[b] = attention.forward(Q[b].float().numpy(), K[b].float().numpy(), V[b].float().numpy(), True, c)[0]
    q = oq.qround(O32, fp8.E4M3, oq.SR, 11, 0, store_id * 256)
    sub = lambda t, b, h: t[b:b + 1, h:h + 1]
    sc = tuple(np.float32(x) for x in (1 / 448, np.abs(dO.float().numpy()).max() / 57344, 4e-5, 2e-5))
    print(f"[te] full size B={B} H={H} S={S} repair scales={sc}", flush=True)
    dev = torch.device("cuda")
    out = lib.te_attn_bwd(Q.to(dev), K.to(dev), V.to(dev), dO.to(dev), torch.tensor(sc, device=dev),
                          O=torch.from_numpy(O32).to(dev), O_codes=torch.from_numpy(q.codes).to(dev),
                          O_scale=torch.tensor([q.scale], dtype=torch.float32, device=dev), source="repair",
                          threshold=thr, causal=True, scale=c, seed=11, store_id=store_id, want_p=True, want_ds=True,
                          want_codes=True, want_pre=True)
    torch.cuda.synchronize()
    for b, h in heads:
        o = {k: (sub(v, b, h) if k != "pre" else v[:, b:b + 1, h:h + 1].contiguous())
             for k, v in out.items() if v is not None and v.dim() == 4 or k == "pre"}
        ref = te.check(*(sub(t, b, h).float().numpy() for t in (Q, K, V, dO)), P=o["P"].cpu().numpy(),
                       dS=o["dS"].cpu().numpy(), O=sub(O32, b, h), O_codes=sub(q.codes, b, h), O_scale=q.scale,
                       causal=True, c=c, scales=sc, source="repair", thr=np.float32(thr))
        compare(o, ref, sub(Q, b, h), sub(K, b, h), True, c, sc, totals=False)
    P = out["P"].cpu().numpy()
    amax, counts = out["amax"].cpu().numpy(), out["counts"].cpu().numpy()
    assert counts[0] == int((P.max(axis=-1) >= np.float32(thr)).sum()) and amax[0] == P.max()
    del P
    assert amax[1] == np.abs(dO.float().numpy()).max() and counts[1] == te.cast(dO.float().numpy(), sc[1], fp8.E5M2)[2]
    dS = out["dS"].cpu().numpy()
    assert amax[2] == np.abs(dS).max() and counts[2] == int((np.abs(dS / sc[2]) > np.float32(57344)).sum())
