"""Benchmark of the per-use backward-state check on one MI355X.

A step is one full estimate of the RMSNorm -> FP8 store -> Linear operator at the
390M-model MLP up-projection shape (X [8192, 1024] bf16, W [1024, 4096], dY [8192, 4096]):
the forward store, K = 256 new roundings per new-rounding use, every contraction and
the reduction, for the three policies U/U, R/R and N/N (plus the U/R reference). Inputs
are resident in HBM before the timed region. The metric is policy-trials per second:
(#policies x K) / step time.

Prints one JSON line. `roofline` is the dominant kernel's live HIP-event timing against
its bound; `cpu_baseline` times the plain CPU oracle on a bounded sample of the same
workload (rank 0, N = 1 only).
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# Peak figures of one MI355X (AMD public specification).
HBM_PEAK_GBPS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0
# One 32-bit VALU operation per lane per clock: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz
# (the non-packed half of the 157.3 TFLOP/s fp32 figure, counting an FMA as 2 flops).
VALU_LANE_OPS = 256 * 64 * 2.4e9
# Operations of one element-trial of stochastic rounding: a quarter of a Philox4x32-10
# call (10 rounds x (2 multiplies 32x32->64 + 2 three-input xors) for 4 words; the key
# schedule is uniform and runs on the scalar unit) plus the threshold test and the count
# update: 5 + 5 + 2 = 12, each counted as one lane operation.
OPS_PER_ELEMENT_TRIAL = 12
# Ceiling on element-trials per second: 3.28e12.
ALU_PEAK_ETPS = VALU_LANE_OPS / OPS_PER_ELEMENT_TRIAL


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=8)
    return ap.parse_args()


def cpu_baseline(cfg, X, g, W, dY, rows):
    """Time the oracle on `rows` rows of dW and entries of dgain / rows of dX (all policies,
    all K trials), and on twice that; extrapolate linearly to the full output."""
    import numpy as np
    from threadpoolctl import threadpool_info
    from oracle import fp8, norm_store, qround

    Xn, gn, Wn, dYn = X.float().numpy(), g.numpy(), W.float().numpy(), dY.float().numpy()
    rng = np.random.default_rng(0)

    def run(r):
        sel = np.sort(rng.choice(cfg["d"], r, replace=False))
        t0 = time.perf_counter()
        norm_store.check(Xn, gn, Wn, dYn, eps=1e-5, fmt=fp8.E4M3, fwd_mode=qround.RNE, policies=cfg["policies"],
                         K=cfg["K"], seed=cfg["seed"], dw_rows=sel, gain_cols=sel, dx_rows=sel)
        return time.perf_counter() - t0

    t1 = run(rows)
    t2 = run(2 * rows)
    per_row = max(t2 - t1, 1e-9) / rows
    fixed = max(t1 - per_row * rows, 0.0)
    full = fixed + per_row * cfg["d"]
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    return {"value": len(cfg["policies"]) * cfg["K"] / full, "unit": "policy-trials/s", "cores": int(threads),
            "kind": "oracle",
            "sample": (f"plain fp64 oracle, all {len(cfg['policies'])} policies x K={cfg['K']} trials on {rows} and "
                       f"{2 * rows} sampled rows of dW (and as many dgain entries / dX rows): {t1:.1f} s and "
                       f"{t2:.1f} s; linear extrapolation to all {cfg['d']} rows = {full:.0f} s per step")}


def side_measurements(bsp, synth, torch, dev, reps=5):
    """The metric's other two figures, timed live with HIP events: the FP8 store's HBM rate
    on the 16384 x 8192 bf16 gradient (E5M2, SR) and the attention backward's MFMA rate at
    B4 H16 S1024 d64 (causal, three D policies, K = 32)."""
    out = {}
    cfg4 = synth.CONFIGS[4]
    _, _, dy, _, _ = synth.linear_bwd_inputs(cfg4["M"], cfg4["k"], cfg4["n"], torch.bfloat16, 4)
    dy = dy.to(dev)
    n = dy.numel()
    bsp.qround(dy, "e5m2", "sr", seed=cfg4["seed"], trial=1, use=1)
    torch.cuda.synchronize()
    bsp.profile_enable(True)
    for _ in range(reps):
        bsp.qround(dy, "e5m2", "sr", seed=cfg4["seed"], trial=1, use=1)
    torch.cuda.synchronize()
    am_ms, am_n = bsp.profile_read("amax")
    q_ms, q_n = bsp.profile_read("quantize")
    bsp.profile_enable(False)
    am_s, q_s = am_ms / am_n / 1e3, q_ms / q_n / 1e3
    out["qround_e5m2_16384x8192"] = {
        "amax_GBps": round(2 * n / am_s / 1e9, 1), "amax_hbm_frac": round(2 * n / am_s / 1e9 / HBM_PEAK_GBPS, 4),
        "quantize_GBps": round(3 * n / q_s / 1e9, 1), "quantize_hbm_frac": round(3 * n / q_s / 1e9 / HBM_PEAK_GBPS, 4),
        "bytes": "amax reads 2 B/elem; quantize reads 2 B and writes 1 B per element", "elements": n}
    del dy
    cfg3 = synth.CONFIGS[3]
    Q, K, V, dO = (t.to(dev) for t in synth.attention_inputs(cfg3["B"], cfg3["H"], cfg3["S"], cfg3["dh"],
                                                             cfg3["dtype"], 3))
    ws = bsp.attn_workspace(cfg3["B"], cfg3["H"], cfg3["S"], cfg3["dh"], 3, cfg3["K"], dev)
    run = lambda: bsp.attn_bwd_policy(Q, K, V, dO, causal=True, policies=cfg3["policies"], K=cfg3["K"],
                                      seed=cfg3["seed"], fwd_mode=cfg3["fwd_mode"], ws=ws)
    run()
    torch.cuda.synchronize()
    bsp.profile_enable(True)
    t0 = time.perf_counter()
    for _ in range(reps):
        run()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / reps
    b_ms, b_n = bsp.profile_read("attn_bwd")
    f_ms, f_n = bsp.profile_read("attn_fwd")
    bsp.profile_enable(False)
    heads, S, dh = cfg3["B"] * cfg3["H"], cfg3["S"], cfg3["dh"]
    # causal matmul of S x S x dh: S^2 dh flops; reference backward (S, dP, dV, dQ, dK) + 3 bias
    # contractions (G = P K and the two dK bias terms)
    flops = 8 * heads * S * S * dh
    b_s = b_ms / b_n / 1e3
    out["attn_bwd_b4_h16_s1024_d64"] = {
        "TFLOPs": round(flops / b_s / 1e12, 1), "mfma_frac": round(flops / b_s / 1e12 / BF16_MFMA_PEAK_TFLOPS, 4),
        "bwd_ms": round(b_s * 1e3, 4), "fwd_ms": round(f_ms / f_n, 4), "call_ms": round(wall * 1e3, 4),
        "policy_trials_per_s": round(len(cfg3["policies"]) * cfg3["K"] / wall, 1),
        "flops": "8 causal S x S x dh matmuls per head (5 of the reference backward + 3 bias contractions)"}
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the per-use check is measured "
              "on one MI355X and its multi-GPU sharding is described, not built.", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2609_39813_amd import bsp, synth

    cfg, (X, g, W, dY) = synth.config_inputs(2)
    dev = torch.device("cuda:0")
    Xd, gd, Wd, dYd = (t.to(dev) for t in (X, g, W, dY))
    pols = cfg["policies"]
    ws = bsp.rmsnorm_linear_workspace(cfg["T"], cfg["d"], cfg["n"], len(pols), cfg["K"], dev)

    def step():
        return bsp.rmsnorm_linear(Xd, gd, Wd, dYd, fmt="e4m3", fwd_mode=cfg["fwd_mode"], policies=pols, K=cfg["K"],
                                  seed=cfg["seed"], want_y=True, want_se=True, ws=ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    bsp.profile_enable(True)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    prof = {k: bsp.profile_read(k) for k in ("fresh_count", "fresh_count_se", "gemm", "quantize", "rmsnorm_fwd")}
    bsp.profile_enable(False)

    ms_per_step = elapsed / args.steps * 1e3
    value = len(pols) * cfg["K"] * args.steps / elapsed

    # dominant kernel: the K-trial stochastic-rounding counter (VALU-bound)
    fc_ms, fc_n = prof["fresh_count"]
    fc_avg_s = fc_ms / max(fc_n, 1) / 1e3
    et_per_launch = cfg["T"] * cfg["d"] * cfg["K"]
    achieved = et_per_launch / fc_avg_s / 1e9 if fc_n else 0.0
    roofline = {"bound": "alu", "kernel": "fresh_count_kernel<false>", "achieved": round(achieved, 1),
                "peak": round(ALU_PEAK_ETPS / 1e9, 1), "unit": "Gelement-trials/s",
                "frac": round(achieved * 1e9 / ALU_PEAK_ETPS, 4), "traffic": None,
                "avg_launch_ms": round(fc_avg_s * 1e3, 4), "launches": fc_n,
                "work_per_launch": f"{et_per_launch} element-trials ({cfg['T']}x{cfg['d']} elements x K={cfg['K']})"}
    se_ms, se_n = prof["fresh_count_se"]
    # secondary figures of the metric: quantize HBM GB/s and contraction MFMA TFLOP/s
    q_ms, q_n = prof["quantize"]
    q_bytes = cfg["T"] * cfg["d"] * (4 + 1)           # read u fp32, write codes
    g_ms, g_n = prof["gemm"]
    # contractions per step: du, dW_ref, Y, U-bias (3 bf16 terms), N-bias: 7 x 2 T d n
    g_flops = 7 * 2.0 * cfg["T"] * cfg["d"] * cfg["n"] * args.steps
    extra = {"quantize_GBps": round(q_bytes / (q_ms / max(q_n, 1) / 1e3) / 1e9, 1) if q_n else None,
             "quantize_hbm_frac": round(q_bytes / (q_ms / max(q_n, 1) / 1e3) / 1e9 / HBM_PEAK_GBPS, 4) if q_n else None,
             "gemm_TFLOPs": round(g_flops / (g_ms / 1e3) / 1e12, 1) if g_n else None,
             "gemm_mfma_frac": round(g_flops / (g_ms / 1e3) / 1e12 / BF16_MFMA_PEAK_TFLOPS, 4) if g_n else None,
             "kernel_ms_per_step": {k: round(v[0] / args.steps, 4) for k, v in prof.items()},
             "fresh_count_se_Getps": round(et_per_launch / (se_ms / max(se_n, 1) / 1e3) / 1e9, 1) if se_n else None,
             "path": "collapsed (per-element up-counts; se at the gain use from per-trial sums)"}

    extra.update(side_measurements(bsp, synth, torch, dev))

    line = {"metric": "policy-trials/sec", "value": round(value, 1), "unit": "policy-trials/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16+u32",
            "data": "synthetic",
            "config": {"workload": "rmsnorm_linear_390m_mlp_up: X[8192,1024] bf16, W[1024,4096], dY[8192,4096], "
                                   "E4M3 RNE store, policies U/U R/R N/N, K=256",
                       "T": cfg["T"], "d": cfg["d"], "n": cfg["n"], "K": cfg["K"], "policies": list(pols)},
            "roofline": roofline, "extra": extra}
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(cfg, X, g, W, dY, args.cpu_rows)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
