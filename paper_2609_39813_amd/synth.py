"""Seeded synthetic inputs shaped like the paper's operators (no method arithmetic here).

The paper's workloads are FineWeb-Edu windows through a 390M Llama-3-style model (App. D.1,
Table "Training recipes"); neither the data nor trained weights are available, so these
generators stand in for them with the operator shapes of that model: width 1024, MLP width
4096, 16 heads of 64, sequences of 1024 or 2048 tokens. Every tensor is drawn from torch's
CPU generator seeded with 1000 * stream + i for the i-th tensor of a seed stream (each workload
below has its own), drawn as fp32 normals and rounded to nearest into the stated dtype. N(0, v)
means variance v.

The same tensors feed the oracle (as fp32 values) and the library (as device tensors).
"""
import torch

# the workloads by name: shapes, policies, K, the Philox seed and the seed stream of the tensors
WORKLOADS = {
    "rmsnorm_linear_256x64x64": dict(T=256, d=64, n=64, dtype=torch.float32, K=64, fwd_mode="rne",
                                     policies=("U/U", "R/R", "N/N"), seed=0xB5F1, stream=1),
    "rmsnorm_linear_390m_mlp_up": dict(T=8192, d=1024, n=4096, dtype=torch.bfloat16, K=256, fwd_mode="rne",
                                       policies=("U/U", "R/R", "N/N"), seed=0xB5F2, stream=2),
    "attention_bwd_b4_h16_s1024_d64": dict(B=4, H=16, S=1024, dh=64, dtype=torch.bfloat16, K=32, fwd_mode="sr",
                                           policies=("U", "R", "N"), seed=0xB5F3, stream=3),
    "linear_bwd_e5m2_16384x2048x8192": dict(M=16384, k=2048, n=8192, dtype=torch.bfloat16, K=64,
                                            sharings=("shared", "per_use"), seed=0xB5F4, stream=4),
    "decoder_layer_b8_s2048_d1024_h16_f4096": dict(B=8, S=2048, d=1024, H=16, F=4096, K=16, fwd_mode="rne",
                                                   seed=0xB5F5, stream=5),
}
for _name, _w in WORKLOADS.items():
    _w["name"] = _name

# The FP8 store of attention probabilities (App. B.2-B.4) at the attention shape above: every
# policy of the paper's table, new roundings drawn K times, the forward's store RNE (as TE's).
PSTORE = dict(name="attention_pstore_b4_h16_s1024_d64", B=4, H=16, S=1024, dh=64, dtype=torch.bfloat16, K=32,
              fwd_mode="rne", policies=("U/R", "R/R", "U/U", "N/N", "R/U", "K/R", "J2/R", "Q2/R"), seed=0xB5F6,
              stream=6)


def _gen(stream, i):
    g = torch.Generator()
    g.manual_seed(1000 * stream + i)
    return g


def normal(shape, std, dtype, stream, i):
    return (torch.randn(*shape, generator=_gen(stream, i), dtype=torch.float32) * std).to(dtype)


def rmsnorm_linear_inputs(T, d, n, dtype, stream=2):
    """X ~ N(0,1) [T,d]; gain = 1 + 0.1 N(0,1) [d] fp32; W ~ N(0, 1/d) [d,n]; dY ~ N(0,1) [T,n]."""
    X = normal((T, d), 1.0, dtype, stream, 0)
    gain = 1.0 + 0.1 * torch.randn(d, generator=_gen(stream, 1), dtype=torch.float32)
    W = normal((d, n), d ** -0.5, dtype, stream, 2)
    dY = normal((T, n), 1.0, dtype, stream, 3)
    return X, gain, W, dY


def attention_inputs(B, H, S, dh, dtype=torch.bfloat16, stream=3):
    """Q, K, V, dO ~ N(0, 1) [B, H, S, dh]."""
    return tuple(normal((B, H, S, dh), 1.0, dtype, stream, i) for i in range(4))


def linear_bwd_inputs(M, k, n, dtype=torch.bfloat16, stream=4, tail_frac=0.01, tail_mult=100.0):
    """X ~ N(0,1) [M,k]; W ~ N(0, 1/k) [k,n]; dY ~ N(0, 1e-2) [M,n] with a seeded 1% of entries
    multiplied by 100 (the heavy tail); probes A [M,k], B [k,n] ~ N(0,1) fp32."""
    X = normal((M, k), 1.0, dtype, stream, 0)
    W = normal((k, n), k ** -0.5, dtype, stream, 1)
    dy = torch.randn(M, n, generator=_gen(stream, 2), dtype=torch.float32) * 0.1
    tail = torch.rand(M, n, generator=_gen(stream, 3)) < tail_frac
    dy = torch.where(tail, dy * tail_mult, dy).to(dtype)
    A = torch.randn(M, k, generator=_gen(stream, 4), dtype=torch.float32)
    Bp = torch.randn(k, n, generator=_gen(stream, 5), dtype=torch.float32)
    return X, W, dy, A, Bp


def decoder_inputs(B, S, d, H, F, vocab=131072, stream=5):
    """One decoder layer: x = embedding rows (N(0,1)) of random tokens in [0, vocab), bf16
    [B*S, d]; weights N(0, 0.02^2) in bf16 (Wqkv [d, 3d], Wo [d, d], Wg, Wu [d, F], Wd [F, d]);
    gains 1 (fp32); dOut ~ N(0, 1) bf16 [B*S, d]. Returns (x, params, dOut), (B, S, H)."""
    g = _gen(stream, 0)
    tok = torch.randint(0, vocab, (B * S,), generator=g)
    # embedding row of token v: a normal vector seeded by (stream, v), drawn on demand
    rows = []
    for v in tok.tolist():
        gv = torch.Generator()
        gv.manual_seed(1000 * stream + 17 + v)
        rows.append(torch.randn(d, generator=gv))
    x = torch.stack(rows).to(torch.bfloat16)
    p = {"gain1": torch.ones(d), "gain2": torch.ones(d),
         "Wqkv": normal((d, 3 * d), 0.02, torch.bfloat16, stream, 1),
         "Wo": normal((d, d), 0.02, torch.bfloat16, stream, 2),
         "Wg": normal((d, F), 0.02, torch.bfloat16, stream, 3),
         "Wu": normal((d, F), 0.02, torch.bfloat16, stream, 4),
         "Wd": normal((F, d), 0.02, torch.bfloat16, stream, 5)}
    dOut = normal((B * S, d), 1.0, torch.bfloat16, stream, 6)
    return (x, p, dOut), (B, S, H)


def workload_inputs(name, **override):
    """(the workload's dict with any override, its input tensors) for the first four workloads."""
    w = dict(WORKLOADS[name])
    w.update(override)
    c = w["stream"]
    if "T" in w:
        return w, rmsnorm_linear_inputs(w["T"], w["d"], w["n"], w["dtype"], c)
    if "dh" in w:
        return w, attention_inputs(w["B"], w["H"], w["S"], w["dh"], w["dtype"], c)
    if "M" in w:
        return w, linear_bwd_inputs(w["M"], w["k"], w["n"], w["dtype"], c)
    raise KeyError(name)
