"""GPU parity: bs_qround against the oracle's FP8 store, bit for bit."""
import numpy as np
import pytest
import torch

from oracle import fp8, philox, qround as oq

pytestmark = pytest.mark.gpu
FMT = {"e4m3": fp8.E4M3, "e5m2": fp8.E5M2}


def run(lib, x, fmt, mode, seed=0, trial=0, use=0, scale=None):
    print(f"[qround] n={x.numel()} dtype={x.dtype} fmt={fmt} mode={mode} seed={seed}", flush=True)
    codes, s, dg = lib.qround(x.cuda(), fmt, mode, seed, trial, use, None if scale is None else scale.cuda())
    torch.cuda.synchronize()
    return codes.cpu().numpy(), float(s.cpu()[0]), lib.diag_dict(dg)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("fmt", ["e4m3", "e5m2"])
@pytest.mark.parametrize("mode", ["rne", "sr"])
@pytest.mark.parametrize("n", [1, 3, 4, 4097, 100003])
def test_codes_bit_exact(lib, dtype, fmt, mode, n):
    g = torch.Generator().manual_seed(n)
    x = (torch.randn(n, generator=g) * 3).to(dtype)
    codes, s, dg = run(lib, x, fmt, mode, seed=0xB5F0 + n, trial=3, use=257)
    ref = oq.qround(x.float().numpy(), FMT[fmt], oq.RNE if mode == "rne" else oq.SR, 0xB5F0 + n, 3, 257)
    assert s == float(ref.scale) and dg["scale"] == float(ref.scale)
    assert dg["amax"] == float(ref.amax) and dg["nonfinite"] == 0
    assert dg["n_saturated"] == ref.n_saturated
    assert np.array_equal(codes, ref.codes)


@pytest.mark.parametrize("fmt", ["e4m3", "e5m2"])
@pytest.mark.parametrize("mode", ["rne", "sr"])
@pytest.mark.parametrize("factor", [0.25, 8.0])
def test_given_scale_clamps_and_coarse(lib, fmt, mode, factor):
    """A caller's scale (a delayed scale): a quarter of the amax scale clamps the largest entries
    (counted), eight times it sends the small entries to subnormals and zero; codes bit for bit."""
    g = torch.Generator().manual_seed(31)
    x = torch.randn(20011, generator=g) * 2
    s_in = np.float32(np.float32(np.abs(x.numpy()).max()) / np.float32(FMT[fmt].fmax) * np.float32(factor))
    codes, s, dg = run(lib, x, fmt, mode, seed=41, trial=2, use=513, scale=torch.tensor([s_in]))
    ref = oq.qround(x.numpy(), FMT[fmt], oq.RNE if mode == "rne" else oq.SR, 41, 2, 513, scale=s_in)
    assert s == float(s_in) and dg["n_saturated"] == ref.n_saturated
    assert dg["amax"] == float(ref.amax) and dg["nonfinite"] == 0    # reported for the caller's history
    assert (ref.n_saturated > 0) == (factor < 1)
    assert np.array_equal(codes, ref.codes)


@pytest.mark.parametrize("fmt", ["e4m3", "e5m2"])
@pytest.mark.parametrize("mode", ["rne", "sr"])
def test_codec_edge_values_unit_scale(lib, fmt, mode):
    f = FMT[fmt]
    grid = np.unique(np.abs(fp8.decode(np.arange(256, dtype=np.uint8), f)))
    grid = grid[grid <= f.fmax]               # drop the NaN pattern of E4M3 / infinities of E5M2
    mids = (grid[1:] + grid[:-1]) / 2
    vals = np.concatenate([grid, -grid, mids, -mids, np.nextafter(mids.astype(np.float32), np.float32(0)),
                           np.nextafter(mids.astype(np.float32), np.float32(1e9)), [0.0, -0.0, f.min_sub / 2,
                           -f.min_sub / 3, 1e-30, -1e-38, f.fmax * 1.5, -f.fmax * 7, 2.0 ** -20, 2.0 ** -27]])
    x = torch.tensor(vals.astype(np.float32))
    one = torch.ones(1)
    codes, s, dg = run(lib, x, fmt, mode, seed=77, trial=1, use=2, scale=one)
    ref = oq.round_scaled(x.numpy(), f, oq.RNE if mode == "rne" else oq.SR, 77, 1, 2)
    assert s == 1.0
    assert ref[1] == 2
    assert dg["n_saturated"] == ref[1]
    assert np.array_equal(codes, ref[0])


def test_zero_tensor_and_empty(lib):
    codes, s, dg = run(lib, torch.zeros(1000), "e4m3", "sr", seed=5)
    assert s == 1.0 and np.all(codes == 0) and dg["amax"] == 0.0
    codes, s, dg = run(lib, torch.zeros(0), "e5m2", "rne")
    assert s == 1.0 and codes.size == 0 and dg["nonfinite"] == 0


@pytest.mark.parametrize("bad", [float("nan"), float("inf"), float("-inf")])
def test_nonfinite_flagged(lib, bad):
    x = torch.randn(5000)
    x[1234] = bad
    _, _, dg = run(lib, x, "e4m3", "rne")
    assert dg["nonfinite"] == 1
    # with a caller's scale the tensor is checked as well
    _, s, dg = run(lib, x, "e5m2", "sr", seed=3, scale=torch.tensor([0.5]))
    assert dg["nonfinite"] == 1 and s == 0.5


def test_large_tensor_sampled_sr(lib):
    # the size of the E5M2 gradient store of the 16384 x 8192 Linear backward
    n = 16384 * 8192
    g = torch.Generator().manual_seed(11)
    x = (torch.randn(n, generator=g) * 0.1).to(torch.bfloat16)
    codes, s, dg = run(lib, x, "e5m2", "sr", seed=0xB5F4, trial=9, use=1025)
    xf = x.float().numpy()
    amax = np.float32(np.abs(xf).max())
    assert dg["amax"] == float(amax)
    sc = oq.scale_of(amax, fp8.E5M2)
    assert s == float(sc)
    idx = np.unique(np.concatenate([np.arange(4096), np.random.default_rng(0).integers(0, n, 200000), [n - 1]]))
    ref, _ = oq.round_scaled(oq.scaled(xf[idx], sc), fp8.E5M2, oq.SR, 0xB5F4, 9, 1025, elements=idx.astype(np.uint64))
    assert np.array_equal(codes[idx], ref)


def test_ragged_tensor_past_one_grid_sweep_sr(lib):
    # more groups of eight than one sweep of the grid (8192 blocks x 256 threads), the ragged last
    # group (five elements) in a later sweep, fp32 input
    n = 8192 * 256 * 8 + 8 * 1000 + 5
    g = torch.Generator().manual_seed(12)
    x = torch.randn(n, generator=g) * 3.0
    codes, s, dg = run(lib, x, "e4m3", "sr", seed=0xB5F7, trial=4, use=6)
    xf = x.numpy()
    amax = np.float32(np.abs(xf).max())
    assert dg["amax"] == float(amax) and dg["nonfinite"] == 0
    sc = oq.scale_of(amax, fp8.E4M3)
    assert s == float(sc)
    idx = np.unique(np.concatenate([np.arange(2048), np.random.default_rng(1).integers(0, n, 100000),
                                    np.arange(n - 4096, n)]))
    ref, _ = oq.round_scaled(oq.scaled(xf[idx], sc), fp8.E4M3, oq.SR, 0xB5F7, 4, 6, elements=idx.astype(np.uint64))
    assert np.array_equal(codes[idx], ref)


@pytest.mark.parametrize("fmt", ["e4m3", "e5m2"])
def test_sr_decision_at_the_full_word_boundary(lib, fmt):
    """Magnitudes just above zero whose rounding threshold F uses all 32 bits (the fraction of
    the smallest step is the whole 24-bit significand), placed so that R + F lands exactly on
    2^32 (rounds up) or one below it (stays down) for each element's own Philox word R."""
    f = FMT[fmt]
    seed, trial, use = 0xB5F9, 2, 3
    n = 1 << 20
    R = oq.philox.words(seed, trial, use, np.arange(n, dtype=np.uint64)).astype(np.int64)
    T = (1 << 32) - R                              # F = T rounds up, F = T - 1 does not
    cand = np.where((T > (1 << 23)) & (T < (1 << 24)))[0]
    assert cand.size > 1000
    # y = M 2^(e-23) with e chosen so that w = 32: F = M exactly (E4M3 e = -18, E5M2 e = -25)
    e = -18 if fmt == "e4m3" else -25
    M = T[cand] - (np.arange(cand.size) & 1)       # even positions: exactly on the boundary
    g = torch.Generator().manual_seed(5)
    x = (torch.randn(n, generator=g) * 0.3).numpy().astype(np.float32)
    sign = np.where(np.arange(cand.size) % 4 < 2, 1.0, -1.0)
    x[cand] = (sign * np.ldexp(M.astype(np.float64), e - 23)).astype(np.float32)
    codes, s, dg = run(lib, torch.from_numpy(x), fmt, "sr", seed=seed, trial=trial, use=use, scale=torch.ones(1))
    ref, nsat = oq.round_scaled(x, f, oq.SR, seed, trial, use)
    bad = np.where(codes != ref)[0]
    assert bad.size == 0, [(int(i), float(x[i]), int(R[i]), int(codes[i]), int(ref[i])) for i in bad[:8]]
    assert dg["n_saturated"] == nsat
    up = (codes[cand] & 0x7F) == 1
    assert np.array_equal(up, (np.arange(cand.size) & 1) == 0)


@pytest.mark.parametrize("fmt", ["e4m3", "e5m2"])
def test_sr_decision_at_the_boundary_normal_range(lib, fmt):
    """Normal magnitudes in [1, 2): F = D 2^(32 - w) with D the w discarded significand bits
    (w = 20 for E4M3, 21 for E5M2). D = ceil((2^32 - R) / 2^(32 - w)) is the smallest fraction that
    rounds up for the element's word R; D - 1 stays down."""
    f = FMT[fmt]
    seed, trial, use = 0xB5FA, 5, 7
    n = 1 << 16
    R = oq.philox.words(seed, trial, use, np.arange(n, dtype=np.uint64)).astype(np.int64)
    w = 23 - f.mbits
    D = -((R - (1 << 32)) // (1 << (32 - w)))        # ceil((2^32 - R) / 2^(32 - w))
    keep = D < (1 << w)
    D = np.where(np.arange(n) & 1, D - 1, D)
    x = np.ldexp(((1 << w) * (1 << f.mbits) + D).astype(np.float64), -23).astype(np.float32)
    x = np.where(np.arange(n) % 4 < 2, x, -x).astype(np.float32)
    x[~keep] = 1.0
    codes, s, dg = run(lib, torch.from_numpy(x), fmt, "sr", seed=seed, trial=trial, use=use, scale=torch.ones(1))
    ref, _ = oq.round_scaled(x, f, oq.SR, seed, trial, use)
    bad = np.where(codes != ref)[0]
    assert bad.size == 0, [(int(i), float(x[i]), int(R[i]), int(codes[i]), int(ref[i])) for i in bad[:8]]
    one = int(fp8.encode(np.array([1.0]), np.array([False]), f)[0])  # the down value of every element
    up = (codes & 0x7F) != one
    assert np.array_equal(up[keep], (np.arange(n)[keep] & 1) == 0)
