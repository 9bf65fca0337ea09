"""Per-tensor amax scaling and the FP8 store (qround).

Test infrastructure (see ``oracle/__init__``).

The forks round the attention output "at the TE output scale" (App. D.2): one
scale for the whole tensor. With FMAX the format's largest finite value:

1. any NaN or infinity makes the call fail (flag ``nonfinite``; no codes);
2. amax = max |x| (exact);
3. s = fl32(amax / FMAX), IEEE single division; s = 1 when amax = 0;
4. y = fl32(x / s), IEEE single division, per element;
5. |y| > FMAX is clamped to FMAX and counted (App. D.2 rounds unbracketed
   top-of-range entries to nearest and counts them);
6. RNE or SR of y onto the grid (``oracle.fp8``); for SR the word of element e
   is Philox(seed; e>>2, trial, use)[e & 3] (``oracle.philox``);
7. code = sign | exponent | mantissa; a negative value rounding to zero keeps
   its sign (code 0x80).

Parity: amax/scale are exact by definition; the codec is pinned in
tests/test_oracle_fp8.py; special cases in tests/test_oracle_qround.py.
"""
from dataclasses import dataclass
import numpy as np

from . import fp8, philox

RNE, SR = 0, 1


@dataclass
class QResult:
    codes: np.ndarray        # uint8, same shape as x
    scale: np.float32
    amax: np.float32
    n_saturated: int
    nonfinite: bool


def scale_of(amax, fmt):
    amax = np.float32(amax)
    if amax == 0:
        return np.float32(1.0)
    return np.float32(amax / np.float32(fmt.fmax))


def scaled(x, s):
    """y = fl32(x / s) for fp32 inputs."""
    return (np.asarray(x, dtype=np.float32) / np.float32(s)).astype(np.float32)


def round_scaled(y, fmt, mode, seed=0, trial=0, use=0, elements=None):
    """Codes of already-scaled fp32 values y, and the number clamped."""
    y = np.asarray(y, dtype=np.float32)
    a = np.abs(y).astype(np.float64)
    sat = a > fmt.fmax
    a = np.where(sat, fmt.fmax, a)
    if mode == RNE:
        mag = fp8.rne_mag(a, fmt)
    else:
        if elements is None:
            elements = np.arange(y.size, dtype=np.uint64).reshape(y.shape)
        R = philox.words(seed, trial, use, elements)
        mag = fp8.sr_mag(a, fmt, R)
    return fp8.encode(mag, np.signbit(y), fmt), int(sat.sum())


def qround(x, fmt, mode, seed=0, trial=0, use=0, scale=None):
    x = np.asarray(x, dtype=np.float32)
    if not np.all(np.isfinite(x)):
        return QResult(None, np.float32(np.nan), np.float32(np.nan), 0, True)
    amax = np.float32(np.max(np.abs(x))) if x.size else np.float32(0)
    s = scale_of(amax, fmt) if scale is None else np.float32(scale)
    codes, nsat = round_scaled(scaled(x, s), fmt, mode, seed, trial, use)
    return QResult(codes, s, amax, nsat, False)


def dequant(codes, s, fmt):
    """deq(C) = val(C) * s, exact in fp64."""
    return fp8.decode(codes, fmt) * np.float64(s)
