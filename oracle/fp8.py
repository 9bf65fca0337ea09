"""FP8 grids and the two rounding rules, in exact fp64 arithmetic.

Test infrastructure (see ``oracle/__init__``).

* Formats: the HYBRID recipe rounds forward tensors to E4M3 and gradients to
  E5M2 (App. D.1). Both are the OCP formats: E4M3 "fn" (bias 7, 3 mantissa
  bits, largest finite 448, no infinity) and E5M2 (bias 15, 2 mantissa bits,
  largest finite 57344).
* Round to nearest, ties to even: the rounding of TE's attention output
  (Sec. 2.1).
* Stochastic rounding: a value bracketed by two neighbouring representable
  numbers goes up or down to one of them with probabilities that make the
  error average to zero (Sec. 2.1). The probability of going up is
  frac = (|y| - lo) / (hi - lo). With a 32-bit random word R and
  F = floor(frac * 2**32), the value rounds up iff R + F >= 2**32, so
  P(up) = F / 2**32. F equals frac * 2**32 exactly whenever at most 32
  fraction bits are discarded (|y| >= 2**-18 for E4M3, >= 2**-25 for E5M2);
  below that it is truncated (bias below 2**-32 of a grid step). The sign is
  kept; the magnitude is rounded.

All inputs here are fp32 values held in fp64, so every operation below is
exact: grid points have at most 4 significant bits and the products and
differences stay far inside 53 bits.

Parity: RNE pinned to torch's float8 casts; decode pinned to torch's float8 ->
float32 conversion; SR pinned by exact rational P(up) and unbiasedness checks
(tests/test_oracle_fp8.py).
"""
from dataclasses import dataclass
import numpy as np


@dataclass(frozen=True)
class Fmt:
    name: str
    ebits: int
    mbits: int
    bias: int
    fmax: float

    @property
    def min_normal(self):
        return 2.0 ** (1 - self.bias)

    @property
    def min_sub(self):
        return 2.0 ** (1 - self.bias - self.mbits)


E4M3 = Fmt("e4m3", 4, 3, 7, 448.0)
E5M2 = Fmt("e5m2", 5, 2, 15, 57344.0)
FORMATS = {0: E4M3, 1: E5M2, "e4m3": E4M3, "e5m2": E5M2}


def bracket(a, fmt):
    """Neighbouring grid magnitudes of magnitudes ``a`` (0 <= a <= fmax).

    Returns (lo, step): lo <= a < lo + step, lo on the grid. When a is on the
    grid, lo == a.
    """
    a = np.asarray(a, dtype=np.float64)
    mant, ex = np.frexp(a)                      # a = mant * 2**ex, mant in [0.5, 1)
    e = ex.astype(np.int64) - 1                 # a in [2**e, 2**(e+1))
    step_normal = np.ldexp(1.0, e - fmt.mbits)
    step = np.where(a < fmt.min_normal, fmt.min_sub, step_normal)
    lo = np.floor(a / step) * step
    return lo, step


def rne_mag(a, fmt):
    """Round magnitudes to the nearest grid value, ties to the even mantissa."""
    lo, step = bracket(a, fmt)
    hi = lo + step
    dlo = a - lo
    dhi = hi - a
    lo_even = (np.floor(lo / step) % 2) == 0
    up = (dhi < dlo) | ((dhi == dlo) & ~lo_even)
    return np.where(dlo == 0, lo, np.where(up, hi, lo))


def sr_threshold(a, fmt):
    """F = floor(frac * 2**32) for each magnitude (uint64), and (lo, step)."""
    lo, step = bracket(a, fmt)
    F = np.floor((a - lo) * np.ldexp(1.0, 32) / step)
    return F.astype(np.uint64), lo, step


def sr_mag(a, fmt, R):
    """Stochastic rounding of magnitudes ``a`` with 32-bit words ``R``."""
    F, lo, step = sr_threshold(a, fmt)
    up = (np.asarray(R, dtype=np.uint64) + F) >= np.uint64(1 << 32)
    up &= F > 0
    return np.where(up, lo + step, lo)


def encode(mag, neg, fmt):
    """FP8 code bits of grid magnitudes ``mag`` with sign flags ``neg``."""
    mag = np.asarray(mag, dtype=np.float64)
    mant, ex = np.frexp(mag)
    e = ex.astype(np.int64) - 1
    normal = mag >= fmt.min_normal
    e_field = np.where(normal, e + fmt.bias, 0)
    m_field = np.where(normal,
                       np.ldexp(mag, -(e - fmt.mbits)) - (1 << fmt.mbits),
                       mag / fmt.min_sub)
    m_field = np.where(mag == 0, 0, m_field)
    code = (e_field.astype(np.int64) << fmt.mbits) | m_field.astype(np.int64)
    code = code | (np.asarray(neg, dtype=np.int64) << 7)
    return code.astype(np.uint8)


def decode(codes, fmt):
    """Real value of each finite FP8 code (fp64)."""
    c = np.asarray(codes, dtype=np.int64)
    neg = (c >> 7) & 1
    e_field = (c >> fmt.mbits) & ((1 << fmt.ebits) - 1)
    m_field = c & ((1 << fmt.mbits) - 1)
    normal = np.ldexp(1.0 + m_field / (1 << fmt.mbits), e_field - fmt.bias)
    sub = m_field * fmt.min_sub
    mag = np.where(e_field == 0, sub, normal)
    return np.where(neg == 1, -mag, mag)


def grid_step(codes, fmt):
    """Grid spacing at a code's magnitude (the step to the next code up)."""
    mag = np.abs(decode(codes, fmt))
    _, step = bracket(mag, fmt)
    return step
