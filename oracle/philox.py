"""Philox4x32-10 counter-based generator, restated from its published definition
(Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC'11).

Test infrastructure (see ``oracle/__init__``).

The paper keys its rounding generator on (rounding seed, stream, rank, step,
micro-batch, layer) and draws a new rounding from a separate stream of the same
law (App. D.2, App. D.4). Here the key is the 64-bit seed and the 128-bit counter
is (element >> 2 as 64 bits, trial, use); an element's 32-bit word is output
word ``element & 3``. One call therefore serves four consecutive elements.

Parity: pinned against PyTorch's independent ATen Philox4x32-10 engine
(tests/test_oracle_philox.py) and by statistical tests.
"""
import numpy as np

_MASK = np.uint64(0xFFFFFFFF)
# Round multipliers and Weyl key increments of Philox-4x32 (SC'11, Table 2 / Sec. 4).
M0 = np.uint64(0xD2511F53)
M1 = np.uint64(0xCD9E8D57)
W0 = np.uint64(0x9E3779B9)
W1 = np.uint64(0xBB67AE85)


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Apply ten Philox rounds to counters (c0..c3) under key (k0, k1).

    All arguments are arrays (or scalars) of 32-bit values held in uint64.
    Returns the four output words as uint64 arrays with values < 2**32.
    """
    c0, c1, c2, c3 = (np.asarray(v, dtype=np.uint64) & _MASK for v in (c0, c1, c2, c3))
    k0 = np.asarray(k0, dtype=np.uint64) & _MASK
    k1 = np.asarray(k1, dtype=np.uint64) & _MASK
    for rnd in range(10):
        if rnd:
            k0 = (k0 + W0) & _MASK
            k1 = (k1 + W1) & _MASK
        p0 = M0 * c0          # 32x32 -> 64-bit product, exact in uint64
        p1 = M1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3


def words(seed, trial, use, elements):
    """32-bit random word of each element index for (seed, trial, use).

    ``elements`` is an integer array of flat element indices. Returns uint64
    values in [0, 2**32).
    """
    e = np.asarray(elements, dtype=np.uint64)
    blk = e >> np.uint64(2)
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    out = philox4x32_10(blk & _MASK, blk >> np.uint64(32),
                        np.uint64(trial & 0xFFFFFFFF), np.uint64(use & 0xFFFFFFFF),
                        np.uint64(seed & 0xFFFFFFFF), np.uint64(seed >> 32))
    sel = (e & np.uint64(3)).astype(np.int64)
    stacked = np.stack([np.broadcast_to(o, e.shape) for o in out])
    return np.take_along_axis(stacked, sel[None, ...], axis=0)[0]
