"""Pins of the oracle's Philox4x32-10 (oracle/philox.py).

The oracle's generator is compared word for word with PyTorch's ATen
``at::philox_engine`` (an independent implementation of the same published
generator, header-only, compiled here into a small shim). ATen's engine keys on
the 64-bit seed and puts (offset lo, offset hi, subsequence lo, subsequence hi)
in its counter, so offset = element >> 2 and subsequence = use << 32 | trial
select the oracle's counter (element >> 2, trial, use).
"""
import ctypes
import os
import subprocess

import numpy as np
import pytest
import torch

from oracle import philox

SHIM = r"""
#include <cstdint>
#include <ATen/core/PhiloxRNGEngine.h>
extern "C" void aten_philox(uint64_t seed, uint64_t subseq, uint64_t offset, uint32_t* out) {
  at::philox_engine e(seed, subseq, offset);
  for (int i = 0; i < 4; ++i) out[i] = e();
}
"""


@pytest.fixture(scope="module")
def aten(tmp_path_factory):
    d = tmp_path_factory.mktemp("philox_shim")
    src = d / "shim.cpp"
    src.write_text(SHIM)
    so = d / "shim.so"
    inc = os.path.join(os.path.dirname(torch.__file__), "include")
    r = subprocess.run(["g++", "-O1", "-std=c++17", "-shared", "-fPIC", f"-I{inc}", str(src), "-o", str(so)],
                       capture_output=True, text=True)
    if r.returncode != 0:
        pytest.skip("cannot build the ATen Philox shim: " + r.stderr[-500:])
    lib = ctypes.CDLL(str(so))
    lib.aten_philox.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64, ctypes.POINTER(ctypes.c_uint32)]

    def call(seed, trial, use, block):
        out = (ctypes.c_uint32 * 4)()
        lib.aten_philox(seed, (use << 32) | trial, block, out)
        return list(out)
    return call


def test_matches_aten_engine(aten):
    rng = np.random.default_rng(7)
    cases = [(0, 0, 0, 0), (0xFFFFFFFFFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, (1 << 62) - 1),
             (0xB5F1, 3, 257, 12345), (1, 0, 0, 1 << 32)]
    for _ in range(200):
        cases.append((int(rng.integers(0, 2**63)) * 2 + 1, int(rng.integers(0, 2**32)),
                      int(rng.integers(0, 2**32)), int(rng.integers(0, 2**62))))
    for seed, trial, use, block in cases:
        want = aten(seed, trial, use, block)
        elems = np.array([block * 4 + i for i in range(4)], dtype=np.uint64)
        got = philox.words(seed, trial, use, elems)
        assert [int(v) for v in got] == want, (seed, trial, use, block)


def test_word_layout_selects_output_word():
    w = philox.words(99, 5, 7, np.arange(16, dtype=np.uint64))
    c = philox.philox4x32_10(np.uint64(2), np.uint64(0), np.uint64(5), np.uint64(7), np.uint64(99), np.uint64(0))
    assert [int(x) for x in w[8:12]] == [int(x) for x in c]


def test_uniformity_and_independence():
    e = np.arange(1 << 18, dtype=np.uint64)
    w = philox.words(0xB5F0, 1, 257, e).astype(np.float64) / 2**32
    # mean and variance of U(0,1) within 5 standard errors
    n = w.size
    assert abs(w.mean() - 0.5) < 5 * np.sqrt(1 / 12 / n)
    assert abs(w.var() - 1 / 12) < 5 * np.sqrt(1 / 180 / n)
    # neighbouring elements, trials and uses are uncorrelated
    w2 = philox.words(0xB5F0, 2, 257, e).astype(np.float64) / 2**32
    w3 = philox.words(0xB5F0, 1, 258, e).astype(np.float64) / 2**32
    for a, b in ((w[:-1], w[1:]), (w, w2), (w, w3)):
        assert abs(np.corrcoef(a, b)[0, 1]) < 5 / np.sqrt(n)


# Planted errors: a generator keyed or countered wrongly must fail the comparison above.
_words = philox.words


def _key_halves_swapped(seed, trial, use, elements):
    return _words(((seed & 0xFFFFFFFF) << 32) | (seed >> 32), trial, use, elements)


def _trial_use_swapped(seed, trial, use, elements):
    return _words(seed, use, trial, elements)


def _element_word_shifted(seed, trial, use, elements):
    return _words(seed, trial, use, np.asarray(elements, dtype=np.uint64) ^ np.uint64(1))


@pytest.mark.parametrize("plant", [_key_halves_swapped, _trial_use_swapped, _element_word_shifted],
                         ids=lambda f: f.__name__.strip("_"))
def test_planted_generator_errors_fail_the_pin(aten, monkeypatch, plant):
    monkeypatch.setattr(philox, "words", plant)
    with pytest.raises(AssertionError):
        test_matches_aten_engine(aten)
