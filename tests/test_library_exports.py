"""The C-ABI library loads and exports every symbol include/bsp.h declares (no GPU calls)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2609_39813_amd", "libbsp.so")


def declared():
    text = open(os.path.join(ROOT, "include", "bsp.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bs_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_five_calls():
    names = declared()
    for call in ("bs_qround", "bs_rmsnorm_linear_fwd_bwd", "bs_attn_bwd_policy", "bs_linear_bwd_policy",
                 "bs_policy_bias_estimate"):
        assert call in names


@pytest.mark.skipif(not os.path.exists(LIB), reason="libbsp.so not built")
def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(LIB)
    missing = [n for n in declared() if not hasattr(lib, n)]
    assert not missing, missing
    lib.bs_status_string.restype = ctypes.c_char_p
    assert lib.bs_status_string(0) == b"ok"
    assert lib.bs_version() >= 100


@pytest.mark.skipif(not os.path.exists(LIB), reason="libbsp.so not built")
def test_workspace_queries_are_host_only():
    lib = ctypes.CDLL(LIB)
    f = lib.bs_rmsnorm_linear_workspace_size
    f.restype = ctypes.c_size_t
    f.argtypes = [ctypes.c_int64] * 3 + [ctypes.c_int] * 2
    a = f(8192, 1024, 4096, 3, 256)
    b = f(256, 64, 64, 3, 64)
    assert a > b > 0 and a % 256 == 0


@pytest.mark.skipif(not os.path.exists(LIB), reason="libbsp.so not built")
def test_decoder_layer_workspace_rejects_bad_shapes():
    lib = ctypes.CDLL(LIB)
    f = lib.bs_decoder_layer_workspace_size
    f.restype = ctypes.c_size_t
    f.argtypes = [ctypes.c_int] * 7
    for opts in (0, 1, 2, 3):  # bit 0: every use at once, bit 1: the per-use se
        assert f(2, 24, 128, 2, 256, 4, opts) > 0
        assert f(2, 24, 128, 3, 256, 4, opts) == 0      # d != 64 * H
        assert f(2, 24, 128, 2, 252, 4, opts) == 0      # F not a multiple of 8
        assert f(2, 24, 128, 2, 256, 0, opts) == 0      # K < 1
        assert f(2, 24, 128, 2, 256, 4097, opts) == 0   # K > 4096
    # sized for the whole layer: at least the fp32 activations and the four stores' estimates
    T, d, F = 48, 128, 256
    assert f(2, 24, d, 2, F, 4, 0) >= 4 * T * (10 * d + 6 * F)
    # the every-use check adds its moved gradients and their trial sums
    assert f(2, 24, d, 2, F, 4, 1) >= f(2, 24, d, 2, F, 4, 0) + 20 * T * d
    # the per-use se adds the se of both normalization stores' weight uses (4 policies each), of
    # dK under U / R / N and of the Wo and Wd weight uses
    se_floats = 4 * d * 3 * d + 4 * d * 2 * F + 3 * T * d + d * d + F * d
    assert f(2, 24, d, 2, F, 4, 2) >= f(2, 24, d, 2, F, 4, 0) + 4 * se_floats


@pytest.mark.skipif(not os.path.exists(LIB), reason="libbsp.so not built")
def test_binding_signs_every_declared_call():
    """The Python binding loads (its ctypes signatures resolve) and names every declared call."""
    from paper_2609_39813_amd import bsp
    assert sorted(bsp.EXPORTED) == declared()
