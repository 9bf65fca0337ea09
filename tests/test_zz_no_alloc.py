"""GPU: bs_policy_bias_estimate_noalloc (the reducer with the library's own device scratch, for
callers that cannot allocate) against bs_policy_bias_estimate, bit for bit, on two calls in a row
(the second with a smaller input), through the C-ABI."""
import ctypes

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def case(K, m, seed):
    g = torch.Generator().manual_seed(seed)
    return (0.01 + 0.1 * torch.randn(K, m, generator=g)).float().cuda(), torch.randn(m, generator=g).cuda()


def same(a, b):
    return all(torch.equal(x, y) or (x.dtype == torch.float64 and np.array_equal(x.cpu().numpy(), y.cpu().numpy(),
                                                                                 equal_nan=True)) for x, y in zip(a, b))


def test_no_alloc_matches_the_workspace_call_twice(lib):
    for K, m, seed, ref in ((9, 3 * 65536 + 77, 1, True), (4, 1000, 2, False), (2, 257, 3, True)):
        print(f"[no-alloc] K={K} m={m} ref={ref}", flush=True)
        delta, g_ref = case(K, m, seed)
        g_ref = g_ref if ref else None
        want = lib.policy_bias_estimate(delta, g_ref)
        got = lib.policy_bias_estimate_noalloc(delta, g_ref)
        torch.cuda.synchronize()
        assert same(got, want), (K, m)


def test_no_alloc_rejects_sizes_above_its_scratch(lib):
    mx = lib.policy_bias_noalloc_max()
    assert mx == 1 << 26
    buf = torch.zeros(64, device="cuda")
    out = torch.zeros(64, device="cuda")
    summ = torch.zeros(3, dtype=torch.float64, device="cuda")
    # the size check comes before any launch: the short buffers are never read
    code = lib._pb_na(ctypes.c_void_p(buf.data_ptr()), 1, mx + 1, None, ctypes.c_void_p(out.data_ptr()),
                      ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(summ.data_ptr()), lib._stream())
    assert code == 2   # BS_ESHAPE
