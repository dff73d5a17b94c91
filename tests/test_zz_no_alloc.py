"""The allocation-free calibration entry point (GPU): oq_calibrate_step_scales_noalloc
against oq_calibrate_step_scales (caller workspace) through the C ABI, bit for
bit, on two calls in a row (the second smaller, so the library's scratch holds
the first call's contents), plus the size limit."""
import ctypes as C

import numpy as np
import pytest
import torch

from paper_2605_28803_amd import _lib

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _with_workspace(lib, Y, p, qmax):
    n, K = Y.shape
    d = torch.empty((K,), dtype=torch.float32, device=DEV)
    work = torch.empty((lib.oq_calibrate_workspace_bytes(K),), dtype=torch.uint8, device=DEV)
    st = C.c_void_p(torch.cuda.current_stream(DEV).cuda_stream)
    assert lib.oq_calibrate_step_scales(Y.data_ptr(), n, K, Y.stride(0), p, qmax, d.data_ptr(), work.data_ptr(),
                                        work.numel(), st) == 0
    return d


def _noalloc(lib, Y, p, qmax):
    n, K = Y.shape
    d = torch.full((K,), -1.0, dtype=torch.float32, device=DEV)
    st = C.c_void_p(torch.cuda.current_stream(DEV).cuda_stream)
    assert lib.oq_calibrate_step_scales_noalloc(Y.data_ptr(), n, K, Y.stride(0), p, qmax, d.data_ptr(), st) == 0
    return d


def test_noalloc_calibration_matches_workspace_entry_point():
    lib = _lib.load()
    g = torch.Generator(device=DEV).manual_seed(5)
    cases = [(3000, 4096, 99.9), (700, 1000, 97.5)]  # the second call smaller in n and K
    for n, K, p in cases:
        print(f"noalloc calibration n={n} K={K} p={p}", flush=True)
        Y = torch.randn((n, K), generator=g, device=DEV) * torch.exp(torch.randn((K,), generator=g, device=DEV))
        Y[:, 5] = 0.0
        Y[::3, 7] = -2.5
        a = _noalloc(lib, Y, p, 7.0)
        b = _with_workspace(lib, Y, p, 7.0)
        torch.cuda.synchronize()
        assert torch.equal(a, b), (n, K)
        assert (a >= 0).all()
    # the largest K it takes, then a column count past the limit
    Y = torch.randn((64, 16384), generator=g, device=DEV)
    a = _noalloc(lib, Y, 99.9, 7.0)
    b = _with_workspace(lib, Y, 99.9, 7.0)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    Yb = torch.zeros((4, 16392), device=DEV)
    d = torch.full((16392,), -1.0, device=DEV)
    st = C.c_void_p(torch.cuda.current_stream(DEV).cuda_stream)
    assert lib.oq_calibrate_step_scales_noalloc(Yb.data_ptr(), 4, 16392, 16392, 99.9, 7.0, d.data_ptr(), st) == -6
    torch.cuda.synchronize()
    assert (d == -1.0).all()
