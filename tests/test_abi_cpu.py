"""The C ABI without a GPU: the library loads, exports every declared entry
point, rejects bad arguments before touching the device, and the host-side
weight preparation matches the oracle."""
import ctypes as C
import os

import numpy as np
import pytest

from paper_2605_28803_amd import _lib
import paper_2605_28803_amd as oq
from oracle import quant
from tests import parity

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "oq.h")

OK, NULL, SHAPE, ALIGN, DEVICE, HIP, WORKSPACE, ARG = 0, -1, -2, -3, -4, -5, -6, -7
P16 = C.c_void_p(0x10000)     # fake, 16-byte aligned; never dereferenced on error paths
P4 = C.c_void_p(0x10004)


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def test_exports_every_declared_symbol(lib):
    names = _lib.header_symbols(HEADER)
    assert len(names) >= 15
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings(lib):
    for code in (OK, NULL, SHAPE, ALIGN, DEVICE, HIP, WORKSPACE, ARG):
        s = lib.oq_status_string(code).decode()
        assert s.startswith("OQ_")
    assert "unknown" in lib.oq_status_string(12345).decode()
    assert "gfx950" in lib.oq_version().decode()


def test_rotate_quantize_rejects_bad_arguments(lib):
    f = lib.oq_rotate_quantize_act
    assert f(None, 4, 64, 64, 64, None, 0, P16, P16, None) == NULL
    assert f(P16, 4, 64, 64, 64, None, 0, None, P16, None) == NULL
    assert f(P16, -1, 64, 64, 64, None, 0, P16, P16, None) == SHAPE
    assert f(P16, 4, 60, 64, 4, None, 0, P16, P16, None) == SHAPE        # K % 8
    assert f(P16, 4, 96, 96, 64, None, 0, P16, P16, None) == SHAPE       # b does not divide K
    assert f(P16, 4, 64, 64, 48, None, 0, P16, P16, None) == SHAPE       # b not a power of two
    assert f(P16, 4, 64, 32, 64, None, 0, P16, P16, None) == SHAPE       # ldx < K
    assert f(P16, 4, 40, 40, 8, None, 0, P16, P16, None) == SHAPE        # K/8 = 5 unsupported
    assert f(P16, 4, 32768, 32768, 64, None, 0, P16, P16, None) == SHAPE  # K too large
    assert f(P4, 4, 64, 64, 64, None, 0, P16, P16, None) == ALIGN
    assert f(P16, 4, 64, 68, 64, None, 0, P16, P16, None) == ALIGN       # ldx % 8
    assert f(P16, 4, 64, 64, 64, None, -1, P16, P16, None) == ARG


def test_gemm_rejects_bad_arguments(lib):
    g = lib.oq_w4a4_linear
    assert g(None, P16, 4, P16, P16, None, 64, 64, P16, 64, 0, None) == NULL
    assert g(P16, None, 4, P16, P16, None, 64, 64, P16, 64, 0, None) == NULL
    assert g(P16, P16, 4, P16, P16, None, 64, 32, P16, 64, 0, None) == SHAPE   # K < 64
    assert g(P16, P16, 4, P16, P16, None, 64, 96, P16, 64, 0, None) == SHAPE   # K % 64
    assert g(P16, P16, 4, P16, P16, None, 0, 64, P16, 64, 0, None) == SHAPE    # N < 1
    assert g(P16, P16, 4, P16, P16, None, 64, 64, P16, 32, 0, None) == SHAPE   # ldy < N
    assert g(P4, P16, 4, P16, P16, None, 64, 64, P16, 64, 0, None) == ALIGN
    assert g(P16, P16, 4, P16, P16, None, 64, 64, P16, 68, 0, None) == ALIGN   # ldy % 8
    assert g(P16, P16, 4, P16, P16, None, 64, 64, P16, 64, 7, None) == ARG     # out dtype
    h = lib.oq_w4a4_gemm_i32
    assert h(P16, 4, None, 64, 64, P16, 64, None) == NULL
    assert h(P16, 4, P16, 64, 64, P16, 66, None) == ALIGN


def test_tiled_calls_reject_bad_arguments(lib):
    # the tiled layout needs K % 128 == 0
    g = lib.oq_w4a4_linear_tiled
    assert g(P16, P16, 4, P16, P16, None, 64, 192, P16, 64, 0, None) == SHAPE
    assert g(None, P16, 4, P16, P16, None, 64, 128, P16, 64, 0, None) == NULL
    assert g(P16, P16, 4, P16, P16, None, 64, 128, P16, 64, 9, None) == ARG
    h = lib.oq_w4a4_gemm_i32_tiled
    assert h(P16, 4, P16, 64, 64, P16, 64, None) == SHAPE
    assert h(P4, 4, P16, 64, 128, P16, 64, None) == ALIGN
    r = lib.oq_rotate_quantize_act_tiled
    assert r(P16, 4, 64, 64, 64, None, 0, P16, P16, None) == SHAPE
    assert r(P16, 4, 128, 128, 128, None, -1, P16, P16, None) == ARG
    c = lib.oq_codes_to_tiled
    assert c(P16, 4, 192, P16, None) == SHAPE
    assert c(P16, -1, 128, P16, None) == SHAPE
    assert c(None, 4, 128, P16, None) == NULL
    assert c(P16, 4, 128, P4, None) == ALIGN
    assert c(None, 0, 128, None, None) == OK


def test_valid_call_without_gpu_fails_cleanly(lib):
    try:
        import torch
        if torch.cuda.is_available():
            pytest.skip("a GPU is present")
    except Exception:
        pass
    st = lib.oq_rotate_quantize_act(P16, 4, 64, 64, 64, None, 0, P16, P16, None)
    assert st in (HIP, DEVICE)


@pytest.mark.parametrize("N,K,b", [(8, 64, 64), (33, 1024, 1024), (16, 1536, 512), (5, 256, 8)])
def test_host_weight_preparation_matches_oracle(N, K, b):
    rng = np.random.default_rng(N * K + b)
    W = rng.standard_normal((N, K)) * 0.02
    Wq, ws = oq.quantize_weights_host(W, b)
    qo, wso, ro = quant.quantize_weights(W, b)
    q = parity.unpack_int4(Wq)
    # Both sides are float64; codes may differ only within 1e-12 of a boundary.
    diff = q != qo
    assert np.all(~diff | (parity.dist_to_boundary(ro) < 1e-12))
    assert np.allclose(ws, wso.astype(np.float32), rtol=1e-7, atol=0)
    assert not np.any((Wq & 0xF) == 8) and not np.any((Wq >> 4) == 8)


def test_host_weight_preparation_rejects_bad_arguments(lib):
    f = lib.oq_quantize_weights_host
    assert f(None, 4, 64, 64, P16, P16) == NULL
    assert f(P16, 4, 64, 48, P16, P16) == SHAPE
    assert f(P16, 0, 64, 64, P16, P16) == SHAPE


def test_dit_config_validation_without_gpu(lib):
    size = C.c_size_t(0)
    good = _lib.oq_dit_config(0, 18, 1024, 4096, 8, 128, 50, 816, 1, 10, 32)
    assert lib.oq_dit_workspace_bytes(C.byref(good), C.byref(size)) == OK
    assert size.value > 50 * 1024 * 4
    bad = _lib.oq_dit_config(0, 18, 1024, 4096, 8, 64, 50, 816, 1, 10, 32)      # heads*hd != D
    assert lib.oq_dit_workspace_bytes(C.byref(bad), C.byref(size)) == SHAPE
    bad = _lib.oq_dit_config(0, 18, 1000, 4096, 8, 125, 50, 816, 1, 10, 32)     # D % 64
    assert lib.oq_dit_workspace_bytes(C.byref(bad), C.byref(size)) == SHAPE
    bad = _lib.oq_dit_config(0, 18, 1024, 4096, 8, 128, 65, 816, 1, 10, 32)     # tokens > 64
    assert lib.oq_dit_workspace_bytes(C.byref(bad), C.byref(size)) == SHAPE
    bad = _lib.oq_dit_config(7, 18, 1024, 4096, 8, 128, 50, 816, 1, 10, 32)     # arch
    assert lib.oq_dit_workspace_bytes(C.byref(bad), C.byref(size)) == ARG
    assert lib.oq_dit_workspace_bytes(None, C.byref(size)) == NULL
    # GR00T-shaped head: 32 x 48 heads, 300 conditioning tokens, batch 64.
    gr = _lib.oq_dit_config(1, 16, 1536, 6144, 32, 48, 16, 300, 64, 4, 32)
    assert lib.oq_dit_workspace_bytes(C.byref(gr), C.byref(size)) == OK
    # The conditioning k|v of the 8 cross-attention blocks: 8 x 64 x 300 x 3072 fp16.
    assert size.value >= 8 * 64 * 300 * 2 * 1536 * 2
    bad = _lib.oq_dit_config(1, 16, 1536, 6144, 48, 32, 16, 0, 64, 4, 32)     # no conditioning tokens
    assert lib.oq_dit_workspace_bytes(C.byref(bad), C.byref(size)) == SHAPE
    bad = _lib.oq_dit_config(1, 16, 1280, 5120, 32, 40, 16, 300, 64, 4, 32)   # head_dim % 16
    assert lib.oq_dit_workspace_bytes(C.byref(bad), C.byref(size)) == SHAPE
    assert lib.oq_dit_set_condition(None, P16, None) == NULL
    assert lib.oq_dit_step(None, P16, 0, None) == NULL
    assert lib.oq_dit_create(C.byref(good), None, C.byref(C.c_void_p())) == NULL


def test_leading_dimension_of_single_rows():
    """A single row may carry any row stride (numpy gives the size-1 axis of
    a fancy-indexed copy its own value, which torch.from_numpy keeps); the
    binding then passes the row length as the leading dimension, and the row
    stride otherwise."""
    import torch
    perm = np.random.default_rng(0).permutation(64)
    one = torch.from_numpy(np.ascontiguousarray(np.zeros((1, 64), np.float16)[:, perm]))
    assert oq._ld(one) == 64
    assert oq._ld(torch.zeros((3, 64), dtype=torch.float16)) == 64
    assert oq._ld(torch.zeros((3, 80), dtype=torch.float16)[:, :64]) == 80
    assert oq._ld(torch.zeros((1, 80), dtype=torch.float16)[:, :64]) == 64
    assert oq._ld(torch.zeros((0, 64), dtype=torch.float16)) == 64
