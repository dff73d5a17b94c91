"""Static per-step, per-channel steps, host side (CPU only): the per-step
weight fold against the oracle and argument validation of the new calls
(every check runs before any device work)."""
import ctypes as C

import numpy as np
import pytest

import paper_2605_28803_amd as oq
from paper_2605_28803_amd import _lib
from oracle import quant
from tests import parity

SHAPE, NULL, ALIGN, ARG, OK = -2, -1, -3, -7, 0
P16 = C.c_void_p(0x10000)
P4 = C.c_void_p(0x10004)


@pytest.mark.parametrize("N,K,b", [(40, 64, 64), (96, 1024, 1024), (33, 1536, 512), (7, 256, 8)])
def test_step_fold_matches_oracle(N, K, b):
    rng = np.random.default_rng(N + K + b)
    w = rng.standard_normal((N, K)) * 0.02
    w[:, rng.choice(K, 3, replace=False)] *= 30
    d = np.exp(rng.standard_normal(K)).astype(np.float32)
    d[rng.choice(K, 2, replace=False)] = 0.0
    wq, ws = oq.quantize_weights_step_host(w, b, d)
    qo, wso, ro = quant.fold_weights_step(w, b, d.astype(np.float64))
    qg = parity.unpack_int4(wq)
    mism = qg != qo
    # both sides are float64 with different butterfly orders: a code may
    # differ only where the exact ratio is a rounding tie up to ~1e-12
    assert np.count_nonzero(mism) <= 2
    assert np.all(parity.dist_to_boundary(ro[mism]) < 1e-9)
    assert np.allclose(ws, wso.astype(np.float32), rtol=1e-7)
    # channels with a zero step contribute nothing
    assert not qg[:, d == 0].any()


def test_static_calls_reject_bad_arguments():
    lib = _lib.load()
    f = lib.oq_rotate_quantize_act_static
    assert f(P16, 4, 1024, 1024, 1024, None, P16, P16, None) == NULL     # delta
    assert f(P16, 4, 1024, 1024, 1024, P4, P16, P16, None) == ALIGN      # delta 16-byte
    assert f(P16, 4, 1024, 1000, 1024, P16, P16, P16, None) == SHAPE     # ldx < K
    assert f(P16, 4, 1024, 1024, 48, P16, P16, P16, None) == SHAPE       # block not a power of two
    assert f(None, 0, 1024, 1024, 1024, None, None, None, None) == OK    # empty
    ft = lib.oq_rotate_quantize_act_static_tiled
    assert ft(P16, 4, 1088, 1088, 64, P16, P16, P16, None) == SHAPE      # K % 128
    r = lib.oq_rotate_act_f32
    assert r(P16, 4, 1024, 1024, 1024, None, None) == NULL
    assert r(P16, 4, 1024, 1024, 1024, P4, None) == ALIGN
    assert r(None, 0, 1024, 1024, 1024, None, None) == OK
    c = lib.oq_calibrate_step_scales
    ws = lib.oq_calibrate_workspace_bytes(1024)
    assert ws == 1024 * 1032 and lib.oq_calibrate_workspace_bytes(0) == 0
    assert c(P16, 100, 1024, 1024, 0.0, 7.0, P16, P16, ws, None) == ARG       # p
    assert c(P16, 100, 1024, 1024, 100.5, 7.0, P16, P16, ws, None) == ARG
    assert c(P16, 100, 1024, 1024, 99.9, 0.0, P16, P16, ws, None) == ARG      # qmax
    assert c(P16, 100, 1024, 1024, 99.9, float("inf"), P16, P16, ws, None) == ARG
    assert c(P16, 0, 1024, 1024, 99.9, 7.0, P16, P16, ws, None) == SHAPE      # empty column
    assert c(P16, 100, 1024, 1000, 99.9, 7.0, P16, P16, ws, None) == SHAPE    # ldy < K
    assert c(P16, 100, 1024, 1024, 99.9, 7.0, P16, P16, ws - 1, None) == SHAPE
    assert c(P16, 100, 1024, 1024, 99.9, 7.0, P16, None, ws, None) == NULL
    assert c(P16, 100, 1024, 1024, 99.9, 7.0, P16, P4, ws, None) == ALIGN     # work 16-byte
    assert c(None, 0, 0, 0, 99.9, 7.0, None, None, 0, None) == OK             # no columns
    h = lib.oq_quantize_weights_step_host
    w = np.zeros((1, 8))
    out = np.zeros(4, dtype=np.uint8)
    sc = np.zeros(1, dtype=np.float32)
    bad = np.array([1, 1, 1, -1, 1, 1, 1, 1], dtype=np.float32)
    nan = np.array([1, 1, 1, np.nan, 1, 1, 1, 1], dtype=np.float32)
    assert h(w.ctypes.data, 1, 8, 8, None, out.ctypes.data, sc.ctypes.data) == NULL
    assert h(w.ctypes.data, 1, 8, 8, bad.ctypes.data, out.ctypes.data, sc.ctypes.data) == ARG
    assert h(w.ctypes.data, 1, 8, 8, nan.ctypes.data, out.ctypes.data, sc.ctypes.data) == ARG


def test_step_fold_device_and_dit_static_calls_reject_bad_arguments():
    lib = _lib.load()
    f = lib.oq_quantize_weights_step
    assert f(P16, 4, 1024, 1024, 1024, None, P16, P16, None) == NULL      # delta
    assert f(P16, 4, 1024, 1024, 1024, P4, P16, P16, None) == ALIGN       # delta 16-byte
    assert f(P16, 4, 1024, 1000, 1024, P16, P16, P16, None) == SHAPE      # ldw < K
    assert f(None, 0, 1024, 1024, 1024, None, None, None, None) == OK     # no rows
    s = lib.oq_dit_set_static_steps
    assert s(None, P16, None) == NULL
    assert lib.oq_dit_in_projection(None, P16, P16, None) == NULL
