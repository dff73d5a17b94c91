"""Low-bit linear, oracle side (test infrastructure only).

eq:lowbit_linear: X'W' ~= Delta_X' Delta_W' Q_X' Q_W' -- an integer product of
the codes scaled by the per-token and per-output-channel steps; the
Implementation Details fold all scales into the dequantization.  With the
weight stored [N x K] (output channel major) the product is
acc[i, n] = sum_k q[i, k] * qw[n, k], and y[i, n] = x_scale[i] * w_scale[n] *
acc[i, n] (+ bias[n]).

The integer product is evaluated as a float64 matrix product of the integer
codes.  That is exact: every product and every partial sum is an integer of
magnitude at most max|q| max|qw| K (49 K for W4A4, 889 K for W4A8) < 2^53,
and float64 adds such integers without rounding in any order.  Pins: an int64 triple loop on tiny shapes, +-identity
and all-ones weights, and unit-scale epilogue.
"""
from __future__ import annotations

import numpy as np

from .quant import QMAX8, rotate_quantize_act, quantize_weights


def int_gemm(q: np.ndarray, qw: np.ndarray) -> np.ndarray:
    """acc[i, n] = sum_k q[i, k] * qw[n, k], exact, int64."""
    q = np.asarray(q)
    qw = np.asarray(qw)
    if q.shape[-1] != qw.shape[-1]:
        raise ValueError("inner dimensions differ")
    K = q.shape[-1]
    mq = int(np.max(np.abs(q))) if q.size else 0
    mw = int(np.max(np.abs(qw))) if qw.size else 0
    if mq * mw * K >= 2 ** 53:
        raise ValueError("K too large for exact float64 accumulation")
    acc = q.astype(np.float64) @ qw.astype(np.float64).T
    out = acc.astype(np.int64)
    assert np.array_equal(out.astype(np.float64), acc)
    return out


def dequant(acc: np.ndarray, x_scale: np.ndarray, w_scale: np.ndarray, bias=None) -> np.ndarray:
    """y[i, n] = x_scale[i] * w_scale[n] * acc[i, n] + bias[n], float64."""
    y = np.asarray(acc, dtype=np.float64) * np.asarray(x_scale, np.float64)[:, None] \
        * np.asarray(w_scale, np.float64)[None, :]
    if bias is not None:
        y = y + np.asarray(bias, dtype=np.float64)[None, :]
    return y


def w4a4_linear(x: np.ndarray, w_u: np.ndarray, b: int, s_t: float = 1.0, bias=None,
                weights=None):
    """Rotated W4A4 linear: rotate + step-scale + quantize the activation,
    quantize the folded weight (or take ``weights`` = (qw, w_scale) already
    quantized), integer product, dequantize.  Returns a dict of every
    intermediate."""
    q, xs, ratio = rotate_quantize_act(x, b, s_t)
    if weights is None:
        qw, ws, wratio = quantize_weights(w_u, b)
    else:
        qw, ws = weights
        wratio = None
    acc = int_gemm(q, qw)
    y = dequant(acc, xs, ws, bias)
    return {"q": q, "x_scale": xs, "ratio": ratio, "qw": qw, "w_scale": ws,
            "wratio": wratio, "acc": acc, "y": y}


def w4a8_linear(x: np.ndarray, w_u: np.ndarray, b: int, s_t: float = 1.0, bias=None, weights=None):
    """Rotated W4A8 linear: as w4a4_linear with the activation quantized per
    token to 8 bits (q_max = 127); the weight stays int4.  Returns a dict of
    every intermediate."""
    q, xs, ratio = rotate_quantize_act(x, b, s_t, QMAX8)
    if weights is None:
        qw, ws, wratio = quantize_weights(w_u, b)
    else:
        qw, ws = weights
        wratio = None
    acc = int_gemm(q, qw)
    y = dequant(acc, xs, ws, bias)
    return {"q": q, "x_scale": xs, "ratio": ratio, "qw": qw, "w_scale": ws,
            "wratio": wratio, "acc": acc, "y": y}
