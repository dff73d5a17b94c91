"""Symmetric uniform quantization, oracle side (test infrastructure only).

Section 4.2, eq:scale and eq:quant: for bit width k, q_max = 2^(k-1) - 1 (7 for
int4); Delta = max|Z| / q_max; Q = clamp(round(Z / Delta), -q_max, q_max);
dequantized value Delta * Q.  Weights get one Delta per output channel,
backbone activations one Delta per token (text after eq:quant).

Per-step activation scale (eq:perstep_scale and the paragraph after it): the
DiT uses a per-(layer, step) scale.  Reading used here: the step scale s_t is a
scalar that multiplies the rotated activation before the per-token quantizer
and is divided back out of the reported token scale, x_scale = Delta / s_t.  In
exact arithmetic the codes and x_scale are then independent of s_t; a
test pins exactly that.

Rounding: round half to even (numpy.rint).  A row whose maximum magnitude is
0 gets Delta = 0 and all-zero codes (the division is not performed).

Pins: the quantizer error bound |z - Delta q| <= Delta/2, the absmax element
maps to +-q_max, no code equals -8, zero / spike / constant rows, a worked
example computed by hand, and the s_t invariance.
"""
from __future__ import annotations

import numpy as np

from .hadamard import fwht

QMAX4 = 7


def quantize_sym(z: np.ndarray, qmax: int = QMAX4):
    """Per-row (last axis) symmetric quantizer.

    Returns (q, delta, ratio): q int64 codes in [-qmax, qmax], delta float64
    per row, ratio = z / delta (float64, the value that is rounded; 0 for a
    zero row).
    """
    z = np.asarray(z, dtype=np.float64)
    a = np.max(np.abs(z), axis=-1)
    delta = a / float(qmax)
    nz = delta > 0
    safe = np.where(nz, delta, 1.0)
    ratio = np.where(nz[..., None], z / safe[..., None], 0.0)
    q = np.clip(np.rint(ratio), -qmax, qmax).astype(np.int64)
    return q, delta, ratio


def rotate_quantize_act(x: np.ndarray, b: int, s_t: float = 1.0):
    """Online rotation, step scale and per-token int4 quantization of an activation.

    x: [M, K] activation already in the U (SVD) basis, any float dtype (fp16
    inputs are converted exactly).  Steps: y = x . blockdiag(H_b)/sqrt(b)
    (eq:transform, eq:blockdiag); z = s_t * y; per-token quantizer (eq:scale,
    eq:quant).  Returns (q [M,K] int64, x_scale [M] = Delta/s_t, ratio [M,K]).
    """
    y = fwht(np.asarray(x, dtype=np.float64), b)
    s = float(s_t)
    z = s * y
    q, delta, ratio = quantize_sym(z)
    return q, delta / s, ratio


def quantize_weights(w_u: np.ndarray, b: int):
    """Fold the Hadamard half of the rotation into the weights and quantize them.

    w_u: [N, K] weight in the same (U) input basis as the activation.  The
    folded weight is W' = w_u . blockdiag(H_b)/sqrt(b) (eq:transform, W' row n
    = w_u row n rotated), quantized per output channel (row) with RTN (the
    DiT-side solver of the Implementation Details).  Returns
    (qw [N,K] int64, w_scale [N], ratio [N,K]).
    """
    wf = fwht(np.asarray(w_u, dtype=np.float64), b)
    return quantize_sym(wf)
