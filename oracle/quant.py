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

The paper's own deployment mode is W4A8 (4-bit weights, 8-bit per-token
activations): the same quantizer with k = 8, q_max = 127, for the activation.

Pins: the quantizer error bound |z - Delta q| <= Delta/2, the absmax element
maps to +-q_max, no code equals -8, zero / spike / constant rows, a worked
example computed by hand (one for W4A4, one for W4A8), and the s_t
invariance.
"""
from __future__ import annotations

import numpy as np

from .hadamard import fwht

QMAX4 = 7
QMAX8 = 127


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


def rotate_quantize_act(x: np.ndarray, b: int, s_t: float = 1.0, qmax: int = QMAX4):
    """Online rotation, step scale and per-token int4 quantization of an activation.

    x: [M, K] activation already in the U (SVD) basis, any float dtype (fp16
    inputs are converted exactly).  Steps: y = x . blockdiag(H_b)/sqrt(b)
    (eq:transform, eq:blockdiag); z = s_t * y; per-token quantizer (eq:scale,
    eq:quant) with q_max = qmax (7 for int4, 127 for the 8-bit activations of
    W4A8).  Returns (q [M,K] int64, x_scale [M] = Delta/s_t, ratio [M,K]).
    """
    y = fwht(np.asarray(x, dtype=np.float64), b)
    s = float(s_t)
    z = s * y
    q, delta, ratio = quantize_sym(z, qmax)
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


# ---------------------------------------------------------------------------
# Per-step static activation scales (eq:perstep_scale, the per-(layer, step,
# channel) table of the paper's text).  Reading: sigma_hat is the 99.9th
# percentile of the magnitudes of the rotated activation over the calibration
# rows (nearest rank: the k-th smallest |y| with k = ceil(p n / 100), p to
# 1e-6 percent so that k is exact), Delta_j =
# sigma_hat_j / q_max, and at inference q = clamp(round(y_j / Delta_j), -7, 7)
# with the table in place of the per-token maximum (clipping is live).  The
# per-channel step cannot be factored out of the sum over channels, so it is
# folded into the weight's input channels: W''[n][j] = W'[n][j] Delta_j,
# quantized per output channel; the token scale is then 1.
# ---------------------------------------------------------------------------

def nearest_rank(p: float, n: int) -> int:
    """k = ceil(p n / 100) clamped to [1, n], with p taken to a resolution of
    1e-6 percent so that the product is formed exactly in integers: p = 99.9
    and n = 1000 give k = 999 (the float product 99.9 / 100 * 1000 is
    999.0000000000001, whose ceiling would be the maximum)."""
    pm = int(round(float(p) * 1e6))  # p in units of 1e-6 percent
    k = -(-(pm * int(n)) // 10 ** 8)
    return min(max(k, 1), int(n))


def percentile_abs(y: np.ndarray, p: float) -> np.ndarray:
    """Nearest-rank p-th percentile of |y| over rows, per column (float64 [K])."""
    a = np.abs(np.asarray(y, dtype=np.float64))
    n = a.shape[0]
    k = nearest_rank(p, n)
    return np.sort(a, axis=0)[k - 1]


def calibrate_step_scales(y: np.ndarray, p: float = 99.9, qmax: int = QMAX4) -> np.ndarray:
    """Delta_j = percentile_abs(y, p) / q_max for the rotated calibration rows y [n, K]."""
    return percentile_abs(y, p) / float(qmax)


def quantize_static(y: np.ndarray, delta: np.ndarray, qmax: int = QMAX4):
    """Codes with a static per-channel step: q = clamp(round(y / Delta_j), -q_max, q_max);
    a channel with Delta_j = 0 gets code 0.  Returns (q, ratio)."""
    y = np.asarray(y, dtype=np.float64)
    d = np.asarray(delta, dtype=np.float64)
    nz = d > 0
    ratio = np.where(nz[None, :], y / np.where(nz, d, 1.0)[None, :], 0.0)
    q = np.clip(np.rint(ratio), -qmax, qmax).astype(np.int64)
    return q, ratio


def rotate_quantize_static(x: np.ndarray, b: int, delta: np.ndarray):
    """Hadamard rotation (as rotate_quantize_act) followed by the static
    per-channel quantizer; token scale 1.  Returns (q, x_scale, ratio)."""
    y = fwht(np.asarray(x, dtype=np.float64), b)
    q, ratio = quantize_static(y, delta)
    return q, np.ones(y.shape[0]), ratio


def fold_weights_step(w_u: np.ndarray, b: int, delta: np.ndarray):
    """W' = rotated weight (as quantize_weights), W'' = W' diag(Delta), per-row RTN."""
    wf = fwht(np.asarray(w_u, dtype=np.float64), b) * np.asarray(delta, dtype=np.float64)[None, :]
    return quantize_sym(wf)
