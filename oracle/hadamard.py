"""Hadamard rotation, oracle side (test infrastructure only).

Section 4.1, "Hadamard rotation": the composite rotation is R = R_SVD . H with
H the normalized Hadamard matrix, entries +-1/sqrt(n); eq:composite_rot.
Section 4.1, "Block-wise Implementation" (eq:blockdiag): the rotation is
applied as a block-diagonal matrix of c x c blocks over contiguous channels.

Reading used here: H_n is the Sylvester (natural-order) Hadamard matrix,
H[i][j] = (-1)^popcount(i & j), n a power of two; the block size b divides the
channel count and the rotation acts on each contiguous group of b channels.

Pins: H H^T = n I (exact, int64); a hand-typed H_8 fixture; the transform
equals a dense matmul with H for every n <= 64; involution, Parseval, spike
and constant-vector closed forms.
"""
from __future__ import annotations

import numpy as np


def is_pow2(n: int) -> bool:
    return n >= 1 and (n & (n - 1)) == 0


def sylvester(n: int) -> np.ndarray:
    """Unnormalized Sylvester Hadamard matrix of order n (int64), H[i][j] = (-1)^popcount(i&j)."""
    if not is_pow2(n):
        raise ValueError("Hadamard order must be a power of two")
    i = np.arange(n, dtype=np.int64)
    bits = np.bitwise_and(i[:, None], i[None, :])
    parity = np.zeros_like(bits)
    while np.any(bits):
        parity ^= bits & 1
        bits >>= 1
    return 1 - 2 * parity


def fwht(x: np.ndarray, b: int) -> np.ndarray:
    """Normalized block-diagonal Walsh-Hadamard transform along the last axis.

    Each contiguous group of b channels is multiplied by H_b / sqrt(b) (rows are
    tokens, so the group g of row i becomes x[i, g] . H_b / sqrt(b); H_b is
    symmetric).  Computed with the iterative butterfly (u, v) -> (u + v, u - v)
    over index bits 0 .. log2(b)-1, in float64.
    """
    x = np.asarray(x, dtype=np.float64)
    K = x.shape[-1]
    if not is_pow2(b) or K % b != 0:
        raise ValueError("block size must be a power of two dividing the channel count")
    lead = x.shape[:-1]
    y = x.reshape(-1, K // b, b).copy()
    h = 1
    while h < b:
        y = y.reshape(y.shape[0], K // b, b // (2 * h), 2, h)
        u = y[:, :, :, 0, :].copy()
        v = y[:, :, :, 1, :].copy()
        y[:, :, :, 0, :] = u + v
        y[:, :, :, 1, :] = u - v
        h *= 2
    y = y.reshape(lead + (K,))
    return y / np.sqrt(float(b))
