"""Seeded random generators shared by the oracle tests, the GPU tests and the bench.

Every tensor is drawn from its own PCG64 stream keyed by (config seed,
crc32(tensor name)), so adding a tensor never shifts the values of another.
Values are produced in float64 on the host; callers cast once (e.g. to fp16)
and feed the same cast buffer to both sides.
"""
from __future__ import annotations

import zlib

import numpy as np


def rng_for(seed: int, name: str) -> np.random.Generator:
    """Independent generator for tensor ``name`` of the workload seeded ``seed``."""
    ss = np.random.SeedSequence([int(seed), zlib.crc32(name.encode())])
    return np.random.Generator(np.random.PCG64(ss))


def gaussian(seed: int, name: str, shape, std: float = 1.0, mean: float = 0.0) -> np.ndarray:
    """float64 array ~ N(mean, std^2)."""
    rng = rng_for(seed, name)
    return rng.standard_normal(size=shape) * std + mean


def outlier_channels(seed: int, name: str, n_channels: int, n_outliers: int) -> np.ndarray:
    """``n_outliers`` distinct channel indices, uniformly chosen, sorted."""
    rng = rng_for(seed, name + "/outliers")
    n = int(min(max(n_outliers, 0), n_channels))
    return np.sort(rng.choice(n_channels, size=n, replace=False))


def with_outliers(x: np.ndarray, channels: np.ndarray, factor: float) -> np.ndarray:
    """Copy of ``x`` with the given last-axis channels multiplied by ``factor``."""
    y = np.array(x, dtype=np.float64, copy=True)
    y[..., channels] *= factor
    return y


def random_orthogonal(seed: int, name: str, n: int) -> np.ndarray:
    """Haar-distributed orthogonal n x n matrix: QR of a Gaussian, signs fixed by diag(R)."""
    a = gaussian(seed, name, (n, n))
    q, r = np.linalg.qr(a)
    return q * np.sign(np.diag(r))[None, :]


def log_uniform(seed: int, name: str, shape, lo: float, hi: float) -> np.ndarray:
    """float64 array, log-uniform on [lo, hi]."""
    rng = rng_for(seed, name)
    return np.exp(rng.uniform(np.log(lo), np.log(hi), size=shape))
