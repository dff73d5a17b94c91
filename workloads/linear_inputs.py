"""Seeded inputs of one rotated linear: activation (fp16 values, outlier
channels), weight, optional random orthogonal basis U and bias."""
from __future__ import annotations

import numpy as np

from .generators import gaussian, outlier_channels, random_orthogonal


def make_linear_inputs(case, with_u=None):
    """Returns dict: x [M,K] (fp16 values, in the U basis), w [N,K] (original
    weight), u [K,K] or None, bias [N] (fp16 values, zeros by default)."""
    M, K, N, sd = case.M, case.K, case.N, case.seed
    x = gaussian(sd, "x", (M, K))
    n_out = case.outlier_count if case.outlier_count else int(round(case.outlier_frac * K))
    x[:, outlier_channels(sd, "x", K, n_out)] *= case.outlier_factor
    x = x.astype(np.float16).astype(np.float64)
    w = gaussian(sd, "w", (N, K), case.w_std).astype(np.float16).astype(np.float64)
    use_u = case.fold_random_orthogonal if with_u is None else with_u
    u = random_orthogonal(sd, "u", K) if use_u else None
    return {"x": x, "w": w, "u": u, "bias": np.zeros(N)}
