"""The composite-rotation oracle against facts outside it (CPU only)."""
import numpy as np

from oracle import composite, hadamard, quant
from tests import oracle_pins as P


def test_zigzag():
    P.check_zigzag(composite.zigzag_permutation)


def test_block_svd_row_energy():
    P.check_block_svd(composite.block_svd_factors)


def test_block_rotations():
    P.check_block_rotations(composite.block_rotations)


def test_rotate_composite():
    P.check_rotate_composite(composite.rotate_composite, composite.block_rotations, hadamard.fwht)


def test_rotate_quantize_composite():
    P.check_rotate_quantize_composite(composite.rotate_quantize_composite, quant.rotate_quantize_act)


def test_channel_energy_is_column_sum_of_squares():
    w = np.arange(12, dtype=np.float64).reshape(3, 4)
    assert np.array_equal(composite.channel_energy(w), np.array([0 + 16 + 64, 1 + 25 + 81, 4 + 36 + 100,
                                                                 9 + 49 + 121], dtype=np.float64))


def test_full_pipeline_invariance_from_svd():
    """perm from column energies, U_b from the SVD, R_b = U_b H / 8: the folded
    linear reproduces X W^T (float64)."""
    rng = np.random.default_rng(30)
    M, N, K, c = 8, 48, 256, 64
    w = rng.standard_normal((N, K)) * 0.02
    w[:, rng.choice(K, 4, replace=False)] *= 30
    x = rng.standard_normal((M, K))
    perm = composite.zigzag_permutation(composite.channel_energy(w), K // c)
    u, _ = composite.block_svd_factors(w, perm, c)
    r = composite.block_rotations(u)
    lhs = composite.rotate_composite(x, perm, r) @ composite.rotate_composite(w, perm, r).T
    ref = x @ w.T
    assert np.max(np.abs(lhs - ref)) <= 1e-12 * np.max(np.abs(ref)) * K


def test_canonical_signs():
    P.check_canonical_signs(composite.canonical_signs)


def test_canonical_signs_mutants_rejected():
    import pytest

    def by_first_entry(u):  # sign of the first entry instead of the largest
        u = np.array(u, dtype=np.float64, copy=True)
        mats = u if u.ndim == 3 else u[None]
        for m in mats:
            for j in range(m.shape[1]):
                if m[0, j] < 0:
                    m[:, j] = -m[:, j]
        return u

    def last_on_ties(u):
        u = np.array(u, dtype=np.float64, copy=True)
        mats = u if u.ndim == 3 else u[None]
        for m in mats:
            for j in range(m.shape[1]):
                a = np.abs(m[:, j])
                r = len(a) - 1 - int(np.argmax(a[::-1]))
                if m[r, j] < 0:
                    m[:, j] = -m[:, j]
        return u
    with pytest.raises(AssertionError):
        P.check_canonical_signs(by_first_entry)
    with pytest.raises(AssertionError):
        P.check_canonical_signs(last_on_ties)
