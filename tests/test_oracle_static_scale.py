"""Per-step static scale table (eq:perstep_scale, per-channel form) in the oracle (CPU only)."""
import numpy as np
import pytest

from oracle import hadamard, quant
from tests import oracle_pins as P


def test_percentile():
    P.check_percentile(quant.percentile_abs)


def test_quantize_static():
    P.check_quantize_static(quant.quantize_static)


def test_fold_step():
    P.check_fold_step(quant.fold_weights_step, hadamard.fwht)


def test_rotate_quantize_static_uses_the_rotation():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((4, 64))
    d = np.full(64, 0.3)
    q, xs, r = quant.rotate_quantize_static(x, 64, d)
    assert np.array_equal(xs, np.ones(4))
    # a spike rotates to a constant magnitude |c| / 8 in every channel
    x = np.zeros((1, 64))
    x[0, 5] = 8 * 0.3 * 2
    q, _, _ = quant.rotate_quantize_static(x, 64, d)
    assert np.all(np.abs(q) == 2)


def test_static_pins_reject_mutants():
    def pct_wrong_rank(y, p):
        a = np.sort(np.abs(np.asarray(y, np.float64)), axis=0)
        n = a.shape[0]
        k = min(max(int(np.floor(p / 100.0 * n)), 1), n)  # floor instead of ceil
        return a[k - 1] if n > 1 else a[0]

    def qs_no_clip(y, d):
        y = np.asarray(y, np.float64)
        return np.rint(y / np.where(d > 0, d, 1)[None, :]) * (d > 0)[None, :], None

    def fold_rows(w, b, d):
        wf = hadamard.fwht(w, b) * np.asarray(d)[: w.shape[0], None] if w.shape[0] <= len(d) else None
        return quant.quantize_sym(wf)

    def pct_float_rank(y, p):
        # the rank formed in floating point: 99.9 / 100 * 1000 = 999.0000000000001 -> 1000
        a = np.sort(np.abs(np.asarray(y, np.float64)), axis=0)
        n = a.shape[0]
        return a[min(max(int(np.ceil(p / 100.0 * n)), 1), n) - 1]

    with pytest.raises(AssertionError):
        P.check_percentile(pct_wrong_rank)
    with pytest.raises(AssertionError):
        P.check_percentile(pct_float_rank)
    with pytest.raises(AssertionError):
        P.check_quantize_static(qs_no_clip)
    with pytest.raises((AssertionError, ValueError, TypeError)):
        P.check_fold_step(fold_rows, hadamard.fwht)
