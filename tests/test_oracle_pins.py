"""The oracle against facts that do not come from the oracle: closed forms,
brute force, hand-worked fixtures and invariants (CPU only)."""
import numpy as np
import pytest

import oracle
from oracle import hadamard, quant, linear
from tests import oracle_pins as P
from workloads import configs, linear_inputs


def test_sylvester():
    P.check_sylvester(hadamard.sylvester)


def test_fwht_equals_dense_hadamard():
    P.check_fwht_dense(hadamard.fwht)


def test_fwht_closed_forms():
    P.check_fwht_closed_forms(hadamard.fwht)


def test_fwht_blockwise():
    P.check_fwht_blockwise(hadamard.fwht)


def test_fwht_rejects_bad_block():
    with pytest.raises(ValueError):
        hadamard.fwht(np.zeros((1, 96)), 64)
    with pytest.raises(ValueError):
        hadamard.fwht(np.zeros((1, 96)), 48)


def test_quantizer():
    P.check_quantizer(quant.quantize_sym)


def test_worked_example_activation():
    P.check_worked_example_activation(quant.rotate_quantize_act)


def test_worked_example_weight():
    P.check_worked_example_weight(quant.quantize_weights)


def test_st_invariance():
    P.check_st_invariance(quant.rotate_quantize_act)


def test_int_gemm():
    P.check_int_gemm(linear.int_gemm)
    P.check_worked_example_gemm(linear.int_gemm)


def test_dequant():
    P.check_dequant(linear.dequant)


def test_rotated_constant_row():
    """A constant row rotates to c sqrt(b) e_0 per block: one +-7, the rest 0."""
    x = np.full((1, 1024), 0.75)
    q, xs, _ = quant.rotate_quantize_act(x, 1024, 1.0)
    assert q[0, 0] == 7 and np.all(q[0, 1:] == 0)
    assert abs(xs[0] - 0.75 * 32 / 7) < 1e-14


def test_rotated_spike_row():
    """A single spike rotates to +-c/sqrt(b) everywhere: every code is +-7."""
    x = np.zeros((1, 256))
    x[0, 37] = -2.0
    q, xs, _ = quant.rotate_quantize_act(x, 256, 1.0)
    assert np.all(np.abs(q) == 7)
    assert abs(xs[0] - 2.0 / 16 / 7) < 1e-16


def test_rotation_invariance_fp64():
    """Section 4.1: Y = XW = (XR)(R^T W).  With the SVD factor U folded into the
    weight (w_u = w U) and the activation expressed in the U basis
    (x_tilde = X U), the Hadamard half leaves the product unchanged, and the
    product equals the unrotated X w^T."""
    case = configs.LINEAR_1024
    inp = linear_inputs.make_linear_inputs(case)
    X = inp["x"] @ inp["u"].T           # the unrotated activation
    w_u = inp["w"] @ inp["u"]
    b = case.had_block
    lhs = hadamard.fwht(inp["x"], b) @ hadamard.fwht(w_u, b).T
    rhs = X @ inp["w"].T
    assert np.linalg.norm(lhs - rhs) / np.linalg.norm(rhs) < 1e-12


def test_hadamard_spreads_outliers():
    """Information, not parity: on outlier-injected activations the rotation
    shrinks the per-token max/RMS ratio and the W4A4 error (the effect
    Section 4.1 and Fig. composite_rotation describe)."""
    case = configs.LINEAR_1024
    inp = linear_inputs.make_linear_inputs(case, with_u=False)
    x = inp["x"]
    ratio_raw = np.max(np.abs(x), 1) / np.sqrt(np.mean(x * x, 1))
    y = hadamard.fwht(x, 1024)
    ratio_rot = np.max(np.abs(y), 1) / np.sqrt(np.mean(y * y, 1))
    assert np.median(ratio_rot) < 0.5 * np.median(ratio_raw)
    ref = x @ inp["w"].T
    with_h = linear.w4a4_linear(x, inp["w"], 1024)["y"]
    q1, xs1, _ = quant.quantize_sym(x)
    qw1, ws1, _ = quant.quantize_sym(inp["w"])
    without_h = linear.dequant(linear.int_gemm(q1, qw1), xs1, ws1)
    nmse = lambda a: np.sum((a - ref) ** 2) / np.sum(ref ** 2)
    assert nmse(with_h) < 0.5 * nmse(without_h)


def test_oracle_header_says_test_only():
    assert "TEST INFRASTRUCTURE ONLY" in oracle.__doc__
