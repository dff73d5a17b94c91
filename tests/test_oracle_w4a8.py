"""W4A8 in the oracle (CPU only): the 8-bit symmetric quantizer, a worked
example computed by hand, the rounding error bound, and mutants."""
import numpy as np
import pytest

from oracle import hadamard, linear, quant
from tests import oracle_pins as P


def test_quantizer_8bit():
    P.check_quantizer(lambda z: quant.quantize_sym(z, quant.QMAX8), qmax=127)


def test_w4a8_worked_example():
    P.check_w4a8_worked_example(linear.w4a8_linear)


def test_w4a8_error_bound():
    P.check_w4a8_error_bound(linear.w4a8_linear, hadamard.fwht)


def test_int_gemm_int8_range():
    """Extreme int8 x int4 magnitudes at K = 16384 are exact."""
    K = 16384
    q = np.full((2, K), 127, np.int64)
    q[1] = -127
    qw = np.full((1, K), -7, np.int64)
    assert np.array_equal(linear.int_gemm(q, qw), np.array([[-889 * K], [889 * K]]))
    q3 = np.random.default_rng(1).integers(-127, 128, size=(3, 40))
    qw3 = np.random.default_rng(2).integers(-7, 8, size=(5, 40))
    assert np.array_equal(linear.int_gemm(q3, qw3), P.triple_loop(q3, qw3))


def _w4a8_with(qmax_act):
    def f(x, w, b, s_t=1.0, bias=None, weights=None):
        q, xs, ratio = quant.rotate_quantize_act(x, b, s_t, qmax_act)
        qw, ws, _ = quant.quantize_weights(w, b)
        acc = linear.int_gemm(q, qw)
        return {"q": q, "x_scale": xs, "ratio": ratio, "qw": qw, "w_scale": ws, "acc": acc,
                "y": linear.dequant(acc, xs, ws, bias)}
    return f


def test_w4a8_mutants_rejected():
    # 4-bit activations, q_max = 128, and a sign error in the epilogue
    with pytest.raises(AssertionError):
        P.check_w4a8_worked_example(_w4a8_with(7))
    with pytest.raises(AssertionError):
        P.check_w4a8_error_bound(_w4a8_with(128), hadamard.fwht)

    def neg(x, w, b, s_t=1.0, bias=None, weights=None):
        r = linear.w4a8_linear(x, w, b, s_t)
        r["y"] = -r["y"]
        return r
    with pytest.raises(AssertionError):
        P.check_w4a8_error_bound(neg, hadamard.fwht)
    with pytest.raises(AssertionError):
        P.check_quantizer(lambda z: quant.quantize_sym(z, 128), qmax=127)
