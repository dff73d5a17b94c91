"""Each pin must reject a plausible mistake planted in a copy of the oracle
(CPU only; the mistakes live in this file, the oracle is untouched)."""
import numpy as np
import pytest

from oracle import hadamard, quant, linear
from tests import oracle_pins as P


def fwht_unnormalized(x, b):
    return hadamard.fwht(x, b) * np.sqrt(float(b))


def fwht_sign_swapped(x, b):
    x = np.asarray(x, np.float64)
    K = x.shape[-1]
    y = x.reshape(-1, K // b, b).copy()
    h = 1
    while h < b:
        y = y.reshape(y.shape[0], K // b, b // (2 * h), 2, h)
        u, v = y[:, :, :, 0, :].copy(), y[:, :, :, 1, :].copy()
        y[:, :, :, 0, :] = u - v
        y[:, :, :, 1, :] = u + v
        h *= 2
    return y.reshape(x.shape) / np.sqrt(b)


def fwht_skip_last_stage(x, b):
    if b <= 1:
        return np.asarray(x, np.float64)
    return hadamard.fwht(x, b // 2) * np.sqrt((b // 2) / b)


def quant_qmax8(z):
    return quant.quantize_sym(z, qmax=8)


def quant_floor(z):
    q, d, r = quant.quantize_sym(z)
    return np.clip(np.floor(r), -7, 7).astype(np.int64), d, r


def rq_scale_not_divided(x, b, s_t=1.0):
    q, xs, r = quant.rotate_quantize_act(x, b, s_t)
    return q, xs * s_t, r


def gemm_not_transposed(q, qw):
    return (np.asarray(q) @ np.asarray(qw)).astype(np.int64)


def dequant_no_wscale(acc, xs, ws, bias=None):
    return linear.dequant(acc, xs, np.ones_like(np.asarray(ws, np.float64)), bias)


def sylvester_wrong_sign(n):
    h = hadamard.sylvester(n).copy()
    if n > 1:
        h[-1, -1] *= -1
    return h


@pytest.mark.parametrize("check,impl", [
    (P.check_sylvester, sylvester_wrong_sign),
    (P.check_fwht_dense, fwht_unnormalized),
    (P.check_fwht_dense, fwht_sign_swapped),
    (P.check_fwht_dense, fwht_skip_last_stage),
    (P.check_fwht_closed_forms, fwht_unnormalized),
    (P.check_quantizer, quant_qmax8),
    (P.check_quantizer, quant_floor),
    (P.check_st_invariance, rq_scale_not_divided),
    (P.check_int_gemm, gemm_not_transposed),
    (P.check_dequant, dequant_no_wscale),
])
def test_pin_rejects_mutant(check, impl):
    with pytest.raises((AssertionError, ValueError)):
        check(impl)


def test_worked_example_rejects_qmax8():
    def rq(x, b, s_t=1.0):
        y = hadamard.fwht(x, b) * s_t
        q, d, r = quant.quantize_sym(y, qmax=8)
        return q, d / s_t, r
    with pytest.raises(AssertionError):
        P.check_worked_example_activation(rq)
