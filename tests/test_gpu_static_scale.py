"""Static per-step, per-channel activation steps on the GPU against the oracle
(eq:perstep_scale with the per-channel table, eq:quant with clipping).

  * oq_rotate_act_f32: the fp32 rotated activation within the elementwise
    rounding bound of the exact transform;
  * oq_calibrate_step_scales: the order statistic is exact, so the steps
    are compared bit for bit with the oracle's nearest-rank percentile of the
    same fp32 input (divided by q_max in double, rounded once);
  * oq_rotate_quantize_act_static(_tiled): codes bit-exact except at rounding
    boundaries within the bound tau_static, token scale exactly 1;
  * the static linear: GPU codes x the host-folded per-step weight through
    oq_w4a4_linear against the oracle fed the same codes (2e-3 relative L2).
"""
import numpy as np
import pytest
import torch

import paper_2605_28803_amd as oq
from oracle import hadamard, linear, quant
from tests import parity
from tests.test_gpu_tiled import untile_np
from workloads import generators as G

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _x(seed, M, K, outlier_frac=0.01, factor=50.0):
    x = G.gaussian(seed, "x", (M, K))
    x[:, G.outlier_channels(seed, "x", K, max(1, int(round(outlier_frac * K))))] *= factor
    return x.astype(np.float16)


ROT_CASES = [
    # matrix-core layouts (b >= 32, K in the compiled set) and the VALU layouts
    (50, 1024, 1024), (64, 4096, 4096), (33, 16384, 16384), (20, 8192, 4096), (7, 1536, 512),
    (50, 1024, 8), (5, 128, 64), (17, 6144, 2048), (130, 1024, 1024), (3, 384, 128),
]


@pytest.mark.parametrize("M,K,b", ROT_CASES)
def test_rotate_act_f32(M, K, b):
    print(f"rotate_act_f32 M={M} K={K} b={b}", flush=True)
    x16 = _x(8000 + M + K, M, K)
    Y = oq.rotate_act_f32(torch.from_numpy(x16).to(DEV), b)
    torch.cuda.synchronize()
    y = Y.cpu().numpy().astype(np.float64)
    ref = hadamard.fwht(x16.astype(np.float64), b)
    err = np.abs(y - ref)
    tau = parity.tau_rotate(x16, b, ref)
    assert np.all(err <= tau), f"max err/tau {np.max(err / np.maximum(tau, 1e-300)):.3g}"


def _quantile_ref(y32, p, qmax):
    v = quant.percentile_abs(y32.astype(np.float64), p)
    return v, (v / qmax).astype(np.float32)


QUANT_CASES = [
    # (n, K, p): single row, tiny odd n, exact-integer ranks, ragged column
    # slabs, more rows than one chunk, several chunks per slab
    (1, 64, 99.9), (7, 100, 50.0), (1000, 1024, 99.9), (1001, 1536, 99.9), (4099, 4160, 99.9),
    (30000, 1024, 99.9), (513, 256, 100.0), (777, 128, 0.01), (2000, 2048, 37.5),
]


@pytest.mark.parametrize("n,K,p", QUANT_CASES)
def test_calibrate_exact_order_statistic(n, K, p):
    print(f"calibrate n={n} K={K} p={p}", flush=True)
    rng = np.random.default_rng(n * 7 + K)
    y = (rng.standard_normal((n, K)) * np.exp(rng.standard_normal(K))[None, :]).astype(np.float32)
    # ties, zeros, negative zero, a constant column, a column of one repeated magnitude
    y[rng.integers(0, n, size=n // 3 + 1), rng.integers(0, K, size=n // 3 + 1)] = 0.0
    y[:, 3 % K] = -0.0
    y[:, 5 % K] = 2.5
    y[::2, 7 % K] = -1.25
    y[1::2, 7 % K] = 1.25
    Y = torch.from_numpy(y).to(DEV)
    d1 = oq.calibrate_step_scales(Y, p=p, qmax=1.0)
    d7 = oq.calibrate_step_scales(Y, p=p, qmax=7.0)
    torch.cuda.synchronize()
    v, d7_ref = _quantile_ref(y, p, 7.0)
    assert np.array_equal(d1.cpu().numpy().astype(np.float64), v)
    assert np.array_equal(d7.cpu().numpy(), d7_ref)


@pytest.mark.parametrize("n,p,k", [(1000, 99.9, 999), (2000, 99.9, 1998), (10000, 99.9, 9990), (1001, 99.9, 1000)])
def test_calibrate_literal_rank(n, p, k):
    """Columns holding the magnitudes 1..n in random orders and signs: the
    nearest rank worked by hand selects the value k (never the maximum when
    p n / 100 is whole)."""
    print(f"calibrate literal rank n={n} p={p}", flush=True)
    rng = np.random.default_rng(n)
    y = np.stack([(rng.permutation(n) + 1.0) * np.where(rng.random(n) < 0.5, -1.0, 1.0) for _ in range(64)], axis=1)
    Y = torch.from_numpy(y.astype(np.float32)).to(DEV)
    d = oq.calibrate_step_scales(Y, p=p, qmax=1.0)
    torch.cuda.synchronize()
    assert np.array_equal(d.cpu().numpy(), np.full(64, float(k), np.float32))


def test_calibrate_strided_rows_and_repeat_calls():
    """Y with ldy > K (a column slice of a wider buffer); the workspace is
    reused by a second call of another size."""
    rng = np.random.default_rng(77)
    big = rng.standard_normal((3000, 1100)).astype(np.float32)
    Yb = torch.from_numpy(big).to(DEV)
    work = torch.empty((oq.calibrate_workspace_bytes(1024),), dtype=torch.uint8, device=DEV)
    d = oq.calibrate_step_scales(Yb[:, :1024], 99.9, 7.0, work=work)
    d2 = oq.calibrate_step_scales(Yb[:500, 64:576], 99.0, 7.0, work=work)
    torch.cuda.synchronize()
    assert np.array_equal(d.cpu().numpy(), _quantile_ref(big[:, :1024], 99.9, 7.0)[1])
    assert np.array_equal(d2.cpu().numpy(), _quantile_ref(big[:500, 64:576], 99.0, 7.0)[1])


def test_calibration_pipeline_against_exact_rotation():
    """fp16 activations -> GPU rotation -> GPU steps equal the oracle's
    percentile of the GPU's fp32 rotation exactly, and the exact rotation's
    percentile within the rotation's rounding bound."""
    n, K, b = 4000, 1024, 1024
    x16 = _x(8100, n, K)
    Y = oq.rotate_act_f32(torch.from_numpy(x16).to(DEV), b)
    d = oq.calibrate_step_scales(Y, 99.9, 7.0)
    torch.cuda.synchronize()
    y = Y.cpu().numpy()
    assert np.array_equal(d.cpu().numpy(), _quantile_ref(y, 99.9, 7.0)[1])
    ref = hadamard.fwht(x16.astype(np.float64), b)
    v_exact = quant.percentile_abs(ref, 99.9)
    # an order statistic moves by at most the largest elementwise error
    tau = parity.tau_rotate(x16, b, ref).max()
    assert np.all(np.abs(d.cpu().numpy().astype(np.float64) * 7.0 - v_exact) <= tau + 4 * parity.U32 * v_exact)


def _steps(seed, x_calib16, b, shrink=1.0):
    """Delta from the oracle's exact calibration, optionally shrunk (more
    clipping), with a zero, an infinite and a NaN entry."""
    d = quant.calibrate_step_scales(hadamard.fwht(x_calib16.astype(np.float64), b), 99.9) * shrink
    d = d.astype(np.float32)
    rng = np.random.default_rng(seed)
    K = d.shape[0]
    i = rng.choice(K, 3, replace=False)
    d[i[0]], d[i[1]], d[i[2]] = 0.0, np.inf, np.nan
    return d


@pytest.mark.parametrize("M,K,b", ROT_CASES)
@pytest.mark.parametrize("shrink", [1.0, 0.25])
def test_rotate_quantize_static(M, K, b, shrink):
    print(f"static rq M={M} K={K} b={b} shrink={shrink}", flush=True)
    x16 = _x(8200 + M + K, M, K)
    d = _steps(K + b, _x(8300 + K, 256, K), b, shrink)
    X = torch.from_numpy(x16).to(DEV)
    D = torch.from_numpy(d).to(DEV)
    Xq, xs = oq.rotate_quantize_act_static(X, b, D)
    torch.cuda.synchronize()
    q = parity.unpack_int4(Xq.cpu().numpy())
    assert np.array_equal(xs.cpu().numpy(), np.ones(M, dtype=np.float32))
    dd = d.astype(np.float64)
    q_o, _, r_o = quant.rotate_quantize_static(x16.astype(np.float64), b, dd)
    n, _ = parity.check_codes(q, q_o, r_o, parity.tau_static(x16, b, dd, r_o))
    clipped = int(np.count_nonzero(np.abs(r_o) > 7.5))
    print(f"mismatches={n} clipped={clipped} of {q.size}")
    if shrink < 1.0:
        assert clipped > 0
    if K % 128 == 0:
        Xt, xst = oq.rotate_quantize_act_static_tiled(X, b, D)
        torch.cuda.synchronize()
        assert np.array_equal(untile_np(Xt.cpu().numpy(), M, K), Xq.cpu().numpy())
        assert np.array_equal(xst.cpu().numpy(), xs.cpu().numpy())


@pytest.mark.parametrize("M,N,K,b", [(50, 1024, 1024, 1024), (50, 3072, 1024, 1024), (64, 1024, 4096, 4096),
                                     (200, 512, 1536, 512)])
def test_static_linear(M, N, K, b):
    """Static codes x the per-step folded weight, through the product and
    epilogue, against the oracle fed the same codes; also the float
    linear's quality (informational)."""
    print(f"static linear M={M} N={N} K={K} b={b}", flush=True)
    x16 = _x(8400 + M + N, M, K)
    w = G.gaussian(8400 + N, "w", (N, K), std=0.02)
    d = quant.calibrate_step_scales(hadamard.fwht(_x(8500 + K, 512, K).astype(np.float64), b), 99.9)
    d32 = d.astype(np.float32)
    Wq, ws = oq.quantize_weights_step_host(w, b, d32)
    X = torch.from_numpy(x16).to(DEV)
    Xq, xs = oq.rotate_quantize_act_static(X, b, torch.from_numpy(d32).to(DEV))
    Y = oq.w4a4_linear(Xq, xs, torch.from_numpy(Wq).to(DEV), torch.from_numpy(ws).to(DEV))
    torch.cuda.synchronize()
    q = parity.unpack_int4(Xq.cpu().numpy())
    qw = parity.unpack_int4(Wq)
    ref = linear.dequant(linear.int_gemm(q, qw), np.ones(M), ws.astype(np.float64), None)
    err = parity.rel_l2(Y.float().cpu().numpy(), ref)
    exact = x16.astype(np.float64) @ w.T
    qual = parity.rel_l2(Y.float().cpu().numpy(), exact)
    print(f"static linear rel_l2 vs oracle {err:.2e}, vs float linear {qual:.3f}")
    assert err <= parity.REL_L2_OUT
    assert np.isfinite(qual) and qual < 1.0


@pytest.mark.parametrize("N,K,b", [(96, 1024, 1024), (3072, 1024, 1024), (1024, 4096, 4096), (200, 1536, 512),
                                   (33, 256, 8)])
def test_quantize_weights_step_device(N, K, b):
    """The device fold W' diag(Delta) + RTN against the oracle's fold of the
    same fp16 weight: codes by the boundary rule, scales to the fp32 bound."""
    print(f"weight step fold N={N} K={K} b={b}", flush=True)
    rng = np.random.default_rng(N + K)
    w16 = (rng.standard_normal((N, K)) * 0.02).astype(np.float16)
    d = np.exp(rng.standard_normal(K) * 0.5).astype(np.float32)
    d[rng.choice(K, 2, replace=False)] = 0.0
    Wq, ws = oq.quantize_weights_step(torch.from_numpy(w16).to(DEV), b, torch.from_numpy(d).to(DEV))
    torch.cuda.synchronize()
    qo, wso, ro = quant.fold_weights_step(w16.astype(np.float64), b, d.astype(np.float64))
    tau = parity.tau_rows_scaled(w16, b, d)
    parity.check_codes(parity.unpack_int4(Wq.cpu().numpy()), qo, ro, tau)
    assert np.allclose(ws.cpu().numpy(), wso, rtol=1e-5, atol=0)
