"""Fused rotate + step-scale + int4 quantize kernel against the oracle (GPU).

Inputs are seeded Gaussian activations with outlier channels; the oracle is
fed the same fp16 values.  Codes must agree except at rounding boundaries
(within the fp32 error bound tau, at most 1e-4 of the elements), the
pre-rounding ratios must agree to tau element by element, and x_scale to the
same relative bound."""
import sys

import numpy as np
import pytest
import torch

import paper_2605_28803_amd as oq
from oracle import quant
from tests import parity
from workloads import generators as G

pytestmark = pytest.mark.gpu

CASES = [
    # (M, K, b, s_t)
    (1, 8, 8, 1.0), (3, 24, 8, 1.0), (5, 64, 64, 1.0), (7, 64, 1, 1.0), (9, 128, 32, 2.0),
    (33, 512, 512, 1.0), (64, 1024, 1024, 1.0), (50, 1024, 1024, 2.7), (37, 1536, 512, 0.8),
    (19, 2048, 2048, 1.0), (50, 4096, 4096, 0.6), (11, 6144, 2048, 3.9), (13, 8192, 8192, 1.0),
    (9, 16384, 16384, 1.3), (4, 16384, 64, 1.0), (5, 4096, 64, 1.0), (6, 12288, 4096, 1.0),
    (129, 2048, 256, 1.0),
    # rows spanning 2 or 4 waves with a partial block: transpose with one
    # wave stage, no transpose, and odd M (a half-valid workgroup)
    (7, 16384, 8192, 1.0), (5, 8192, 4096, 1.0), (3, 16384, 1024, 1.5), (257, 8192, 8192, 0.7),
    (301, 16384, 16384, 2.0), (1000, 4096, 4096, 1.0), (999, 1024, 256, 1.0),
    # more rows than one round of resident workgroups
    (6000, 4096, 4096, 1.0), (6001, 4096, 1024, 1.3), (1100, 8192, 8192, 1.0), (1030, 16384, 16384, 0.9),
    # four-wave rows over several rounds of resident workgroups (b = 4096 at
    # K = 16384: no wave transpose)
    (4000, 8192, 8192, 1.0), (2049, 16384, 16384, 0.7), (2500, 16384, 4096, 1.0),
    # three waves per row, one Hadamard block (or several) each: K = 1536 / 6144
    (1024, 1536, 512, 1.0), (1025, 6144, 2048, 1.7), (130, 6144, 64, 1.0), (3, 1536, 32, 2.0),
    # K = 4096 with at most 512 rows: two waves per row (odd M, the last
    # two-wave row count, one wave stage or none)
    (511, 4096, 4096, 1.1), (512, 4096, 2048, 0.9), (513, 4096, 4096, 1.0), (33, 4096, 128, 1.0),
]


def _x(M, K, seed, outliers=0.01, factor=50.0):
    x = G.gaussian(seed, "x", (M, K))
    x[:, G.outlier_channels(seed, "x", K, max(1, int(round(outliers * K))))] *= factor
    return x.astype(np.float16)


def _run(x16, b, s, ldx=None):
    M, K = x16.shape
    dev = torch.device("cuda:0")
    if ldx is None:
        X = torch.from_numpy(x16).to(dev)
    else:
        buf = torch.zeros((M, ldx), dtype=torch.float16, device=dev)
        buf[:, :K] = torch.from_numpy(x16).to(dev)
        X = buf[:, :K]
    st = np.array([s], dtype=np.float32)
    Xq, xs = oq.rotate_quantize_act(X, b, s_table=st, t=0)
    ratio, xs2 = oq.rotate_debug_f32(X, b, s_table=st, t=0)
    torch.cuda.synchronize()
    return Xq.cpu().numpy(), xs.cpu().numpy(), ratio.cpu().numpy(), xs2.cpu().numpy()


def _check(x16, b, s, Xq, xs, ratio, xs2):
    x = x16.astype(np.float64)
    s32 = float(np.float32(s))
    q_o, xs_o, r_o = quant.rotate_quantize_act(x, b, s32)
    tau = parity.tau_rows(x, b)
    q = parity.unpack_int4(Xq)
    n_mis, n_ulp = parity.check_codes(q, q_o, r_o, tau, r_gpu=ratio)
    assert np.all(np.abs(ratio - r_o) <= tau[:, None] + 1e-30), "pre-rounding ratio outside tau"
    rel = np.abs(xs.astype(np.float64) - xs_o) / np.where(xs_o > 0, xs_o, 1.0)
    assert np.all(rel <= tau / 7 + 4 * parity.U32)
    assert np.array_equal(xs, xs2)
    assert not np.any((Xq & 0xF) == 8) and not np.any((Xq >> 4) == 8)
    return n_mis, n_ulp


@pytest.mark.parametrize("M,K,b,s", CASES)
def test_rotate_quantize_parity(M, K, b, s):
    print(f"rq parity M={M} K={K} b={b} s={s}", flush=True)
    x16 = _x(M, K, seed=M * 7 + K)
    res = _run(x16, b, s)
    n_mis, n_ulp = _check(x16, b, s, *res)
    print(f"  mismatches={n_mis} within-1ulp={n_ulp} of {M * K}")


def test_rotate_quantize_strided_rows():
    x16 = _x(20, 1024, seed=11)
    res = _run(x16, 1024, 1.0, ldx=1096)
    _check(x16, 1024, 1.0, *res)


def test_rotate_quantize_special_rows():
    K = 2048
    x = np.zeros((4, K), dtype=np.float16)
    x[1, :] = 0.75                         # constant row -> one +-7, rest 0
    x[2, 100] = -3.0                       # spike -> every code +-7
    x[3, :] = _x(1, K, seed=3)[0]
    Xq, xs, ratio, xs2 = _run(x, K, 1.0)
    q = parity.unpack_int4(Xq)
    assert np.all(q[0] == 0) and xs[0] == 0.0
    assert q[1, 0] == 7 and np.all(q[1, 1:] == 0)
    assert np.all(np.abs(q[2]) == 7)
    _check(x, K, 1.0, Xq, xs, ratio, xs2)


def test_step_scale_invariance_on_gpu():
    """The step scale cancels: codes for s_t and for 1 agree except at boundaries."""
    x16 = _x(50, 4096, seed=5)
    a = _run(x16, 4096, 1.0)
    for s in (0.5, 2.25, 4.0):
        b_ = _run(x16, 4096, s)
        qa, qb = parity.unpack_int4(a[0]), parity.unpack_int4(b_[0])
        _, _, r_o = quant.rotate_quantize_act(x16.astype(np.float64), 4096, 1.0)
        tau = parity.tau_rows(x16.astype(np.float64), 4096)
        parity.check_codes(qb, qa, r_o, 2 * tau, record=False)
        assert np.allclose(a[1], b_[1], rtol=1e-5)


def test_empty_rows_is_noop():
    X = torch.zeros((0, 64), dtype=torch.float16, device="cuda:0")
    Xq, xs = oq.rotate_quantize_act(X, 64)
    assert Xq.shape == (0, 32)


def test_device_weight_quantization_matches_oracle():
    rng = np.random.default_rng(9)
    W = (rng.standard_normal((300, 1024)) * 0.02).astype(np.float16)
    Wq, ws = oq.quantize_weights(torch.from_numpy(W).cuda(), 1024)
    torch.cuda.synchronize()
    q_o, ws_o, r_o = quant.quantize_weights(W.astype(np.float64), 1024)
    tau = parity.tau_rows(W.astype(np.float64), 1024)
    parity.check_codes(parity.unpack_int4(Wq.cpu().numpy()), q_o, r_o, tau)
    assert np.allclose(ws.cpu().numpy(), ws_o, rtol=1e-5)


@pytest.mark.parametrize("M,K", [(16384, 16384), (16384, 4096), (65536, 1024)])
def test_rotate_quantize_full_size_sampled(M, K):
    """Full-size launch (the prefill / sweep shapes, b = K); sampled rows
    against the oracle on the same fp16 input."""
    print(f"rq full-size M={M} K={K}", flush=True)
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(M + K)
    X = torch.randn((M, K), generator=g, device=dev, dtype=torch.float32)
    ch = torch.randperm(K, generator=g, device=dev)[: max(1, K // 100)]
    X[:, ch] *= 50.0
    X = X.half()
    Xq, xs = oq.rotate_quantize_act(X, K)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.random.default_rng(K).choice(M, 48, replace=False), [0, M - 1]]))
    x16 = X[torch.from_numpy(rows).to(dev)].cpu().numpy()
    q_o, xs_o, r_o = quant.rotate_quantize_act(x16.astype(np.float64), K, 1.0)
    tau = parity.tau_rows(x16.astype(np.float64), K)
    q = parity.unpack_int4(Xq[torch.from_numpy(rows).to(dev)].cpu().numpy())
    n_mis, _ = parity.check_codes(q, q_o, r_o, tau)
    xs_g = xs[torch.from_numpy(rows).to(dev)].cpu().numpy().astype(np.float64)
    assert np.all(np.abs(xs_g - xs_o) <= (tau / 7 + 4 * parity.U32) * xs_o)
    print(f"  sampled {len(rows)} rows: mismatches={n_mis}")
