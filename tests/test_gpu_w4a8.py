"""W4A8 on the GPU against the oracle: 8-bit per-token activation codes
(eq:scale, eq:quant at k = 8) against the int4 weights.

  * oq_rotate_quantize_act_i8: codes bit-exact except at rounding boundaries
    within tau (the W4A4 bound with q_max = 127), x_scale within 1e-6;
  * oq_w4a8_gemm_i32: int32 accumulators bit-exact against the oracle's
    integer product, including |acc| = 889 K at K = 16384;
  * oq_w4a8_linear: outputs within 2e-3 relative L2 of the oracle fed the
    same codes, fp16 and bf16, both GEMM tilings, ragged edges;
  * the whole W4A8 linear against the oracle's, and its error below the
    W4A4 linear's on the same inputs (informational quality check).
"""
import numpy as np
import pytest
import torch

import paper_2605_28803_amd as oq
from oracle import linear, quant
from tests import parity
from workloads import generators as G

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _x(seed, M, K):
    x = G.gaussian(seed, "x", (M, K))
    x[:, G.outlier_channels(seed, "x", K, max(1, int(round(0.01 * K))))] *= 50.0
    return x.astype(np.float16)


RQ_CASES = [
    (50, 1024, 1024, 1.0), (64, 4096, 4096, 2.37), (33, 16384, 16384, 0.5), (20, 8192, 4096, 1.0),
    (7, 1536, 512, 1.0), (50, 1024, 8, 1.0), (5, 128, 64, 4.0), (17, 6144, 2048, 1.0), (130, 1024, 1024, 1.0),
    (3, 384, 128, 1.0),
]


@pytest.mark.parametrize("M,K,b,s", RQ_CASES)
def test_rotate_quantize_i8(M, K, b, s):
    print(f"rotate_quantize_i8 M={M} K={K} b={b} s={s}", flush=True)
    x16 = _x(9000 + M + K, M, K)
    st = np.array([s], dtype=np.float32)
    Xq8, xs = oq.rotate_quantize_act_i8(torch.from_numpy(x16).to(DEV), b, s_table=st, t=0)
    torch.cuda.synchronize()
    q = Xq8.cpu().numpy().astype(np.int64)
    q_o, xs_o, r_o = quant.rotate_quantize_act(x16.astype(np.float64), b, float(np.float32(s)), quant.QMAX8)
    n, _ = parity.check_codes(q, q_o, r_o, parity.tau_rows(x16, b, 127), qmax=127)
    assert np.allclose(xs.cpu().numpy(), xs_o, rtol=1e-6, atol=0)
    assert q.min() >= -127 and np.abs(q).max() == 127


GEMM_CASES = [
    # small-M tilings (M <= 64), the 128 x 128 tiling (M > 64), ragged N and
    # M, K % 128 == 64 tails, deep K
    (1, 2560, 2048), (16, 2048, 16384), (17, 200, 2048), (50, 3072, 1024), (50, 8192, 1024),
    (64, 520, 4160), (3, 100, 64), (65, 320, 1536), (130, 1000, 1024), (256, 4096, 4096),
    (1000, 2048, 2112), (50, 1024, 4096),
]


@pytest.mark.parametrize("M,N,K", GEMM_CASES)
def test_w4a8_gemm_i32_bit_exact(M, N, K):
    print(f"w4a8 gemm M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M * 13 + N * 3 + K)
    q, qw = rng.integers(-127, 128, size=(M, K)), rng.integers(-7, 8, size=(N, K))
    acc = oq.w4a8_gemm_i32(torch.from_numpy(q.astype(np.int8)).to(DEV), torch.from_numpy(parity.pack_int4(qw)).to(DEV))
    torch.cuda.synchronize()
    assert np.array_equal(acc.cpu().numpy().astype(np.int64), linear.int_gemm(q, qw))


@pytest.mark.parametrize("M", [3, 200])
def test_w4a8_gemm_extreme_magnitudes(M):
    """Every code at its extreme at K = 16384: |acc| = 889 K."""
    K = 16384
    q = np.full((M, K), 127)
    q[1] = -127
    q[2, ::2] = -127
    qw = np.full((4, K), 7)
    qw[1] = -7
    qw[2, 1::2] = -7
    acc = oq.w4a8_gemm_i32(torch.from_numpy(q.astype(np.int8)).to(DEV), torch.from_numpy(parity.pack_int4(qw)).to(DEV))
    acc = acc.cpu().numpy().astype(np.int64)
    assert np.array_equal(acc, linear.int_gemm(q, qw))
    assert acc[0, 0] == 889 * K and acc[1, 0] == -889 * K


@pytest.mark.parametrize("out_dtype", [oq.OUT_F16, oq.OUT_BF16])
@pytest.mark.parametrize("M,N,K", [(50, 1024, 1024), (9, 1000, 4096), (70, 256, 2048), (512, 2048, 1024)])
def test_w4a8_linear_epilogue(M, N, K, out_dtype):
    print(f"w4a8 linear M={M} N={N} K={K} out={out_dtype}", flush=True)
    rng = np.random.default_rng(M * N + K + out_dtype)
    q, qw = rng.integers(-127, 128, size=(M, K)), rng.integers(-7, 8, size=(N, K))
    xs = rng.uniform(0.001, 0.1, M).astype(np.float32)
    ws = rng.uniform(1e-4, 1e-2, N).astype(np.float32)
    bias = (rng.standard_normal(N) * 0.1).astype(np.float16)
    Y = oq.w4a8_linear(torch.from_numpy(q.astype(np.int8)).to(DEV), torch.from_numpy(xs).to(DEV),
                       torch.from_numpy(parity.pack_int4(qw)).to(DEV), torch.from_numpy(ws).to(DEV),
                       bias=torch.from_numpy(bias).to(DEV), out_dtype=out_dtype)
    ref = linear.dequant(linear.int_gemm(q, qw), xs, ws, bias.astype(np.float64))
    err = parity.rel_l2(Y.float().cpu().numpy(), ref)
    assert err <= parity.REL_L2_OUT


@pytest.mark.parametrize("M,N,K,b", [(50, 1024, 1024, 1024), (64, 3072, 4096, 4096), (300, 2048, 2048, 2048)])
def test_w4a8_rotated_linear(M, N, K, b):
    """fp16 activations through the GPU's 8-bit path and the host-quantized
    weight, against the oracle fed the GPU's codes; W4A8 must be closer to
    the float linear than W4A4 on the same inputs."""
    print(f"w4a8 rotated linear M={M} N={N} K={K} b={b}", flush=True)
    x16 = _x(9100 + M + N, M, K)
    w = G.gaussian(9100 + N, "w", (N, K), std=0.02)
    Wq, ws = oq.quantize_weights_host(w, b)
    X = torch.from_numpy(x16).to(DEV)
    Wd, wsd = torch.from_numpy(Wq).to(DEV), torch.from_numpy(ws).to(DEV)
    Xq8, xs = oq.rotate_quantize_act_i8(X, b)
    Y8 = oq.w4a8_linear(Xq8, xs, Wd, wsd)
    Xq4, xs4 = oq.rotate_quantize_act(X, b)
    Y4 = oq.w4a4_linear(Xq4, xs4, Wd, wsd)
    torch.cuda.synchronize()
    q = Xq8.cpu().numpy().astype(np.int64)
    ref = linear.dequant(linear.int_gemm(q, parity.unpack_int4(Wq)), xs.cpu().numpy(), ws, None)
    assert parity.rel_l2(Y8.float().cpu().numpy(), ref) <= parity.REL_L2_OUT
    exact = x16.astype(np.float64) @ w.T
    e8 = parity.rel_l2(Y8.float().cpu().numpy(), exact)
    e4 = parity.rel_l2(Y4.float().cpu().numpy(), exact)
    print(f"error vs float linear: W4A8 {e8:.4f}, W4A4 {e4:.4f}")
    assert e8 < e4
