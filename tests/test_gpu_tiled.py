"""Token codes in the 16-row tiled layout (GPU).

The layout is restated here from its definition in include/oq.h (independent
of the library's code): re-layout must be bit-exact, the tiled rotate-quantize
must write exactly the codes and scales of the row-layout call (which the
oracle pins), and the tiled product must give bit-exact int32 accumulators
against the oracle's integer product and the dequantized outputs within the
2e-3 relative L2 bound."""
import numpy as np
import pytest
import torch

import paper_2605_28803_amd as oq
from oracle import linear, quant
from tests import parity
from workloads import generators as G

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def tile_np(Q: np.ndarray, K: int) -> np.ndarray:
    """Packed codes [R][K/2] -> tiled bytes: byte p of row r at
    ((r // 16) * (K // 128) + p // 64) * 1024 + ((p // 16) % 4) * 256 + (r % 16) * 16 + p % 16."""
    R = Q.shape[0]
    R16 = (R + 15) // 16 * 16
    out = np.zeros(R16 * K // 2, dtype=np.uint8)
    r = np.arange(R)[:, None]
    p = np.arange(K // 2)[None, :]
    off = ((r // 16) * (K // 128) + p // 64) * 1024 + ((p // 16) % 4) * 256 + (r % 16) * 16 + p % 16
    out[off.reshape(-1)] = Q.reshape(-1)
    return out


def untile_np(T: np.ndarray, R: int, K: int) -> np.ndarray:
    r = np.arange(R)[:, None]
    p = np.arange(K // 2)[None, :]
    off = ((r // 16) * (K // 128) + p // 64) * 1024 + ((p // 16) % 4) * 256 + (r % 16) * 16 + p % 16
    return T[off]


@pytest.mark.parametrize("R,K", [(1, 128), (15, 256), (16, 1024), (17, 1536), (50, 1024), (64, 4096),
                                 (100, 2048), (33, 16384)])
def test_codes_to_tiled_bit_exact(R, K):
    print(f"codes_to_tiled R={R} K={K}", flush=True)
    rng = np.random.default_rng(R * 7 + K)
    Q = rng.integers(0, 256, size=(R, K // 2), dtype=np.uint8)
    T = oq.codes_to_tiled(torch.from_numpy(Q).to(DEV), K)
    torch.cuda.synchronize()
    assert np.array_equal(T.cpu().numpy(), tile_np(Q, K))


ROTATE_CASES = [
    # (M, K, b, s): matrix-core rows (b >= 32, K in the compiled set), VALU rows
    # (b < 32 or other K), several tiled row blocks with a ragged last block
    (50, 1024, 1024, 2.7), (50, 4096, 4096, 0.6), (7, 1536, 512, 0.8), (64, 2048, 2048, 1.0),
    (33, 16384, 16384, 1.3), (20, 8192, 4096, 1.0), (5, 128, 64, 1.0), (50, 1024, 8, 1.0),
    (17, 6144, 2048, 3.9), (130, 1024, 1024, 1.0), (3, 384, 128, 1.0),
]


@pytest.mark.parametrize("M,K,b,s", ROTATE_CASES)
def test_rotate_quantize_tiled_matches_row_layout(M, K, b, s):
    print(f"rotate_quantize_tiled M={M} K={K} b={b} s={s}", flush=True)
    seed = 7000 + M + K
    x = G.gaussian(seed, "x", (M, K))
    x[:, G.outlier_channels(seed, "x", K, max(1, int(round(0.01 * K))))] *= 50.0
    x16 = x.astype(np.float16)
    X = torch.from_numpy(x16).to(DEV)
    st = np.array([s], dtype=np.float32)
    Xq, xs = oq.rotate_quantize_act(X, b, s_table=st, t=0)
    Xt, xst = oq.rotate_quantize_act_tiled(X, b, s_table=st, t=0)
    torch.cuda.synchronize()
    Xq, xs, Xt, xst = Xq.cpu().numpy(), xs.cpu().numpy(), Xt.cpu().numpy(), xst.cpu().numpy()
    assert np.array_equal(untile_np(Xt, M, K), Xq)
    assert np.array_equal(xs, xst)
    # and against the oracle (boundary rule)
    q_o, _, r_o = quant.rotate_quantize_act(x16.astype(np.float64), b, float(np.float32(s)))
    parity.check_codes(parity.unpack_int4(untile_np(Xt, M, K)), q_o, r_o, parity.tau_rows(x16, b))


GEMM_CASES = [
    # (M, N, K): the DiT Pi-0.5 linears, decode-sized rows, ragged row blocks,
    # M > 64 (row groups along grid.y), narrow and deep K
    (50, 3072, 1024), (50, 1024, 1024), (50, 8192, 1024), (50, 1024, 4096),
    (1, 2560, 2048), (16, 2048, 16384), (17, 200, 2048), (64, 4096, 128), (65, 320, 1536),
    (130, 1000, 1024), (33, 48, 6144), (8, 32768, 2048),
    # M > 64 in 64-row blocks (wide or deep enough that 16-row blocks would
    # exceed 4096 waves), ragged last block
    (200, 8192, 1024), (100, 2048, 4096),
]


def _tiled_operands(q, K):
    return torch.from_numpy(tile_np(parity.pack_int4(q), K)).to(DEV)


@pytest.mark.parametrize("M,N,K", GEMM_CASES)
def test_gemm_i32_tiled_bit_exact(M, N, K):
    print(f"gemm i32 tiled M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M * 31 + N * 7 + K)
    q, qw = rng.integers(-7, 8, size=(M, K)), rng.integers(-7, 8, size=(N, K))
    acc = oq.w4a4_gemm_i32_tiled(_tiled_operands(q, K), M, torch.from_numpy(parity.pack_int4(qw)).to(DEV))
    torch.cuda.synchronize()
    assert np.array_equal(acc.cpu().numpy().astype(np.int64), linear.int_gemm(q, qw))


def test_gemm_i32_tiled_extreme_magnitudes():
    """Every code +-7 at K = 16384 through the tiled operand: |acc| = 49 K."""
    K = 16384
    q = np.full((3, K), 7)
    q[1] = -7
    q[2, ::2] = -7
    qw = np.full((4, K), 7)
    qw[1] = -7
    qw[2, 1::2] = -7
    acc = oq.w4a4_gemm_i32_tiled(_tiled_operands(q, K), 3, torch.from_numpy(parity.pack_int4(qw)).to(DEV))
    acc = acc.cpu().numpy()
    assert np.array_equal(acc.astype(np.int64), linear.int_gemm(q, qw))
    assert acc[0, 0] == 49 * K and acc[1, 0] == -49 * K


@pytest.mark.parametrize("out_dtype", [oq.OUT_F16, oq.OUT_BF16])
@pytest.mark.parametrize("M,N,K", [(50, 1024, 1024), (50, 8192, 1024), (9, 1000, 4096), (70, 256, 2048)])
def test_linear_tiled_epilogue(M, N, K, out_dtype):
    print(f"linear tiled M={M} N={N} K={K} out={out_dtype}", flush=True)
    rng = np.random.default_rng(M * N + K + out_dtype)
    q, qw = rng.integers(-7, 8, size=(M, K)), rng.integers(-7, 8, size=(N, K))
    xs = rng.uniform(0.01, 2.0, M).astype(np.float32)
    ws = rng.uniform(1e-4, 1e-2, N).astype(np.float32)
    bias = (rng.standard_normal(N) * 0.1).astype(np.float16)
    Y = oq.w4a4_linear_tiled(_tiled_operands(q, K), torch.from_numpy(xs).to(DEV),
                             torch.from_numpy(parity.pack_int4(qw)).to(DEV), torch.from_numpy(ws).to(DEV),
                             bias=torch.from_numpy(bias).to(DEV), out_dtype=out_dtype)
    ref = linear.dequant(linear.int_gemm(q, qw), xs, ws, bias.astype(np.float64))
    err = parity.rel_l2(Y.float().cpu().numpy(), ref)
    print(f"tiled dequant rel_l2={err:.3e}")
    assert err <= parity.REL_L2_OUT


def test_tiled_and_row_layout_linears_agree_bitwise():
    """The same codes through both operand layouts give identical fp16 outputs."""
    M, N, K = 50, 3072, 1024
    rng = np.random.default_rng(5)
    q, qw = rng.integers(-7, 8, size=(M, K)), rng.integers(-7, 8, size=(N, K))
    xs = torch.from_numpy(rng.uniform(0.01, 2.0, M).astype(np.float32)).to(DEV)
    ws = torch.from_numpy(rng.uniform(1e-4, 1e-2, N).astype(np.float32)).to(DEV)
    Wq = torch.from_numpy(parity.pack_int4(qw)).to(DEV)
    Xq = torch.from_numpy(parity.pack_int4(q)).to(DEV)
    Y0 = oq.w4a4_linear(Xq, xs, Wq, ws)
    Y1 = oq.w4a4_linear_tiled(oq.codes_to_tiled(Xq), xs, Wq, ws)
    torch.cuda.synchronize()
    assert torch.equal(Y0, Y1)
