"""Online full composite rotation (zigzag permutation, block 64 SVD factor
times Hadamard) + step scale + per-token int4 codes against the oracle (GPU),
with the permutation applied online and with it folded into the producer
(perm = NULL, the input already in the permuted order).

The oracle is fed the same fp16 activation and the same fp16 block matrices
(as float64).  The GPU forms the exact fp16 x fp16 products and sums each
64-term block product in fp32, so |y_gpu - y| <= gamma_64 S_j with S_j =
sum_r |(XP)_r R_b[r][j]|; with the derivation of the Hadamard kernel's bound
the pre-rounding ratio differs by at most tau_row = 14 gamma_64 max_j S_j /
max|y| + 21 * 2^-24.  Codes must match except inside that band (at most 1e-4
of the elements, each by one step); token scales to the same bound."""
import numpy as np
import pytest
import torch

import paper_2605_28803_amd as oq
from oracle import composite, linear, quant
from tests import parity
from workloads import generators as G

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
U32 = 2.0 ** -24


def _operands(seed, M, N, K, c=64, identity=False):
    x = G.gaussian(seed, "x", (M, K))
    x[:, G.outlier_channels(seed, "x", K, max(1, K // 100))] *= 50.0
    w = G.gaussian(seed, "w", (N, K), 0.02)
    w[:, G.outlier_channels(seed, "w", K, max(1, K // 128))] *= 20.0
    if identity:
        perm = np.arange(K)
        u = np.stack([np.eye(c)] * (K // c))
    else:
        perm = composite.zigzag_permutation(composite.channel_energy(w), K // c)
        u, _ = composite.block_svd_factors(w, perm, c)
    r16 = composite.block_rotations(u).astype(np.float16)
    return x.astype(np.float16), w, perm, r16


def _device(perm, r16):
    p = torch.from_numpy(perm.astype(np.int32)).to(DEV)
    rt = torch.from_numpy(np.ascontiguousarray(np.transpose(r16, (0, 2, 1))).view(np.int16)).to(DEV)
    return p, rt


def _tau(x16, perm, r16):
    xp = np.abs(x16.astype(np.float64)[:, perm])
    M, K = xp.shape
    nb, c, _ = r16.shape
    S = np.einsum("mbr,brj->mbj", xp.reshape(M, nb, c), np.abs(r16.astype(np.float64))).reshape(M, K)
    y = composite.rotate_composite(x16, perm, r16.astype(np.float64))
    amax = np.abs(y).max(axis=1)
    d = c
    gamma = d * U32 / (1 - d * U32)
    safe = np.where(amax > 0, amax, 1.0)
    return np.where(amax > 0, 14 * gamma * S.max(axis=1) / safe + 21 * U32, 0.0)


# Above K = 4096 (and at K = 4096 with P folded and M > 1024) the rows are
# split into chunks of channels whose workgroups exchange row maxima: 16-row
# tiles of up to 4096 channels with the online permutation, 32-row tiles of up
# to 1024 channels with it folded; several tiles, a partial last tile, and
# every chunk width.
CASES = [(50, 1024, 1.0), (64, 1024, 2.3), (33, 2048, 0.7), (17, 4096, 1.0), (9, 6144, 3.1), (5, 8192, 1.0),
         (3, 16384, 1.4), (1000, 1024, 1.0), (130, 1536, 0.9), (257, 4096, 1.0), (1, 64, 1.0),
         (100, 8192, 1.0), (257, 16384, 0.8), (33, 6144, 1.2), (40, 4608, 1.0), (17, 5120, 2.0),
         (1500, 4096, 1.0)]


@pytest.mark.parametrize("M,K,s", CASES)
def test_composite_codes(M, K, s):
    print(f"composite M={M} K={K} s={s}", flush=True)
    x16, _, perm, r16 = _operands(5000 + M + K, M, 96, K)
    p, rt = _device(perm, r16)
    X = torch.from_numpy(x16).to(DEV)
    Xq, xs = oq.rotate_quantize_act_composite(X, p, rt, s_table=np.array([s], np.float32), t=0)
    torch.cuda.synchronize()
    q_o, xs_o, r_o = composite.rotate_quantize_composite(x16, perm, r16.astype(np.float64), float(np.float32(s)))
    tau = _tau(x16, perm, r16)
    n_mis, _ = parity.check_codes(parity.unpack_int4(Xq.cpu().numpy()), q_o, r_o, tau)
    rel = np.abs(xs.cpu().numpy().astype(np.float64) - xs_o) / np.where(xs_o > 0, xs_o, 1.0)
    assert np.all(rel <= tau / 7 + 4 * U32)
    print(f"  boundary code differences {n_mis} of {M * K}")


@pytest.mark.parametrize("M,K,s", CASES)
def test_composite_prepermuted_codes(M, K, s):
    """perm = NULL: the activation arrives already in the permuted channel
    order (P folded into its producer); the codes of X P through R_hat equal
    the oracle's composite transform of X with P (same boundary rule)."""
    print(f"composite prepermuted M={M} K={K} s={s}", flush=True)
    x16, _, perm, r16 = _operands(5100 + M + K, M, 96, K)
    _, rt = _device(perm, r16)
    Xp = torch.from_numpy(np.ascontiguousarray(x16[:, perm])).to(DEV)
    Xq, xs = oq.rotate_quantize_act_composite(Xp, None, rt, s_table=np.array([s], np.float32), t=0)
    torch.cuda.synchronize()
    q_o, xs_o, r_o = composite.rotate_quantize_composite(x16, perm, r16.astype(np.float64), float(np.float32(s)))
    tau = _tau(x16, perm, r16)
    n_mis, _ = parity.check_codes(parity.unpack_int4(Xq.cpu().numpy()), q_o, r_o, tau)
    rel = np.abs(xs.cpu().numpy().astype(np.float64) - xs_o) / np.where(xs_o > 0, xs_o, 1.0)
    assert np.all(rel <= tau / 7 + 4 * U32)
    print(f"  boundary code differences {n_mis} of {M * K}")


@pytest.mark.parametrize("K", [2048, 8192])
def test_composite_prepermuted_strided_rows_and_zero_row(K):
    M = 40
    x16, _, perm, r16 = _operands(78 + K, M, 64, K)
    x16[7] = 0
    buf = torch.zeros((M, K + 64), dtype=torch.float16, device=DEV)
    buf[:, :K] = torch.from_numpy(np.ascontiguousarray(x16[:, perm])).to(DEV)
    _, rt = _device(perm, r16)
    Xq, xs = oq.rotate_quantize_act_composite(buf[:, :K], None, rt)
    torch.cuda.synchronize()
    q_o, xs_o, r_o = composite.rotate_quantize_composite(x16, perm, r16.astype(np.float64))
    parity.check_codes(parity.unpack_int4(Xq.cpu().numpy()), q_o, r_o, _tau(x16, perm, r16))
    assert xs.cpu().numpy()[7] == 0 and not Xq.cpu().numpy()[7].any()


@pytest.mark.parametrize("K", [2048, 8192])
def test_composite_strided_rows_and_zero_row(K):
    M = 40
    x16, _, perm, r16 = _operands(77 + K, M, 64, K)
    x16[7] = 0
    buf = torch.zeros((M, K + 64), dtype=torch.float16, device=DEV)
    buf[:, :K] = torch.from_numpy(x16).to(DEV)
    p, rt = _device(perm, r16)
    Xq, xs = oq.rotate_quantize_act_composite(buf[:, :K], p, rt)
    torch.cuda.synchronize()
    q_o, xs_o, r_o = composite.rotate_quantize_composite(x16, perm, r16.astype(np.float64))
    parity.check_codes(parity.unpack_int4(Xq.cpu().numpy()), q_o, r_o, _tau(x16, perm, r16))
    assert xs.cpu().numpy()[7] == 0 and not Xq.cpu().numpy()[7].any()


def test_identity_transform_is_the_hadamard_path():
    """perm = identity and U_b = I: the composite call computes the block-64
    Hadamard rotation of oq_rotate_quantize_act (both checked against the
    oracle's Hadamard path by the boundary rule)."""
    M, K = 64, 1024
    x16, _, perm, r16 = _operands(91, M, 64, K, identity=True)
    p, rt = _device(perm, r16)
    X = torch.from_numpy(x16).to(DEV)
    Xq, xs = oq.rotate_quantize_act_composite(X, p, rt)
    torch.cuda.synchronize()
    q_o, xs_o, r_o = quant.rotate_quantize_act(x16, 64)
    # H_64 / 8 has entries +-1/8, exact in fp16, so the oracle's Hadamard path
    # is the same map; the fp32 band is the composite one
    parity.check_codes(parity.unpack_int4(Xq.cpu().numpy()), q_o, r_o, _tau(x16, perm, r16))


def test_composite_linear_end_to_end():
    """Activation codes from the GPU call, weight folded with the same (perm,
    R) by the host preparation, product and epilogue on the GPU: within 2e-3
    of the oracle's product of the same codes; against the unquantized X W^T
    the W4A4 error is reported with and without the SVD factor."""
    M, N, K = 64, 1024, 1024
    x16, w, perm, r16 = _operands(123, M, N, K)
    p, rt = _device(perm, r16)
    Xq, xs = oq.rotate_quantize_act_composite(torch.from_numpy(x16).to(DEV), p, rt)
    rt_host = np.ascontiguousarray(np.transpose(r16, (0, 2, 1))).view(np.uint16)
    Wq, ws = oq.quantize_weights_composite_host(w, perm.astype(np.int32), rt_host)
    Y = oq.w4a4_linear(Xq, xs, torch.from_numpy(Wq).to(DEV), torch.from_numpy(ws).to(DEV))
    torch.cuda.synchronize()
    ref = linear.dequant(linear.int_gemm(parity.unpack_int4(Xq.cpu().numpy()), parity.unpack_int4(Wq)),
                         xs.cpu().numpy().astype(np.float64), ws.astype(np.float64))
    assert parity.rel_l2(Y.float().cpu().numpy(), ref) <= parity.REL_L2_OUT
    exact = x16.astype(np.float64) @ w.T
    err_c = parity.rel_l2(Y.float().cpu().numpy(), exact)
    # Hadamard-only path on the same data for comparison (information)
    Xh, xh = oq.rotate_quantize_act(torch.from_numpy(x16).to(DEV), 64)
    Wh, wh = oq.quantize_weights_host(w, 64)
    Yh = oq.w4a4_linear(Xh, xh, torch.from_numpy(Wh).to(DEV), torch.from_numpy(wh).to(DEV))
    torch.cuda.synchronize()
    err_h = parity.rel_l2(Yh.float().cpu().numpy(), exact)
    print(f"W4A4 rel. error vs X W^T: composite (zigzag + SVD + H64) {err_c:.4f}, Hadamard-64 only {err_h:.4f}")
    # quantization quality on synthetic data is information, not parity (the
    # paper's quality numbers need its weights and activations)
    assert np.isfinite(err_c) and np.isfinite(err_h) and err_c < 1.0 and err_h < 1.0


def test_chunked_calls_in_a_row():
    """Consecutive calls above K = 4096 with growing, shrinking and growing M:
    the exchange slots and the inverse permutation are re-initialised by every
    call (a stale slot would release a tile early, or a stale permutation
    would misplace channels)."""
    K = 8192
    x16, _, perm, r16 = _operands(4242, 3000, 64, K)
    p, rt = _device(perm, r16)
    X = torch.from_numpy(x16).to(DEV)
    q_o, xs_o, r_o = composite.rotate_quantize_composite(x16, perm, r16.astype(np.float64))
    tau = _tau(x16, perm, r16)
    for M in (1000, 40, 3000):
        print(f"composite chunked call M={M} K={K}", flush=True)
        Xq, xs = oq.rotate_quantize_act_composite(X[:M], p, rt)
        torch.cuda.synchronize()
        parity.check_codes(parity.unpack_int4(Xq.cpu().numpy()), q_o[:M], r_o[:M], tau[:M])
        rel = np.abs(xs.cpu().numpy().astype(np.float64) - xs_o[:M]) / np.where(xs_o[:M] > 0, xs_o[:M], 1.0)
        assert np.all(rel <= tau[:M] / 7 + 4 * U32)
