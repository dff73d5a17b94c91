"""Full-size launches of the composite rotation, the static steps, W4A8 and
the GPU weight preparation, in the configurations bench.py times, checked
on sampled outputs that the oracle computes one by one (GPU).

  * composite rotate-quantize at M = 16384, K = 1024, 4096, 8192 and 16384,
    with the online permutation and with it folded into the input: sampled
    rows' codes by the boundary rule against the oracle fed the same fp16 R_b;
  * static rotate-quantize at M = 16384, K = 4096: sampled rows by the
    static boundary rule;
  * W4A8 at M = K = N = 16384 (the 128 x 128 tiling with 8-bit token codes)
    and a ragged shape on the same tiling: sampled int32 accumulators
    bit-exact;
  * weight preparation at the Gemma-2B-shaped gate|up (32768 x 2048): the
    permutation exact, sampled blocks' squared singular values within the
    fp64 bound, sampled weight rows' codes in the boundary band of the fold.
"""
import numpy as np
import pytest
import torch

import paper_2605_28803_amd as oq
from oracle import composite, hadamard, linear, quant
from tests import parity
from tests.test_gpu_composite import _tau
from workloads import generators as G

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _rows(M, n, seed):
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([rng.choice(M, n, replace=False), [0, M - 1]]))


@pytest.mark.parametrize("K,folded", [(1024, False), (4096, False), (8192, False), (16384, False), (1024, True),
                                      (4096, True), (8192, True), (16384, True)])
def test_composite_full_size_sampled(K, folded):
    """folded: perm = None on the input already in the permuted order (the
    GPU is handed X P, the oracle X and P)."""
    M = 16384
    print(f"composite full size M={M} K={K} folded={folded}", flush=True)
    energy = G.gaussian(11, f"composite/energy{K}", (K,)) ** 2
    perm = composite.zigzag_permutation(energy, K // 64)
    u = np.stack([G.random_orthogonal(11, f"composite/u{K}/{b}", 64) for b in range(K // 64)])
    r16 = composite.block_rotations(u).astype(np.float16)
    g = torch.Generator(device=DEV).manual_seed(13)
    X = torch.randn((M, K), generator=g, device=DEV).half()
    p = torch.from_numpy(perm.astype(np.int32)).to(DEV)
    rt = torch.from_numpy(np.ascontiguousarray(np.transpose(r16, (0, 2, 1))).view(np.int16)).to(DEV)
    if folded:
        Xq, xs = oq.rotate_quantize_act_composite(X[:, p.long()].contiguous(), None, rt)
    else:
        Xq, xs = oq.rotate_quantize_act_composite(X, p, rt)
    torch.cuda.synchronize()
    rows = _rows(M, 48, K)
    ri = torch.from_numpy(rows).to(DEV)
    x16 = X[ri].cpu().numpy()
    q_g = parity.unpack_int4(Xq[ri].cpu().numpy())
    q_o, xs_o, r_o = composite.rotate_quantize_composite(x16, perm, r16.astype(np.float64))
    tau = _tau(x16, perm, r16)
    parity.check_codes(q_g, q_o, r_o, tau)
    rel = np.abs(xs[ri].cpu().numpy().astype(np.float64) - xs_o) / np.where(xs_o > 0, xs_o, 1.0)
    assert np.all(rel <= tau / 7 + 4 * parity.U32)


def test_static_full_size_sampled():
    M, K = 16384, 4096
    g = torch.Generator(device=DEV).manual_seed(17)
    X = torch.randn((M, K), generator=g, device=DEV).half()
    Yc = oq.rotate_act_f32(torch.randn((16384, K), generator=g, device=DEV).half(), K)
    delta = oq.calibrate_step_scales(Yc, 99.9, 7.0)
    Xq, xs = oq.rotate_quantize_act_static(X, K, delta)
    torch.cuda.synchronize()
    rows = _rows(M, 48, 5)
    ri = torch.from_numpy(rows).to(DEV)
    x16 = X[ri].cpu().numpy()
    d = delta.cpu().numpy().astype(np.float64)
    q_o, _, r_o = quant.rotate_quantize_static(x16.astype(np.float64), K, d)
    parity.check_codes(parity.unpack_int4(Xq[ri].cpu().numpy()), q_o, r_o, parity.tau_static(x16, K, d, r_o))
    assert torch.all(xs == 1.0)


def _packed_int4(R, K, gen):
    u = torch.randint(0, 15, (R, K), generator=gen, device=DEV, dtype=torch.int16) - 7
    n = (u & 0xF).to(torch.uint8)
    return (n[:, 0::2] | (n[:, 1::2] << 4)).contiguous()


@pytest.mark.parametrize("M,N,K", [(16384, 16384, 16384), (2100, 4160, 192)])
def test_w4a8_large_tiles_sampled(M, N, K):
    print(f"w4a8 large M={M} N={N} K={K}", flush=True)
    gen = torch.Generator(device=DEV).manual_seed(M + N + K)
    X8 = (torch.randint(0, 255, (M, K), generator=gen, device=DEV, dtype=torch.int16) - 127).to(torch.int8)
    Wq = _packed_int4(N, K, gen)
    acc = oq.w4a8_gemm_i32(X8, Wq)
    torch.cuda.synchronize()
    rows = _rows(M, 24, K)
    cols = _rows(N, 256, N)
    q = X8[torch.from_numpy(rows).to(DEV)].cpu().numpy().astype(np.int64)
    qw = parity.unpack_int4(Wq[torch.from_numpy(cols).to(DEV)].cpu().numpy())
    a = acc[torch.from_numpy(rows).to(DEV)][:, torch.from_numpy(cols).to(DEV)].cpu().numpy().astype(np.int64)
    assert np.array_equal(a, linear.int_gemm(q, qw))


def test_prepare_full_size_sampled():
    N, K = 32768, 2048
    g = torch.Generator(device=DEV).manual_seed(23)
    W = (torch.randn((N, K), generator=g, device=DEV) * 0.02).half()
    perm, Rt, Wq, ws = oq.prepare_weights_composite(W)
    e = oq.channel_energy(W)
    U, lam = oq.block_svd(W, perm)
    torch.cuda.synchronize()
    w16 = W.cpu().numpy()
    w64 = w16.astype(np.float64)
    perm_o = composite.zigzag_permutation(composite.channel_energy(w64), K // 64)
    assert np.array_equal(perm.cpu().numpy(), perm_o)
    lam = lam.cpu().numpy()
    for b in (0, 13, K // 64 - 1):
        wb = w64[:, perm_o[b * 64:(b + 1) * 64]].T
        ev = np.sort(np.linalg.eigvalsh(wb @ wb.T))[::-1]
        assert np.all(np.abs(lam[b] - ev) <= 64 * N * 2.0 ** -52 * ev.max()), b
    rows = _rows(N, 64, 3)
    r16 = np.transpose(Rt.cpu().numpy().view(np.float16), (0, 2, 1))
    q_o, ws_o, ratio = composite.fold_weights_composite(w64[rows], perm_o, r16.astype(np.float64))
    parity.check_codes(parity.unpack_int4(Wq.cpu().numpy()[rows]), q_o, ratio, _tau(w16[rows], perm_o, r16))
    assert np.allclose(ws.cpu().numpy()[rows], ws_o, rtol=1e-5)
