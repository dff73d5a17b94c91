"""Offline preparation of the composite-rotation weight on the GPU against
the oracle (Section 4.1).

  * channel energies: fp64 sums in another order, within N * 2^-52 relative;
  * zigzag permutation from the same energies: bit-exact (ties included);
  * block SVD factor: squared singular values within the fp64 rounding of the
    Gram matrix; each singular vector (both sides with the canonical sign)
    within the eigenvector perturbation bound 10 N eps lambda_max / gap
    wherever its singular value is separated; every U_b orthogonal;
  * R_b in fp16 from the oracle's own U_b: bit-exact (both round once, half
    to even);
  * the whole preparation: the permutation equal to the oracle's, R_b equal
    up to a few one-ulp differences at fp16 rounding boundaries, and the
    folded weight codes within the composite kernel's boundary band against
    the oracle's fold with the GPU's R_b.
"""
import numpy as np
import pytest
import torch

import paper_2605_28803_amd as oq
from oracle import composite
from tests import parity
from tests.test_gpu_composite import _tau
from workloads import generators as G

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
EPS = 2.0 ** -52


def _weight(seed, N, K):
    w = G.gaussian(seed, "w", (N, K), 0.02)
    w[:, G.outlier_channels(seed, "w", K, max(1, K // 128))] *= 20.0
    return w.astype(np.float16)


@pytest.mark.parametrize("N,K", [(96, 64), (1024, 1024), (40, 256), (3000, 4096), (17, 16384)])
def test_channel_energy(N, K):
    w16 = _weight(6000 + N + K, N, K)
    e = oq.channel_energy(torch.from_numpy(w16).to(DEV))
    torch.cuda.synchronize()
    ref = composite.channel_energy(w16.astype(np.float64))
    assert np.all(np.abs(e.cpu().numpy() - ref) <= 2 * N * EPS * ref)


@pytest.mark.parametrize("K,block", [(8, 2), (64, 64), (1024, 64), (4096, 64), (16384, 64), (96, 32)])
def test_zigzag_device(K, block):
    rng = np.random.default_rng(K + block)
    e = rng.exponential(size=K)
    e[rng.choice(K, min(K, 9), replace=False)] = e[1]  # ties
    e[rng.choice(K, min(K, 3), replace=False)] = 0.0
    perm = oq.zigzag_permutation(torch.from_numpy(e).to(DEV), block)
    torch.cuda.synchronize()
    assert np.array_equal(perm.cpu().numpy(), composite.zigzag_permutation(e, K // block))


def test_zigzag_device_golden():
    from tests.oracle_pins import load_golden_rows
    g = load_golden_rows("zigzag_example.txt")
    perm = oq.zigzag_permutation(torch.from_numpy(g["energy"]).to(DEV), 4)
    torch.cuda.synchronize()
    assert np.array_equal(perm.cpu().numpy(), g["perm"].astype(np.int32))


def _svd_ref(w16, perm):
    u, s = composite.block_svd_factors(w16.astype(np.float64), perm, 64)
    lam = np.stack([np.concatenate([si ** 2, np.zeros(64 - si.shape[0])]) for si in s])
    return composite.canonical_signs(u), lam


@pytest.mark.parametrize("N,K", [(1024, 1024), (4096, 256), (64, 128), (40, 128), (3000, 4096), (100, 64)])
def test_block_svd(N, K):
    print(f"block_svd N={N} K={K}", flush=True)
    w16 = _weight(6100 + N + K, N, K)
    perm = composite.zigzag_permutation(composite.channel_energy(w16.astype(np.float64)), K // 64)
    U, lam = oq.block_svd(torch.from_numpy(w16).to(DEV), torch.from_numpy(perm.astype(np.int32)).to(DEV))
    torch.cuda.synchronize()
    U, lam = U.cpu().numpy(), lam.cpu().numpy()
    u_o, lam_o = _svd_ref(w16, perm)
    worst = 0.0
    for b in range(K // 64):
        lmax = lam_o[b].max()
        assert np.all(np.abs(lam[b] - lam_o[b]) <= 64 * N * EPS * lmax), "squared singular values"
        assert np.allclose(U[b].T @ U[b], np.eye(64), atol=1e-12), "not orthogonal"
        assert np.all(np.diff(lam[b]) <= 64 * N * EPS * lmax), "not descending"
        # separated, non-null singular values: the vectors are unique up to sign
        for i in range(64):
            if lam_o[b, i] <= 1e-9 * lmax:
                continue
            others = np.delete(lam_o[b], i)
            gap = np.min(np.abs(others - lam_o[b, i]))
            if gap <= 1e-6 * lmax:
                continue
            tol = 10 * N * EPS * lmax / gap
            err = np.max(np.abs(U[b][:, i] - u_o[b][:, i]))
            worst = max(worst, err / tol)
            assert err <= tol, (b, i, err, tol)
        # signs: the largest-magnitude entry of every column is positive
        idx = np.argmax(np.abs(U[b]), axis=0)
        assert np.all(U[b][idx, np.arange(64)] > 0)
    print(f"  worst vector error / bound = {worst:.3g}")


@pytest.mark.parametrize("K", [64, 1024, 4096])
def test_block_rotations_device(K):
    rng = np.random.default_rng(K)
    u = np.stack([np.linalg.qr(rng.standard_normal((64, 64)))[0] for _ in range(K // 64)])
    Rt = oq.block_rotations(torch.from_numpy(u).to(DEV))
    torch.cuda.synchronize()
    ref = composite.block_rotations(u).astype(np.float16)  # numpy rounds fp64 -> fp16 once, half to even
    got = np.transpose(Rt.cpu().numpy().view(np.float16), (0, 2, 1))
    assert np.array_equal(got.view(np.uint16), ref.view(np.uint16))


@pytest.mark.parametrize("N,K", [(96, 1024), (1024, 4096), (300, 2048), (64, 64)])
def test_prepare_weights_composite(N, K):
    print(f"prepare N={N} K={K}", flush=True)
    w16 = _weight(6200 + N + K, N, K)
    perm, Rt, Wq, ws = oq.prepare_weights_composite(torch.from_numpy(w16).to(DEV))
    torch.cuda.synchronize()
    perm, Rt, Wq, ws = perm.cpu().numpy(), Rt.cpu().numpy(), Wq.cpu().numpy(), ws.cpu().numpy()
    w64 = w16.astype(np.float64)
    perm_o = composite.zigzag_permutation(composite.channel_energy(w64), K // 64)
    assert np.array_equal(perm, perm_o)
    u_o, _ = _svd_ref(w16, perm_o)
    r_o = composite.block_rotations(u_o).astype(np.float16)
    got = np.transpose(Rt.view(np.float16), (0, 2, 1))
    d = np.abs(got.view(np.uint16).astype(np.int64) - r_o.view(np.uint16).astype(np.int64))
    # the two U_b agree to ~1e-12, so fp16 entries differ (by one ulp) only
    # next to a rounding boundary
    assert d.max() <= 1 and np.count_nonzero(d) <= max(4, d.size // 10000), np.count_nonzero(d)
    # the fold with the GPU's own R_b: per-output-channel codes in the band
    r16 = got.astype(np.float16)
    q_o, ws_o, ratio = composite.fold_weights_composite(w64, perm, r16.astype(np.float64))
    parity.check_codes(parity.unpack_int4(Wq), q_o, ratio, _tau(w16, perm, r16))
    assert np.allclose(ws, ws_o, rtol=1e-5)
