"""Run-twice determinism and output guard bands, every kernel family at full
size (GPU).

Each call runs twice on the same inputs into fresh output buffers that carry
guard bands -- padding past the end of a dense output, or extra rows and
columns around a strided one -- filled with a different sentinel byte each
time.  The two results must agree bit for bit (int4 codes, integer
accumulators and floating-point outputs alike: the integer sums are exact and
every floating-point reduction has a fixed order, including the calibration's
histogram, whose counts are order-free integer sums), and no byte outside the
output may change.  The DiT step is run twice by the step-equivalence tests."""
import numpy as np
import pytest
import torch

import paper_2605_28803_amd as oq

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
PAD = 4096  # guard bytes past a dense output


def _dense(shape, dtype, fill):
    """A dense output view of `shape` inside a byte buffer that continues for
    PAD bytes of `fill` past its end.  Returns (buffer, view)."""
    n = int(np.prod(shape)) * torch.tensor([], dtype=dtype).element_size()
    buf = torch.full((n + PAD,), fill, dtype=torch.uint8, device=DEV)
    return buf, buf[:n].view(dtype).view(shape)


def _strided(M, N, dtype, fill, extra_rows=3, extra_cols=8):
    """An [M, N] output view with row stride N + extra_cols inside a
    (M + extra_rows) x (N + extra_cols) buffer filled with `fill` bytes."""
    es = torch.tensor([], dtype=dtype).element_size()
    buf = torch.full(((M + extra_rows) * (N + extra_cols) * es,), fill, dtype=torch.uint8, device=DEV)
    full = buf.view(dtype).view(M + extra_rows, N + extra_cols)
    return buf, full[:M, :N]


def _bits(t):
    return t.contiguous().view(torch.uint8).cpu().numpy()


def _guard_ok(buf, view, fill):
    """Every byte of buf outside the view still equals fill."""
    mask = torch.ones_like(buf, dtype=torch.bool)
    es = view.element_size()
    off = view.data_ptr() - buf.data_ptr()
    if view.is_contiguous():
        mask[off: off + view.numel() * es] = False
    else:  # a row-strided 2-D view
        M, N = view.shape
        rows = off + torch.arange(M, device=DEV)[:, None] * view.stride(0) * es
        mask[(rows + torch.arange(N * es, device=DEV)[None, :]).reshape(-1)] = False
    return bool(torch.all(buf[mask] == fill).item())


def _twice(run, outs):
    """run(views) fills the views; outs: list of (kind, shape, dtype) with kind
    'dense' or 'strided'.  Checks determinism and the guard bands."""
    results = []
    for fill in (0xA5, 0x5A):
        bufs = []
        for kind, shape, dtype in outs:
            bufs.append(_dense(shape, dtype, fill) if kind == "dense" else _strided(*shape, dtype, fill))
        run([v for _, v in bufs])
        torch.cuda.synchronize()
        for b, v in bufs:
            assert _guard_ok(b, v, fill), "a byte outside the output changed"
        results.append([_bits(v) for _, v in bufs])
    for a, b in zip(*results):
        assert np.array_equal(a, b), "two runs differ"


def _x(M, K, seed, outlier_frac=0.01):
    g = torch.Generator(device=DEV).manual_seed(seed)
    X = torch.randn((M, K), generator=g, device=DEV)
    X[:, torch.randperm(K, generator=g, device=DEV)[: max(1, int(outlier_frac * K))]] *= 50.0
    return X.half()


def _w(N, K, seed):
    g = torch.Generator(device=DEV).manual_seed(seed)
    return (torch.randn((N, K), generator=g, device=DEV) * 0.02).half()


@pytest.mark.parametrize("M,K", [(16384, 4096), (16384, 16384)])
def test_rotate_quantize(M, K):
    print(f"determinism rotate-quantize M={M} K={K}", flush=True)
    X = _x(M, K, 1)
    st = np.array([1.7], np.float32)
    _twice(lambda v: oq.rotate_quantize_act(X, K, s_table=st, t=0, Xq=v[0], x_scale=v[1]),
           [("dense", (M, K // 2), torch.uint8), ("dense", (M,), torch.float32)])


def test_rotate_quantize_static_and_calibration():
    M, K = 16384, 4096
    print("determinism calibration + static rotate-quantize", flush=True)
    X = _x(M, K, 2)
    Y = oq.rotate_act_f32(X, K)
    work = torch.empty((oq.calibrate_workspace_bytes(K),), dtype=torch.uint8, device=DEV)
    _twice(lambda v: oq.calibrate_step_scales(Y, 99.9, 7.0, delta=v[0], work=work),
           [("dense", (K,), torch.float32)])
    _twice(lambda v: oq.calibrate_step_scales_noalloc(Y, 99.9, 7.0, delta=v[0]), [("dense", (K,), torch.float32)])
    d = oq.calibrate_step_scales(Y, 99.9, 7.0)
    _twice(lambda v: oq.rotate_quantize_act_static(X, K, d, Xq=v[0], x_scale=v[1]),
           [("dense", (M, K // 2), torch.uint8), ("dense", (M,), torch.float32)])


@pytest.mark.parametrize("M,N,K", [(50, 8192, 1024), (50, 1024, 4096)])
def test_small_m_gemm(M, N, K):
    print(f"determinism small-M GEMM M={M} N={N} K={K}", flush=True)
    X, W = _x(M, K, 3), _w(N, K, 4)
    Wq, ws = oq.quantize_weights(W, K)
    Xt, xs = oq.rotate_quantize_act_tiled(X, K)
    Xq, xs2 = oq.rotate_quantize_act(X, K)
    _twice(lambda v: oq.w4a4_linear_tiled(Xt, xs, Wq, ws, Y=v[0]), [("strided", (M, N), torch.float16)])
    _twice(lambda v: oq.w4a4_linear(Xq, xs2, Wq, ws, out_dtype=oq.OUT_BF16, Y=v[0]),
           [("strided", (M, N), torch.bfloat16)])
    _twice(lambda v: oq.w4a4_gemm_i32(Xq, Wq, acc=v[0]), [("dense", (M, N), torch.int32)])


@pytest.mark.parametrize("M,N,K", [(4096, 4096, 4096), (1024, 1536, 6144), (256, 16384, 1536),
                                   (1024, 4608, 1536), (816, 2560, 2048)])
def test_large_gemm(M, N, K):
    """The 256 x 256, 128 x 128 and 64 x 64 tilings, with and without K groups."""
    print(f"determinism GEMM M={M} N={N} K={K}", flush=True)
    b = K & -K
    X, W = _x(M, K, 5), _w(N, K, 6)
    Wq, ws = oq.quantize_weights(W, b)
    Xq, xs = oq.rotate_quantize_act(X, b)
    _twice(lambda v: oq.w4a4_linear(Xq, xs, Wq, ws, Y=v[0]), [("strided", (M, N), torch.float16)])
    _twice(lambda v: oq.w4a4_gemm_i32(Xq, Wq, acc=v[0]), [("dense", (M, N), torch.int32)])


def test_w4a8():
    M, N, K = 4096, 4096, 4096
    print("determinism W4A8", flush=True)
    X, W = _x(M, K, 7), _w(N, K, 8)
    Wq, ws = oq.quantize_weights(W, K)
    X8, xs = oq.rotate_quantize_act_i8(X, K)
    _twice(lambda v: oq.rotate_quantize_act_i8(X, K, Xq8=v[0], x_scale=v[1]),
           [("dense", (M, K), torch.int8), ("dense", (M,), torch.float32)])
    _twice(lambda v: oq.w4a8_linear(X8, xs, Wq, ws, Y=v[0]), [("strided", (M, N), torch.float16)])


def test_composite_and_weight_preparation():
    """Column energies, zigzag, per-block eigen-decomposition (Jacobi) and the
    composite rotate-quantize with the online gather."""
    N, K, M = 3072, 4096, 16384
    print("determinism composite rotation and weight preparation", flush=True)
    W = _w(N, K, 9)
    X = _x(M, K, 10)
    _twice(lambda v: oq.channel_energy(W, energy=v[0]), [("dense", (K,), torch.float64)])
    e = oq.channel_energy(W)
    _twice(lambda v: oq.zigzag_permutation(e, 64, perm=v[0]), [("dense", (K,), torch.int32)])
    perm = oq.zigzag_permutation(e, 64)
    _twice(lambda v: oq.block_svd(W, perm, 64, U=v[0], sigma2=v[1]),
           [("dense", (K // 64, 64, 64), torch.float64), ("dense", (K // 64, 64), torch.float64)])
    U, _ = oq.block_svd(W, perm, 64)
    Rt = oq.block_rotations(U)
    _twice(lambda v: oq.rotate_quantize_act_composite(X, perm, Rt, Xq=v[0], x_scale=v[1]),
           [("dense", (M, K // 2), torch.uint8), ("dense", (M,), torch.float32)])


@pytest.mark.parametrize("K", [8192, 16384])
def test_composite_chunked(K):
    """The chunked composite kernel (row maxima exchanged between the chunks'
    workgroups), with the online permutation and with it folded."""
    M = 16384
    print(f"determinism composite chunked K={K}", flush=True)
    W = _w(1024, K, 11)
    X = _x(M, K, 12)
    e = oq.channel_energy(W)
    perm = oq.zigzag_permutation(e, 64)
    U, _ = oq.block_svd(W, perm, 64)
    Rt = oq.block_rotations(U)
    _twice(lambda v: oq.rotate_quantize_act_composite(X, perm, Rt, Xq=v[0], x_scale=v[1]),
           [("dense", (M, K // 2), torch.uint8), ("dense", (M,), torch.float32)])
    _twice(lambda v: oq.rotate_quantize_act_composite(X, None, Rt, Xq=v[0], x_scale=v[1]),
           [("dense", (M, K // 2), torch.uint8), ("dense", (M,), torch.float32)])
