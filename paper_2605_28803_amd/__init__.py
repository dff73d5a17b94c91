"""MI355X (gfx950) W4A4 rotated linear: Python binding of liboq.so.

Thin marshalling layer over the C ABI in include/oq.h: every computation runs
in the library's HIP kernels; torch only provides device memory and the
stream.  Functions have the names of the C entry points without the ``oq_``
prefix.  Raises OQError on a non-zero status.
"""
from __future__ import annotations

import ctypes as C

import numpy as np
import torch

from . import _lib

OUT_F16, OUT_BF16 = 0, 1


class OQError(RuntimeError):
    def __init__(self, status: int, where: str):
        lib = _lib.load()
        super().__init__(f"{where}: {lib.oq_status_string(status).decode()} ({status})")
        self.status = status


def lib():
    return _lib.load()


def _check(status: int, where: str):
    if status != 0:
        raise OQError(status, where)


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return C.c_void_p(s.cuda_stream)


def _ld(t):
    """Leading dimension (elements from one row to the next) of a 2-D tensor.
    The stride of a single row is unconstrained (numpy and torch may give it
    any value), and only row 0 is read, so its leading dimension is the row
    length."""
    return t.stride(0) if t.shape[0] > 1 else t.shape[1]


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _s_table(s_table):
    if s_table is None:
        return None, None
    arr = np.ascontiguousarray(np.asarray(s_table, dtype=np.float32).reshape(-1))
    return arr, arr.ctypes.data_as(C.POINTER(C.c_float))


def version() -> str:
    return lib().oq_version().decode()


def check_device() -> int:
    return lib().oq_check_device()


def status_string(code: int) -> str:
    return lib().oq_status_string(code).decode()


def rotate_quantize_act(X, had_block, s_table=None, t=0, Xq=None, x_scale=None, stream=None):
    """X: fp16 [M, K] (row stride X.stride(0); any stride for a single row).  Returns (Xq uint8 [M, K/2], x_scale f32 [M])."""
    M, K = X.shape
    if Xq is None:
        Xq = torch.empty((M, K // 2), dtype=torch.uint8, device=X.device)
    if x_scale is None:
        x_scale = torch.empty((M,), dtype=torch.float32, device=X.device)
    keep, sp = _s_table(s_table)
    _check(lib().oq_rotate_quantize_act(_ptr(X), M, K, _ld(X), had_block, sp, t, _ptr(Xq),
                                        _ptr(x_scale), _stream(stream)), "oq_rotate_quantize_act")
    del keep
    return Xq, x_scale


def tiled_bytes(rows: int, K: int) -> int:
    """Size of the 16-row tiled code layout of a rows x K code matrix."""
    return (rows + 15) // 16 * 16 * (K // 2)


def rotate_quantize_act_tiled(X, had_block, s_table=None, t=0, Xt=None, x_scale=None, stream=None):
    """As rotate_quantize_act, codes in the 16-row tiled layout (uint8 [tiled_bytes(M, K)])."""
    M, K = X.shape
    if Xt is None:
        Xt = torch.empty((tiled_bytes(M, K),), dtype=torch.uint8, device=X.device)
    if x_scale is None:
        x_scale = torch.empty((M,), dtype=torch.float32, device=X.device)
    keep, sp = _s_table(s_table)
    _check(lib().oq_rotate_quantize_act_tiled(_ptr(X), M, K, _ld(X), had_block, sp, t, _ptr(Xt),
                                              _ptr(x_scale), _stream(stream)), "oq_rotate_quantize_act_tiled")
    del keep
    return Xt, x_scale


def codes_to_tiled(Q, K=None, T=None, stream=None):
    """Packed codes uint8 [R, K/2] -> the 16-row tiled layout (uint8 [tiled_bytes(R, K)])."""
    R, Kh = Q.shape
    K = 2 * Kh if K is None else K
    if T is None:
        T = torch.empty((tiled_bytes(R, K),), dtype=torch.uint8, device=Q.device)
    _check(lib().oq_codes_to_tiled(_ptr(Q), R, K, _ptr(T), _stream(stream)), "oq_codes_to_tiled")
    return T


def rotate_quantize_act_composite(X, perm, Rt, s_table=None, t=0, Xq=None, x_scale=None, stream=None):
    """Full composite rotation (block 64) + step scale + per-token int4 codes.
    X fp16 [M, K]; perm int32 [K] (None: X is already in the permuted channel
    order) and Rt fp16 [K/64, 64, 64] (column-major blocks) on the device.
    Returns (Xq uint8 [M, K/2], x_scale f32 [M])."""
    M, K = X.shape
    if Xq is None:
        Xq = torch.empty((M, K // 2), dtype=torch.uint8, device=X.device)
    if x_scale is None:
        x_scale = torch.empty((M,), dtype=torch.float32, device=X.device)
    keep, sp = _s_table(s_table)
    _check(lib().oq_rotate_quantize_act_composite(_ptr(X), M, K, _ld(X), _ptr(perm), _ptr(Rt), sp, t,
                                                  _ptr(Xq), _ptr(x_scale), _stream(stream)),
           "oq_rotate_quantize_act_composite")
    del keep
    return Xq, x_scale


def zigzag_permutation_host(energy: np.ndarray, block: int) -> np.ndarray:
    """Zigzag channel permutation (int32 [K]) from per-channel weight energies."""
    e = np.ascontiguousarray(energy, dtype=np.float64)
    perm = np.empty(e.shape[0], dtype=np.int32)
    _check(lib().oq_zigzag_permutation_host(e.ctypes.data, e.shape[0], block, perm.ctypes.data),
           "oq_zigzag_permutation_host")
    return perm


def block_rotations_host(U: np.ndarray) -> np.ndarray:
    """fp16 column-major blocks Rt [nb, c, c] (as uint16) of U_b H_c / sqrt(c)."""
    u = np.ascontiguousarray(U, dtype=np.float64)
    nb, c, _ = u.shape
    Rt = np.empty((nb, c, c), dtype=np.uint16)
    _check(lib().oq_block_rotations_host(u.ctypes.data, nb * c, c, Rt.ctypes.data), "oq_block_rotations_host")
    return Rt


def quantize_weights_composite_host(W_u: np.ndarray, perm: np.ndarray, Rt: np.ndarray):
    """float64 host weight [N, K] folded with (perm, Rt) and RTN-quantized:
    (Wq uint8 [N, K/2], w_scale f32 [N])."""
    W = np.ascontiguousarray(W_u, dtype=np.float64)
    N, K = W.shape
    p = np.ascontiguousarray(perm, dtype=np.int32)
    r = np.ascontiguousarray(Rt, dtype=np.uint16)
    Wq = np.empty((N, K // 2), dtype=np.uint8)
    ws = np.empty((N,), dtype=np.float32)
    _check(lib().oq_quantize_weights_composite_host(W.ctypes.data, N, K, r.shape[-1], p.ctypes.data,
                                                    r.ctypes.data, Wq.ctypes.data, ws.ctypes.data),
           "oq_quantize_weights_composite_host")
    return Wq, ws


def rotate_debug_f32(X, had_block, s_table=None, t=0, stream=None):
    """Pre-rounding ratios z/Delta (f32 [M, K]) and x_scale."""
    M, K = X.shape
    ratio = torch.empty((M, K), dtype=torch.float32, device=X.device)
    x_scale = torch.empty((M,), dtype=torch.float32, device=X.device)
    keep, sp = _s_table(s_table)
    _check(lib().oq_rotate_debug_f32(_ptr(X), M, K, _ld(X), had_block, sp, t, _ptr(ratio),
                                     _ptr(x_scale), _stream(stream)), "oq_rotate_debug_f32")
    del keep
    return ratio, x_scale


def w4a4_linear(Xq, x_scale, Wq, w_scale, bias=None, out_dtype=OUT_F16, Y=None, stream=None):
    """Y [M, N] (fp16 or bf16) = dequant(Xq . Wq^T)."""
    M = Xq.shape[0]
    N, Kh = Wq.shape
    K = 2 * Kh
    if Y is None:
        dt = torch.float16 if out_dtype == OUT_F16 else torch.bfloat16
        Y = torch.empty((M, N), dtype=dt, device=Xq.device)
    _check(lib().oq_w4a4_linear(_ptr(Xq), _ptr(x_scale), M, _ptr(Wq), _ptr(w_scale), _ptr(bias), N, K,
                                _ptr(Y), _ld(Y), out_dtype, _stream(stream)), "oq_w4a4_linear")
    return Y


def w4a4_gemm_i32(Xq, Wq, acc=None, stream=None):
    M = Xq.shape[0]
    N, Kh = Wq.shape
    if acc is None:
        acc = torch.empty((M, N), dtype=torch.int32, device=Xq.device)
    _check(lib().oq_w4a4_gemm_i32(_ptr(Xq), M, _ptr(Wq), N, 2 * Kh, _ptr(acc), _ld(acc),
                                  _stream(stream)), "oq_w4a4_gemm_i32")
    return acc


def w4a4_linear_tiled(Xt, x_scale, Wq, w_scale, bias=None, out_dtype=OUT_F16, Y=None, stream=None):
    """As w4a4_linear with the token codes in the 16-row tiled layout (M = len(x_scale))."""
    M = x_scale.shape[0]
    N, Kh = Wq.shape
    K = 2 * Kh
    if Y is None:
        dt = torch.float16 if out_dtype == OUT_F16 else torch.bfloat16
        Y = torch.empty((M, N), dtype=dt, device=Wq.device)
    _check(lib().oq_w4a4_linear_tiled(_ptr(Xt), _ptr(x_scale), M, _ptr(Wq), _ptr(w_scale), _ptr(bias), N, K,
                                      _ptr(Y), _ld(Y), out_dtype, _stream(stream)), "oq_w4a4_linear_tiled")
    return Y


def w4a4_gemm_i32_tiled(Xt, M, Wq, acc=None, stream=None):
    N, Kh = Wq.shape
    if acc is None:
        acc = torch.empty((M, N), dtype=torch.int32, device=Wq.device)
    _check(lib().oq_w4a4_gemm_i32_tiled(_ptr(Xt), M, _ptr(Wq), N, 2 * Kh, _ptr(acc), _ld(acc),
                                        _stream(stream)), "oq_w4a4_gemm_i32_tiled")
    return acc


def quantize_weights(W_u, had_block, Wq=None, w_scale=None, stream=None):
    """W_u fp16 [N, K] on the device -> (Wq uint8 [N, K/2], w_scale f32 [N])."""
    N, K = W_u.shape
    if Wq is None:
        Wq = torch.empty((N, K // 2), dtype=torch.uint8, device=W_u.device)
    if w_scale is None:
        w_scale = torch.empty((N,), dtype=torch.float32, device=W_u.device)
    _check(lib().oq_quantize_weights(_ptr(W_u), N, K, _ld(W_u), had_block, _ptr(Wq), _ptr(w_scale),
                                     _stream(stream)), "oq_quantize_weights")
    return Wq, w_scale


def quantize_weights_host(W_u: np.ndarray, had_block: int):
    """float64 host weight [N, K] -> (Wq uint8 [N, K/2], w_scale f32 [N]) numpy arrays."""
    W = np.ascontiguousarray(W_u, dtype=np.float64)
    N, K = W.shape
    Wq = np.empty((N, K // 2), dtype=np.uint8)
    ws = np.empty((N,), dtype=np.float32)
    _check(lib().oq_quantize_weights_host(W.ctypes.data, N, K, had_block, Wq.ctypes.data, ws.ctypes.data),
           "oq_quantize_weights_host")
    return Wq, ws


def rotate_quantize_act_i8(X, had_block, s_table=None, t=0, Xq8=None, x_scale=None, stream=None):
    """W4A8 activation side: 8-bit per-token codes (int8 [M, K]) and x_scale f32 [M]."""
    M, K = X.shape
    if Xq8 is None:
        Xq8 = torch.empty((M, K), dtype=torch.int8, device=X.device)
    if x_scale is None:
        x_scale = torch.empty((M,), dtype=torch.float32, device=X.device)
    keep, sp = _s_table(s_table)
    _check(lib().oq_rotate_quantize_act_i8(_ptr(X), M, K, _ld(X), had_block, sp, t, _ptr(Xq8),
                                           _ptr(x_scale), _stream(stream)), "oq_rotate_quantize_act_i8")
    del keep
    return Xq8, x_scale


def w4a8_linear(Xq8, x_scale, Wq, w_scale, bias=None, out_dtype=OUT_F16, Y=None, stream=None):
    """Y [M, N] = dequant(Xq8 . Wq^T) with 8-bit token codes and int4 weights."""
    M, K = Xq8.shape
    N = Wq.shape[0]
    if Y is None:
        dt = torch.float16 if out_dtype == OUT_F16 else torch.bfloat16
        Y = torch.empty((M, N), dtype=dt, device=Xq8.device)
    _check(lib().oq_w4a8_linear(_ptr(Xq8), _ptr(x_scale), M, _ptr(Wq), _ptr(w_scale), _ptr(bias), N, K,
                                _ptr(Y), _ld(Y), out_dtype, _stream(stream)), "oq_w4a8_linear")
    return Y


def w4a8_gemm_i32(Xq8, Wq, acc=None, stream=None):
    M, K = Xq8.shape
    N = Wq.shape[0]
    if acc is None:
        acc = torch.empty((M, N), dtype=torch.int32, device=Xq8.device)
    _check(lib().oq_w4a8_gemm_i32(_ptr(Xq8), M, _ptr(Wq), N, K, _ptr(acc), _ld(acc), _stream(stream)),
           "oq_w4a8_gemm_i32")
    return acc


def channel_energy(W, energy=None, stream=None):
    """fp64 [K] column energies sum_n W[n][j]^2 of a device fp16 weight [N, K]."""
    N, K = W.shape
    if energy is None:
        energy = torch.empty((K,), dtype=torch.float64, device=W.device)
    _check(lib().oq_channel_energy(_ptr(W), N, K, _ld(W), _ptr(energy), _stream(stream)), "oq_channel_energy")
    return energy


def zigzag_permutation(energy, block=64, perm=None, stream=None):
    """Device zigzag permutation (int32 [K]) from device fp64 energies."""
    K = energy.shape[0]
    if perm is None:
        perm = torch.empty((K,), dtype=torch.int32, device=energy.device)
    _check(lib().oq_zigzag_permutation(_ptr(energy), K, block, _ptr(perm), _stream(stream)), "oq_zigzag_permutation")
    return perm


def block_svd(W, perm, block=64, U=None, sigma2=None, stream=None):
    """(U fp64 [K/64, 64, 64], sigma2 fp64 [K/64, 64]) of every block of the permuted weight."""
    N, K = W.shape
    nb = K // block
    if U is None:
        U = torch.empty((nb, block, block), dtype=torch.float64, device=W.device)
    if sigma2 is None:
        sigma2 = torch.empty((nb, block), dtype=torch.float64, device=W.device)
    _check(lib().oq_block_svd(_ptr(W), N, K, _ld(W), _ptr(perm), block, _ptr(U), _ptr(sigma2),
                              _stream(stream)), "oq_block_svd")
    return U, sigma2


def block_rotations(U, Rt=None, stream=None):
    """fp16 column-major blocks (int16 [nb, 64, 64]) of U_b H_64 / 8."""
    nb, c, _ = U.shape
    if Rt is None:
        Rt = torch.empty((nb, c, c), dtype=torch.int16, device=U.device)
    _check(lib().oq_block_rotations(_ptr(U), nb * c, c, _ptr(Rt), _stream(stream)), "oq_block_rotations")
    return Rt


def prepare_weights_composite(W, stream=None):
    """Device fp16 weight [N, K] -> (perm int32 [K], Rt int16 [K/64, 64, 64],
    Wq uint8 [N, K/2], w_scale f32 [N]), all on the device."""
    N, K = W.shape
    dev = W.device
    perm = torch.empty((K,), dtype=torch.int32, device=dev)
    Rt = torch.empty((K // 64, 64, 64), dtype=torch.int16, device=dev)
    Wq = torch.empty((N, K // 2), dtype=torch.uint8, device=dev)
    ws = torch.empty((N,), dtype=torch.float32, device=dev)
    nbytes = int(lib().oq_prepare_weights_workspace_bytes(K))
    work = torch.empty((max(nbytes, 16),), dtype=torch.uint8, device=dev)
    _check(lib().oq_prepare_weights_composite(_ptr(W), N, K, _ld(W), _ptr(perm), _ptr(Rt), _ptr(Wq), _ptr(ws),
                                              _ptr(work), work.numel(), _stream(stream)),
           "oq_prepare_weights_composite")
    return perm, Rt, Wq, ws


def rotate_act_f32(X, had_block, Y=None, stream=None):
    """Rotated activation y = x H_b / sqrt(b) in fp32 [M, K] (calibration input)."""
    M, K = X.shape
    if Y is None:
        Y = torch.empty((M, K), dtype=torch.float32, device=X.device)
    _check(lib().oq_rotate_act_f32(_ptr(X), M, K, _ld(X), had_block, _ptr(Y), _stream(stream)),
           "oq_rotate_act_f32")
    return Y


def calibrate_workspace_bytes(K: int) -> int:
    return int(lib().oq_calibrate_workspace_bytes(K))


def calibrate_step_scales(Y, p=99.9, qmax=7.0, delta=None, work=None, stream=None):
    """Static steps delta f32 [K] = nearest-rank p-th percentile of |Y[:, j]| / qmax."""
    n, K = Y.shape
    if delta is None:
        delta = torch.empty((K,), dtype=torch.float32, device=Y.device)
    if work is None:
        work = torch.empty((max(calibrate_workspace_bytes(K), 16),), dtype=torch.uint8, device=Y.device)
    _check(lib().oq_calibrate_step_scales(_ptr(Y), n, K, _ld(Y), float(p), float(qmax), _ptr(delta),
                                          _ptr(work), work.numel(), _stream(stream)), "oq_calibrate_step_scales")
    return delta


def calibrate_step_scales_noalloc(Y, p=99.9, qmax=7.0, delta=None, stream=None):
    """As calibrate_step_scales, with the library's own device scratch (K <=
    16384; the call itself allocates nothing; pass delta to allocate nothing
    here either)."""
    n, K = Y.shape
    if delta is None:
        delta = torch.empty((K,), dtype=torch.float32, device=Y.device)
    _check(lib().oq_calibrate_step_scales_noalloc(_ptr(Y), n, K, _ld(Y), float(p), float(qmax), _ptr(delta),
                                                  _stream(stream)), "oq_calibrate_step_scales_noalloc")
    return delta


def rotate_quantize_act_static(X, had_block, delta, Xq=None, x_scale=None, stream=None):
    """Rotation + static per-channel steps delta (f32 [K], device): (Xq uint8 [M, K/2], x_scale = 1)."""
    M, K = X.shape
    if Xq is None:
        Xq = torch.empty((M, K // 2), dtype=torch.uint8, device=X.device)
    if x_scale is None:
        x_scale = torch.empty((M,), dtype=torch.float32, device=X.device)
    _check(lib().oq_rotate_quantize_act_static(_ptr(X), M, K, _ld(X), had_block, _ptr(delta), _ptr(Xq),
                                               _ptr(x_scale), _stream(stream)), "oq_rotate_quantize_act_static")
    return Xq, x_scale


def rotate_quantize_act_static_tiled(X, had_block, delta, Xt=None, x_scale=None, stream=None):
    """As rotate_quantize_act_static, codes in the 16-row tiled layout."""
    M, K = X.shape
    if Xt is None:
        Xt = torch.empty((tiled_bytes(M, K),), dtype=torch.uint8, device=X.device)
    if x_scale is None:
        x_scale = torch.empty((M,), dtype=torch.float32, device=X.device)
    _check(lib().oq_rotate_quantize_act_static_tiled(_ptr(X), M, K, _ld(X), had_block, _ptr(delta),
                                                     _ptr(Xt), _ptr(x_scale), _stream(stream)),
           "oq_rotate_quantize_act_static_tiled")
    return Xt, x_scale


def quantize_weights_step(W_u, had_block, delta, Wq=None, w_scale=None, stream=None):
    """Device fp16 weight [N, K] rotated, scaled by the device step row delta
    (f32 [K]) per input channel and RTN-quantized: (Wq uint8 [N, K/2], w_scale f32 [N])."""
    N, K = W_u.shape
    if Wq is None:
        Wq = torch.empty((N, K // 2), dtype=torch.uint8, device=W_u.device)
    if w_scale is None:
        w_scale = torch.empty((N,), dtype=torch.float32, device=W_u.device)
    _check(lib().oq_quantize_weights_step(_ptr(W_u), N, K, _ld(W_u), had_block, _ptr(delta), _ptr(Wq),
                                          _ptr(w_scale), _stream(stream)), "oq_quantize_weights_step")
    return Wq, w_scale


def quantize_weights_step_host(W_u: np.ndarray, had_block: int, delta: np.ndarray):
    """float64 host weight [N, K] rotated, scaled by the step row delta [K] per
    input channel and RTN-quantized: (Wq uint8 [N, K/2], w_scale f32 [N])."""
    W = np.ascontiguousarray(W_u, dtype=np.float64)
    N, K = W.shape
    d = np.ascontiguousarray(delta, dtype=np.float32)
    Wq = np.empty((N, K // 2), dtype=np.uint8)
    ws = np.empty((N,), dtype=np.float32)
    _check(lib().oq_quantize_weights_step_host(W.ctypes.data, N, K, had_block, d.ctypes.data, Wq.ctypes.data,
                                               ws.ctypes.data), "oq_quantize_weights_step_host")
    return Wq, ws


from .dit import DiT  # noqa: E402,F401
