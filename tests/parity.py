"""Helpers of the GPU-vs-oracle parity tests (test code; shares nothing with
the HIP path).

Tolerances (the three bars of the parity criterion):
  * int4 codes: bit-exact, except elements whose exact ratio r = z/Delta lies
    within the fp32 error bound tau of a rounding boundary (a half integer);
    such a mismatch must be exactly one code, and the count must stay below
    1e-4 of the elements.
  * int32 accumulators: bit-exact when the oracle is fed the GPU's codes.
  * fp16 / bf16 outputs: relative L2 error <= 2e-3 against the oracle fed the
    same codes and scales.

tau.  The kernel forms the unnormalized transform u in fp32 with a summation
tree of depth d, so |u_hat - u| <= gamma_d * l1 with gamma_d = d 2^-24 /
(1 - d 2^-24) and l1 the largest per-block sum of |x|.  The first five
butterfly stages may run on the matrix cores as one 32-term fp32 sum whose
internal order is not specified; bounding it as a sequential sum (31 adds)
gives d <= log2(b) - 5 + 31 + 1 < log2(b) + 32.
The row maximum inherits the same error, and three more fp32 roundings form
the multiplier g ~ 7 / max|u|.  Hence
    |r_gpu - r_exact| <= 14 gamma_d l1 / max|u| + 21 * 2^-24  =: tau_row.
"""
from __future__ import annotations

import numpy as np

U32 = 2.0 ** -24
CODE_MISMATCH_FRAC = 1e-4
REL_L2_OUT = 2e-3


def unpack_int4(packed: np.ndarray) -> np.ndarray:
    """uint8 [R, K/2] (low nibble = even channel, two's complement) -> int64 [R, K]."""
    p = np.asarray(packed, dtype=np.uint8)
    lo = (p & 0xF).astype(np.int64)
    hi = (p >> 4).astype(np.int64)
    lo = np.where(lo >= 8, lo - 16, lo)
    hi = np.where(hi >= 8, hi - 16, hi)
    out = np.empty(p.shape[:-1] + (2 * p.shape[-1],), dtype=np.int64)
    out[..., 0::2] = lo
    out[..., 1::2] = hi
    return out


def tau_rows(x: np.ndarray, b: int, qmax: int = 7) -> np.ndarray:
    """Per-row bound on |r_gpu - r_exact| for activation rows x [M, K]; the
    constants 14 = 2 q_max and 21 = 3 q_max scale with q_max (127 for the
    8-bit activations of W4A8)."""
    x = np.asarray(x, dtype=np.float64)
    M, K = x.shape
    d = int(np.log2(b)) + 32
    gamma = d * U32 / (1 - d * U32)
    l1 = np.abs(x).reshape(M, K // b, b).sum(axis=2).max(axis=1)
    # max|u| (unnormalized) = sqrt(b) * max|y|; recomputed from the data.
    from oracle.hadamard import fwht  # the oracle's transform, exact to ~1e-15
    umax = np.abs(fwht(x, b)).max(axis=1) * np.sqrt(b)
    safe = np.where(umax > 0, umax, 1.0)
    return np.where(umax > 0, 2 * qmax * gamma * l1 / safe + 3 * qmax * U32, 0.0)


def block_l1(x: np.ndarray, b: int) -> np.ndarray:
    """Per element: the sum of |x| over the Hadamard block that holds it [M, K]."""
    x = np.asarray(x, dtype=np.float64)
    M, K = x.shape
    l1 = np.abs(x).reshape(M, K // b, b).sum(axis=2)
    return np.repeat(l1, b, axis=1)


def tau_rotate(x: np.ndarray, b: int, y_ref: np.ndarray) -> np.ndarray:
    """Elementwise bound on |y_gpu - y_exact| for the fp32 rotation output:
    the butterfly error gamma_d l1 / sqrt(b) and two roundings of the
    normalization (the factor 1 / sqrt(b) and the product)."""
    d = int(np.log2(b)) + 32
    gamma = d * U32 / (1 - d * U32)
    return gamma * block_l1(x, b) / np.sqrt(b) + 2 * U32 * np.abs(y_ref)


def tau_static(x: np.ndarray, b: int, delta: np.ndarray, r_ref: np.ndarray) -> np.ndarray:
    """Elementwise bound on |r_gpu - r_exact| of the static quantizer, r =
    y / Delta_j formed as u * (fl(1 / sqrt(b)) * rcp(Delta_j)): the butterfly
    error divided by sqrt(b) Delta_j, plus relative roundings of the factor,
    the hardware reciprocal (one ulp), their product and the final product
    (at most 6 * 2^-24 |r| together).  Zero where the step is not positive."""
    d = int(np.log2(b)) + 32
    gamma = d * U32 / (1 - d * U32)
    dl = np.asarray(delta, dtype=np.float64)
    ok = (dl > 0) & np.isfinite(dl)
    safe = np.where(ok, dl, 1.0)
    t = gamma * block_l1(x, b) / (np.sqrt(b) * safe[None, :]) + 6 * U32 * np.abs(r_ref)
    return np.where(ok[None, :], t, 0.0)


def tau_rows_scaled(x: np.ndarray, b: int, cm: np.ndarray) -> np.ndarray:
    """Per-row bound for the per-row quantizer of the rotated row scaled by
    cm per channel (the per-step weight fold): the fp32 butterfly error
    gamma_d l1 of each channel's block, times cm_j, relative to the row
    maximum of |u cm|, plus one more rounding (the product by cm) on top of
    the per-token kernel's 21 * 2^-24."""
    x = np.asarray(x, dtype=np.float64)
    cm = np.asarray(cm, dtype=np.float64)
    M, K = x.shape
    d = int(np.log2(b)) + 32
    gamma = d * U32 / (1 - d * U32)
    l1 = block_l1(x, b) * cm[None, :]
    from oracle.hadamard import fwht
    umax = np.abs(fwht(x, b) * cm[None, :]).max(axis=1) * np.sqrt(b)
    safe = np.where(umax > 0, umax, 1.0)
    return np.where(umax > 0, 14 * gamma * l1.max(axis=1) / safe + 28 * U32, 0.0)


def dist_to_boundary(r: np.ndarray) -> np.ndarray:
    """Distance of each ratio to the nearest half integer."""
    return np.abs(np.abs(r - np.floor(r)) - 0.5)


# Running totals over every check_codes call of the session (reported at the
# end of the run by tests/conftest.py): elements compared, code mismatches,
# mismatches whose exact ratio lies more than one fp32 ulp from the rounding
# boundary, elements within one ulp of a boundary, and the largest measured
# |r_gpu - r_exact| in fp32 ulps of r_exact (where the GPU's ratios are known).
STATS = {"elements": 0, "mismatches": 0, "mismatches_beyond_1ulp": 0, "within_1ulp": 0,
         "ratio_elements": 0, "max_ratio_err_ulp": 0.0}


def ulp32(r) -> np.ndarray:
    """One fp32 ulp at |r|, taken at least at 0.5 (the nearest rounding
    boundary of a ratio below 0.5 is 0.5 itself), as float64."""
    a = np.maximum(np.abs(np.asarray(r, dtype=np.float64)), 0.5)
    return np.spacing(a.astype(np.float32)).astype(np.float64)


def check_codes(q_gpu, q_ref, r_ref, tau_row, qmax: int = 7, r_gpu=None, record=True):
    """Returns (n_mismatch, n_boundary_1ulp) and asserts the code criterion.
    r_gpu: optionally the GPU's own pre-rounding ratios, to measure their
    distance from the exact ones in fp32 ulps.  record: add to STATS (off
    where q_ref is not the oracle's)."""
    q_gpu = np.asarray(q_gpu)
    q_ref = np.asarray(q_ref)
    mism = q_gpu != q_ref
    n = int(mism.sum())
    total = q_ref.size
    tau = np.asarray(tau_row, dtype=np.float64)
    dist = dist_to_boundary(r_ref)
    near = dist <= (tau if tau.ndim == 2 else tau[:, None])
    if n:
        assert np.all(np.abs(q_gpu[mism] - q_ref[mism]) == 1), "a code differs by more than one step"
        assert np.all(near[mism]), "a code differs away from a rounding boundary"
    assert n <= CODE_MISMATCH_FRAC * total, f"{n} code mismatches of {total}"
    assert q_gpu.min() >= -qmax and q_gpu.max() <= qmax, f"code outside [-{qmax}, {qmax}]"
    ulp = ulp32(r_ref)
    within = dist <= ulp
    n_ulp = int(within.sum())
    if not record:
        return n, n_ulp
    STATS["elements"] += int(total)
    STATS["mismatches"] += n
    STATS["mismatches_beyond_1ulp"] += int((mism & ~within).sum())
    STATS["within_1ulp"] += n_ulp
    if r_gpu is not None:
        err = np.abs(np.asarray(r_gpu, dtype=np.float64) - r_ref) / ulp
        STATS["ratio_elements"] += int(err.size)
        STATS["max_ratio_err_ulp"] = max(STATS["max_ratio_err_ulp"], float(err.max()) if err.size else 0.0)
    return n, n_ulp


def rel_l2(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (den if den > 0 else 1.0))


def pack_int4(codes: np.ndarray) -> np.ndarray:
    """int [R, K] codes in [-8, 7] -> uint8 [R, K/2], low nibble = even channel."""
    c = np.asarray(codes, dtype=np.int64) & 0xF
    return (c[..., 0::2] | (c[..., 1::2] << 4)).astype(np.uint8)
