"""Full composite rotation of Section 4.1, oracle side (test infrastructure only).

Section 4.1, "Block-wise Implementation" and eq:blockdiag / eq:transform: the
activation is multiplied by P R_hat, where P is a channel permutation and
R_hat = BlockDiag(R_1 .. R_K) with R_b = U_b H_c (U_b the left singular
vectors of the weight rows of block b, H_c the normalized Hadamard matrix of
the block size c).  The weight gets the transposed transform, so that
X' W' = X P R_hat R_hat^T P^T W = X W.

Orientation here (as in the rest of the oracle): activations are [M, K] rows,
the weight is stored [N, K] (output-major), so the paper's W (C_in x C_out) is
W_ours^T.  The paper's weight row j (input channel j) is column j of W_ours.

Readings (listed with the others in the design notes):
  * P: channels sorted by descending energy ||W_{j,:}||^2 (paper orientation,
    i.e. the sum of squares of column j of W_ours), ties to the lower index,
    then dealt to the K blocks in snake (zigzag) order: sorted position i goes
    to round r = i // K, block r-even ? i % K : K - 1 - i % K, slot r.
    perm[b*c + r] is the source channel of slot r of block b, so that
    (X P)[:, k] = X[:, perm[k]].
  * U_b: left singular vectors of W_b = (W_ours[:, perm])[:, block b]^T, a
    c x N matrix (the c x c factor; the printed U_SVD(W_b^T) has the wrong
    dimension for a block of c channels).
  * R_b = U_b . H_c / sqrt(c).  The GPU path receives R_b rounded to fp16 and
    the oracle is then fed the same rounded values (as float64).

Pins: a hand-worked zigzag example (golden fixture), permutation and balance
properties; the paper's row-energy statement ||(U_b^T W_b)_i||^2 = sigma_i^2
checked against eigenvalues of W_b W_b^T (a different routine); orthogonality
of R_b; rotation invariance of the linear in float64; identity permutation
with U_b = I reduces to the block Walsh-Hadamard transform of hadamard.fwht.
"""
from __future__ import annotations

import numpy as np

from .hadamard import sylvester
from .quant import quantize_sym


def zigzag_permutation(energy: np.ndarray, n_blocks: int) -> np.ndarray:
    """perm (int64 [K]) from per-channel energies: descending sort (ties to the
    lower index), snake order over n_blocks blocks of K / n_blocks slots."""
    e = np.asarray(energy, dtype=np.float64)
    K = e.shape[0]
    if K % n_blocks:
        raise ValueError("channel count must be a multiple of the block count")
    c = K // n_blocks
    order = sorted(range(K), key=lambda j: (-e[j], j))
    perm = np.empty(K, dtype=np.int64)
    for i, ch in enumerate(order):
        r, p = divmod(i, n_blocks)
        b = p if r % 2 == 0 else n_blocks - 1 - p
        perm[b * c + r] = ch
    return perm


def channel_energy(w_ours: np.ndarray) -> np.ndarray:
    """||W_{j,:}||^2 of the paper's orientation = sum over outputs of column j."""
    w = np.asarray(w_ours, dtype=np.float64)
    return np.sum(w * w, axis=0)


def block_svd_factors(w_ours: np.ndarray, perm: np.ndarray, c: int):
    """U_b (c x c) and singular values of every block of the permuted weight."""
    w = np.asarray(w_ours, dtype=np.float64)[:, perm]
    K = w.shape[1]
    us, ss = [], []
    for b in range(K // c):
        wb = w[:, b * c:(b + 1) * c].T  # c x N, rows = the block's input channels
        u, s, _ = np.linalg.svd(wb, full_matrices=True)
        us.append(u)
        ss.append(s)
    return np.stack(us), ss


def canonical_signs(u: np.ndarray) -> np.ndarray:
    """Each column of u (or of every matrix in a stack) multiplied by -1 when
    its entry of largest magnitude (the first one on ties) is negative.  A
    singular vector is defined up to its sign; this fixes one representative
    so that two computations of U_b can be compared column by column."""
    u = np.array(u, dtype=np.float64, copy=True)
    mats = u if u.ndim == 3 else u[None]
    for m in mats:
        for j in range(m.shape[1]):
            r = int(np.argmax(np.abs(m[:, j])))
            if m[r, j] < 0:
                m[:, j] = -m[:, j]
    return u


def block_rotations(u_blocks: np.ndarray) -> np.ndarray:
    """R_b = U_b . H_c / sqrt(c) for every block (float64 [K/c, c, c])."""
    u = np.asarray(u_blocks, dtype=np.float64)
    c = u.shape[-1]
    h = sylvester(c).astype(np.float64) / np.sqrt(float(c))
    return np.stack([ub @ h for ub in u])


def rotate_composite(x: np.ndarray, perm: np.ndarray, r_blocks: np.ndarray) -> np.ndarray:
    """y = x P R_hat: gather the channels by perm, then multiply block b of
    every row by R_b (float64)."""
    x = np.asarray(x, dtype=np.float64)[:, perm]
    r = np.asarray(r_blocks, dtype=np.float64)
    nb, c, _ = r.shape
    M = x.shape[0]
    y = np.empty_like(x)
    for b in range(nb):
        y[:, b * c:(b + 1) * c] = x[:, b * c:(b + 1) * c] @ r[b]
    assert y.shape == (M, nb * c)
    return y


def rotate_quantize_composite(x: np.ndarray, perm: np.ndarray, r_blocks: np.ndarray, s_t: float = 1.0):
    """Online composite transform, step scale and per-token int4 quantizer
    (eq:transform, eq:perstep_scale in the scalar reading, eq:scale, eq:quant).
    Returns (q [M,K] int64, x_scale [M] = Delta / s_t, ratio [M,K])."""
    y = rotate_composite(x, perm, r_blocks)
    s = float(s_t)
    q, delta, ratio = quantize_sym(s * y)
    return q, delta / s, ratio


def fold_weights_composite(w_ours: np.ndarray, perm: np.ndarray, r_blocks: np.ndarray):
    """W'_ours = W_ours P R_hat (the paper's W' = R_hat^T P^T W in the
    output-major storage) quantized per output channel with RTN.  Returns
    (qw [N,K] int64, w_scale [N], ratio [N,K])."""
    return quantize_sym(rotate_composite(w_ours, perm, r_blocks))
