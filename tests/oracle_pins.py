"""Checks that pin the oracle to facts outside itself.

Each check takes the implementation under test as an argument, so the same
check runs on the oracle (where it must pass) and on deliberately broken
copies of it (where it must fail; see test_oracle_mutations.py).  None of
these checks calls the function it is checking to produce its expected value.
"""
from __future__ import annotations

import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load_golden_rows(name):
    rows = {}
    order = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            rows[key] = np.array([float(v) for v in vals])
            order.append(key)
    return rows


def load_golden_matrix(name):
    data = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                data.append([int(v) for v in line.split()])
    return np.array(data, dtype=np.int64)


def hadamard_by_doubling(n):
    """Textbook Sylvester construction H_2n = [[H, H], [H, -H]] (independent of
    the popcount closed form the oracle uses)."""
    h = np.ones((1, 1), dtype=np.int64)
    while h.shape[0] < n:
        h = np.block([[h, h], [h, -h]])
    return h


# --------------------------------------------------------------------------
# Hadamard
# --------------------------------------------------------------------------

def check_sylvester(sylvester):
    for e in range(0, 7):
        n = 1 << e
        h = sylvester(n)
        assert h.dtype.kind in "iu"
        assert np.array_equal(h @ h.T, n * np.eye(n, dtype=np.int64)), n
        assert np.array_equal(h, hadamard_by_doubling(n)), n
    assert np.array_equal(sylvester(8), load_golden_matrix("hadamard_8.txt"))


def check_fwht_dense(fwht, seed=1):
    """Brute force: equals x . H_n / sqrt(n) for every power of two n <= 64,
    on unit vectors and random vectors."""
    rng = np.random.default_rng(seed)
    for e in range(0, 7):
        n = 1 << e
        h = hadamard_by_doubling(n).astype(np.float64)
        eye = np.eye(n)
        assert np.allclose(fwht(eye, n), eye @ h / np.sqrt(n), rtol=0, atol=1e-15), n
        x = rng.standard_normal((5, n))
        assert np.allclose(fwht(x, n), x @ h / np.sqrt(n), rtol=0, atol=1e-13), n


def check_fwht_closed_forms(fwht, seed=2):
    rng = np.random.default_rng(seed)
    for n in (128, 1024, 16384):
        x = rng.standard_normal((3, n))
        y = fwht(x, n)
        # Parseval: the normalized transform is orthogonal.
        assert np.allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x, axis=1), rtol=1e-13, atol=0)
        # Involution: (H/sqrt(n))^2 = I.
        assert np.allclose(fwht(y, n), x, rtol=0, atol=1e-12)
        # Spike c e_i -> every entry +-c/sqrt(n).
        i = int(rng.integers(n))
        e = np.zeros((1, n))
        e[0, i] = 3.0
        ys = fwht(e, n)
        assert np.allclose(np.abs(ys), 3.0 / np.sqrt(n), rtol=1e-14, atol=0)
        # Constant c 1 -> c sqrt(n) e_0.
        c = np.full((1, n), -1.5)
        yc = fwht(c, n)
        expect = np.zeros((1, n))
        expect[0, 0] = -1.5 * np.sqrt(n)
        assert np.allclose(yc, expect, rtol=0, atol=1e-12)


def check_fwht_blockwise(fwht, seed=3):
    """Block-diagonal form: K = 4b acts as four independent b-blocks."""
    rng = np.random.default_rng(seed)
    b = 64
    h = hadamard_by_doubling(b).astype(np.float64) / np.sqrt(b)
    x = rng.standard_normal((4, 4 * b))
    y = fwht(x, b)
    for g in range(4):
        sl = slice(g * b, (g + 1) * b)
        assert np.allclose(y[:, sl], x[:, sl] @ h, rtol=0, atol=1e-13)


# --------------------------------------------------------------------------
# Quantizer
# --------------------------------------------------------------------------

def check_quantizer(quantize_sym, seed=4, qmax=7):
    """quantize_sym(z) at bit width log2(qmax + 1) + 1 (qmax 7 or 127)."""
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((64, 256)) * rng.uniform(0.01, 100, size=(64, 1))
    q, d, _ = quantize_sym(z)
    # Error bound |z - Delta q| <= Delta/2 (absmax scaling never clips).
    err = np.abs(z - d[:, None] * q)
    assert np.all(err <= d[:, None] / 2 * (1 + 1e-12))
    # The absmax element maps to +-q_max, and -(q_max + 1) never appears.
    idx = np.argmax(np.abs(z), axis=1)
    assert np.array_equal(np.abs(q[np.arange(64), idx]), np.full(64, qmax))
    assert q.min() >= -qmax and q.max() <= qmax
    assert np.allclose(d, np.max(np.abs(z), axis=1) / qmax, rtol=1e-15, atol=0)
    # Zero row -> zero codes and zero scale.
    q0, d0, _ = quantize_sym(np.zeros((2, 16)))
    assert np.all(q0 == 0) and np.all(d0 == 0)
    # All-equal-magnitude row -> every code +-q_max.
    s = np.sign(rng.standard_normal((1, 32))) * 2.5
    qs, _, _ = quantize_sym(s)
    assert np.array_equal(qs, (qmax * np.sign(s)).astype(np.int64))
    # Every code value is reachable: a ramp over [-max, max] hits all 2 q_max + 1 codes.
    ramp = np.linspace(-1.0, 1.0, 8 * qmax + 1)[None, :]
    qr, _, _ = quantize_sym(ramp)
    assert np.array_equal(np.unique(qr), np.arange(-qmax, qmax + 1))


def check_worked_example_activation(rotate_quantize_act):
    g = load_golden_rows("worked_example.txt")
    x = g["x"][None, :]
    b = int(g["b"][0])
    for s_t in (1.0, 2.0):
        q, xs, ratio = rotate_quantize_act(x, b, s_t)
        assert np.array_equal(q[0], g["q"].astype(np.int64)), s_t
        assert abs(xs[0] - g["x_scale"][0]) <= 1e-15, s_t


def check_worked_example_weight(quantize_weights):
    g = load_golden_rows("worked_example.txt")
    qw, ws, _ = quantize_weights(g["w"][None, :], 4)
    assert np.array_equal(qw[0], g["wq"].astype(np.int64))
    assert abs(ws[0] - g["w_scale"][0]) <= 1e-16


def check_st_invariance(rotate_quantize_act, seed=5):
    """Codes and x_scale do not depend on s_t in exact arithmetic; in float64
    the codes may differ only where the ratio is within 1e-9 of a half
    integer, and x_scale agrees to 1e-14 relative."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((16, 1024)).astype(np.float16).astype(np.float64)
    q1, xs1, r1 = rotate_quantize_act(x, 1024, 1.0)
    for s in (0.5, 1.7, 4.0):
        qs, xss, _ = rotate_quantize_act(x, 1024, s)
        assert np.allclose(xss, xs1, rtol=1e-14, atol=0)
        diff = qs != q1
        near = np.abs(np.abs(r1 - np.floor(r1)) - 0.5) < 1e-9
        assert np.all(~diff | near)


# --------------------------------------------------------------------------
# Integer product and epilogue
# --------------------------------------------------------------------------

def triple_loop(q, qw):
    M, K = q.shape
    N = qw.shape[0]
    acc = np.zeros((M, N), dtype=np.int64)
    for i in range(M):
        for n in range(N):
            s = 0
            for k in range(K):
                s += int(q[i, k]) * int(qw[n, k])
            acc[i, n] = s
    return acc


def check_int_gemm(int_gemm, seed=6):
    rng = np.random.default_rng(seed)
    for (M, N, K) in ((1, 1, 2), (3, 5, 8), (7, 4, 16), (5, 9, 34)):
        q = rng.integers(-7, 8, size=(M, K))
        qw = rng.integers(-7, 8, size=(N, K))
        assert np.array_equal(int_gemm(q, qw), triple_loop(q, qw)), (M, N, K)
    # +-identity weights return +-codes; all-ones weights return row sums.
    K = 32
    q = rng.integers(-7, 8, size=(6, K))
    eye = np.eye(K, dtype=np.int64)
    assert np.array_equal(int_gemm(q, eye), q)
    assert np.array_equal(int_gemm(q, -eye), -q)
    assert np.array_equal(int_gemm(q, np.ones((3, K), np.int64)), np.repeat(q.sum(1, keepdims=True), 3, 1))
    # Extreme magnitudes: every code +-7 at K = 16384 gives +-49 K exactly.
    big = np.full((2, 16384), 7, np.int64)
    big[1] = -7
    assert np.array_equal(int_gemm(big, big[:1]), np.array([[49 * 16384], [-49 * 16384]]))


def check_dequant(dequant):
    g = load_golden_rows("worked_example.txt")
    acc = g["acc"].astype(np.int64)[None, :]
    y = dequant(acc, g["x_scale"], g["ws"], g["bias"])
    assert np.allclose(y[0], g["out"], rtol=1e-15, atol=1e-15)
    # Unit scales and no bias return the accumulator itself.
    acc2 = np.array([[3, -5], [0, 123456]], np.int64)
    assert np.array_equal(dequant(acc2, np.ones(2), np.ones(2)), acc2.astype(np.float64))


def check_worked_example_gemm(int_gemm):
    g = load_golden_rows("worked_example.txt")
    q = g["q"].astype(np.int64)[None, :]
    qw = np.stack([g["qw0"], g["qw1"]]).astype(np.int64)
    assert np.array_equal(int_gemm(q, qw)[0], g["acc"].astype(np.int64))


# --------------------------------------------------------------------------
# Full composite rotation (zigzag permutation, per-block SVD factor, Hadamard)
# --------------------------------------------------------------------------

def random_orthogonal(rng, n):
    a = rng.standard_normal((n, n))
    q, r = np.linalg.qr(a)
    return q * np.sign(np.diag(r))


def check_zigzag(zigzag_permutation, seed=20):
    g = load_golden_rows("zigzag_example.txt")
    perm = zigzag_permutation(g["energy"], 2)
    assert np.array_equal(np.asarray(perm), g["perm"].astype(np.int64))
    rng = np.random.default_rng(seed)
    for K, B in ((64, 4), (96, 3), (128, 16), (256, 4)):
        e = rng.exponential(size=K)
        e[rng.choice(K, 5, replace=False)] = e[0]  # ties
        perm = np.asarray(zigzag_permutation(e, B))
        c = K // B
        assert np.array_equal(np.sort(perm), np.arange(K)), "not a permutation"
        # every block takes exactly one channel from each run of B consecutive
        # ranks of the descending order
        rank = np.empty(K, dtype=np.int64)
        rank[np.array(sorted(range(K), key=lambda j: (-e[j], j)))] = np.arange(K)
        for b in range(B):
            rounds = np.sort(rank[perm[b * c:(b + 1) * c]] // B)
            assert np.array_equal(rounds, np.arange(c)), "a block skips a round"
        # block energies differ by at most the spread of all energies
        sums = np.array([e[perm[b * c:(b + 1) * c]].sum() for b in range(B)])
        assert sums.max() - sums.min() <= e.max() - e.min() + 1e-12


def check_block_svd(block_svd_factors, seed=21):
    """The paper's statement after the SVD rotation: row i of U_b^T W_b has
    squared norm sigma_i^2, with sigma_i^2 taken here from the eigenvalues of
    W_b W_b^T (a different routine); U_b orthogonal."""
    rng = np.random.default_rng(seed)
    N, K, c = 40, 32, 8
    w = rng.standard_normal((N, K)) * np.exp(rng.standard_normal(K))[None, :]
    perm = rng.permutation(K)
    u, _ = block_svd_factors(w, perm, c)
    u = np.asarray(u)
    assert u.shape == (K // c, c, c)
    for b in range(K // c):
        wb = w[:, perm][:, b * c:(b + 1) * c].T
        assert np.allclose(u[b].T @ u[b], np.eye(c), atol=1e-12)
        energy = np.sum((u[b].T @ wb) ** 2, axis=1)
        ev = np.sort(np.linalg.eigvalsh(wb @ wb.T))[::-1]
        assert np.allclose(energy, ev, rtol=1e-10, atol=1e-10)
        # U_b^T W_b = Sigma V^T has mutually orthogonal rows: U_b diagonalizes W_b W_b^T
        g = (u[b].T @ wb) @ (u[b].T @ wb).T
        assert np.max(np.abs(g - np.diag(np.diag(g)))) <= 1e-10 * np.max(np.abs(g))


def check_canonical_signs(canonical_signs, seed=25):
    """Hand example, then: the largest-magnitude entry of every column is
    positive, columns equal +-the input's, orthogonality kept, idempotent."""
    u = np.array([[0.6, -0.8], [-0.8, -0.6]])
    assert np.array_equal(np.asarray(canonical_signs(u)), np.array([[-0.6, 0.8], [0.8, 0.6]]))
    tie = np.array([[-0.5, 1.0], [0.5, 0.0]])  # first entry wins a magnitude tie
    assert np.array_equal(np.asarray(canonical_signs(tie)), np.array([[0.5, 1.0], [-0.5, 0.0]]))
    rng = np.random.default_rng(seed)
    q = np.stack([random_orthogonal(rng, 16) for _ in range(3)])
    c = np.asarray(canonical_signs(q))
    for b in range(3):
        idx = np.argmax(np.abs(c[b]), axis=0)
        assert np.all(c[b][idx, np.arange(16)] > 0)
        assert np.allclose(np.abs(c[b]), np.abs(q[b]), atol=0)
        assert np.all(np.isin(np.sign(c[b] * q[b]).sum(0) / 16, [-1.0, 1.0]))
        assert np.allclose(c[b].T @ c[b], np.eye(16), atol=1e-12)
    assert np.array_equal(np.asarray(canonical_signs(c)), c)


def check_block_rotations(block_rotations, seed=22):
    rng = np.random.default_rng(seed)
    for c in (8, 64):
        u = np.stack([random_orthogonal(rng, c) for _ in range(3)])
        r = np.asarray(block_rotations(u))
        for b in range(3):
            assert np.allclose(r[b] @ r[b].T, np.eye(c), atol=1e-12), "not orthogonal"
        # U = I leaves the normalized Hadamard matrix: a spike maps to +-1/sqrt(c)
        ri = np.asarray(block_rotations(np.eye(c)[None]))[0]
        assert np.allclose(np.abs(ri), 1.0 / np.sqrt(c), atol=1e-15)
        assert np.allclose(ri[0], 1.0 / np.sqrt(c)) and np.allclose(ri[:, 0], 1.0 / np.sqrt(c))


def check_rotate_composite(rotate_composite, block_rotations, fwht, seed=23):
    rng = np.random.default_rng(seed)
    M, N, K, c = 6, 20, 256, 64
    x = rng.standard_normal((M, K))
    # identity permutation with U_b = I is the block Walsh-Hadamard transform
    r_id = np.asarray(block_rotations(np.stack([np.eye(c)] * (K // c))))
    assert np.allclose(rotate_composite(x, np.arange(K), r_id), fwht(x, c), atol=1e-12)
    # R_b = I leaves the gather (X P)[:, k] = X[:, perm[k]]
    perm = rng.permutation(K)
    eye = np.stack([np.eye(c)] * (K // c))
    assert np.array_equal(rotate_composite(x, perm, eye), x[:, perm])
    # invariance of the linear: (X P R)(W P R)^T = X W^T for orthogonal R
    u = np.stack([random_orthogonal(rng, c) for _ in range(K // c)])
    r = np.asarray(block_rotations(u))
    w = rng.standard_normal((N, K))
    lhs = rotate_composite(x, perm, r) @ rotate_composite(w, perm, r).T
    ref = x @ w.T
    assert np.max(np.abs(lhs - ref)) <= 1e-12 * np.max(np.abs(ref)) * K
    # energy equalization (the purpose of U_b H_c): with U_b the left singular
    # vectors of the block's weight rows (here eigenvectors of W_b W_b^T), every
    # rotated weight row of the block carries the block's mean sigma^2
    wp = w[:, perm]
    ub = []
    for b in range(K // c):
        wb = wp[:, b * c:(b + 1) * c].T
        ev, vec = np.linalg.eigh(wb @ wb.T)
        ub.append(vec[:, ::-1])
    r = np.asarray(block_rotations(np.stack(ub)))
    wr = rotate_composite(w, perm, r)
    for b in range(K // c):
        wb = wp[:, b * c:(b + 1) * c].T
        energy = np.sum(wr[:, b * c:(b + 1) * c] ** 2, axis=0)
        assert np.allclose(energy, np.trace(wb @ wb.T) / c, rtol=1e-10), "block energy not equalized"


def check_rotate_quantize_composite(rqc, rotate_quantize_act, seed=24):
    """Identity permutation and U_b = I: the composite path is the Hadamard
    path (block c); quantizer bound |z - Delta q| <= Delta / 2 in general."""
    rng = np.random.default_rng(seed)
    M, K, c = 5, 128, 64
    x = rng.standard_normal((M, K))
    h = np.array([[1.0]])
    while h.shape[0] < c:
        h = np.block([[h, h], [h, -h]])
    r_id = np.stack([h / np.sqrt(c)] * (K // c))
    q1, xs1, _ = rqc(x, np.arange(K), r_id, 2.5)
    q2, xs2, _ = rotate_quantize_act(x, c, 2.5)
    assert np.array_equal(q1, q2) and np.allclose(xs1, xs2, rtol=1e-14)
    perm = rng.permutation(K)
    r = np.stack([random_orthogonal(rng, c) for _ in range(K // c)])
    q, xs, _ = rqc(x, perm, r, 1.0)
    y = x[:, perm].reshape(M, K // c, c)
    y = np.einsum("mbi,bij->mbj", y, r).reshape(M, K)
    assert np.all(np.abs(y - xs[:, None] * q) <= xs[:, None] / 2 * (1 + 1e-12))
    assert np.all(np.abs(q).max(axis=1) == 7)


# --------------------------------------------------------------------------
# Per-step static scales
# --------------------------------------------------------------------------

# Nearest ranks k = ceil(p n / 100) worked out by hand: p = 99.9 selects the
# 999th of 1000, the 1998th of 2000, the 9990th of 10000 (never the maximum
# when p n / 100 is a whole number), the 1000th of 1001 (1000.0 -> 1000 ...
# 99.9 * 1001 / 100 = 999.999 -> 1000), the 7th of 7 and the 1st of 1; p = 50
# the 500th of 1000 and the 4th of 7; p = 100 the last.
PERCENTILE_RANKS = {(99.9, 1000): 999, (99.9, 2000): 1998, (99.9, 10000): 9990, (99.9, 1001): 1000,
                    (99.9, 7): 7, (99.9, 1): 1, (50.0, 1000): 500, (50.0, 7): 4, (100.0, 1001): 1001}


def check_percentile(percentile_abs, seed=50):
    rng = np.random.default_rng(seed)
    for (p, n), k in PERCENTILE_RANKS.items():
        # distinct magnitudes 1..n in a random order: the k-th smallest is k
        y = (rng.permutation(n) + 1.0) * np.where(rng.random(n) < 0.5, -1.0, 1.0)
        v = np.asarray(percentile_abs(y[:, None], p))
        assert v.shape == (1,) and v[0] == float(k), (p, n, v, k)
    for n in (1, 7, 1000, 1001):
        y = rng.standard_normal((n, 5)) * np.array([1, 10, 0.1, 3, 0])
        for p in (50.0, 99.9, 100.0):
            v = np.asarray(percentile_abs(y, p))
            a = np.abs(y)
            k = PERCENTILE_RANKS.get((p, n))
            for j in range(5):
                # v is an element of the column; with the hand-worked rank, at
                # least k values are <= v and fewer than k below it
                assert v[j] in a[:, j]
                if k is not None:
                    assert np.count_nonzero(a[:, j] <= v[j]) >= k
                    assert np.count_nonzero(a[:, j] < v[j]) < k
            if p == 100.0:
                assert np.array_equal(v, a.max(axis=0))


def check_quantize_static(quantize_static, seed=51):
    rng = np.random.default_rng(seed)
    y = rng.standard_normal((64, 32)) * 3
    d = np.abs(rng.standard_normal(32)) * 0.5 + 0.05
    d[3] = 0.0
    q, _ = quantize_static(y, d)
    q = np.asarray(q)
    assert q.min() >= -7 and q.max() <= 7
    assert not q[:, 3].any()
    live = np.abs(y) <= 7 * d[None, :]
    live[:, 3] = False
    err = np.abs(y - d[None, :] * q)
    assert np.all(err[live] <= d[None, :].repeat(64, 0)[live] / 2 + 1e-15), "unclipped error above Delta/2"
    big = np.abs(y) >= 7.5 * d[None, :]
    big[:, 3] = False
    assert np.all(np.abs(q[big]) == 7) and np.all(np.sign(q[big]) == np.sign(y[big])), "clipping"
    # a constant step equal to the row maximum / 7 is the per-token quantizer on that row
    row = y[:1]
    dd = np.full(32, np.abs(row).max() / 7)
    qs, _ = quantize_static(row, dd)
    qt = np.clip(np.rint(row / dd[0]), -7, 7)
    assert np.array_equal(np.asarray(qs), qt)


def check_fold_step(fold_weights_step, fwht, seed=52):
    """Activations on the step grid (y = Delta_j * integer, no activation
    error): the folded weight applied to the integer codes reproduces y W'^T
    up to the weight's own RTN error bound; folding into the wrong axis fails."""
    rng = np.random.default_rng(seed)
    M, N, K, b = 6, 40, 64, 64
    d = np.exp(rng.standard_normal(K))
    q = rng.integers(-7, 8, size=(M, K))
    y = q * d[None, :]
    w = rng.standard_normal((N, K))
    qw, ws, _ = fold_weights_step(w, b, d)
    out = (q @ np.asarray(qw).T) * np.asarray(ws)[None, :]
    wp = fwht(w, b)
    ref = y @ wp.T
    # |W'' - ws qw| <= ws / 2 elementwise, so the output error is bounded by
    # sum_j |q_j| ws / 2
    bound = np.abs(q).sum(axis=1)[:, None] * np.asarray(ws)[None, :] / 2
    assert np.all(np.abs(out - ref) <= bound * (1 + 1e-12))


# --------------------------------------------------------------------------
# W4A8 (8-bit per-token activations against int4 weights)
# --------------------------------------------------------------------------

def check_w4a8_worked_example(w4a8_linear):
    g = load_golden_rows("w4a8_example.txt")
    x = g["x"][None, :]
    b = int(g["b"][0])
    w = np.stack([g["w0"], g["w1"]])
    r = w4a8_linear(x, w, b)
    assert np.array_equal(r["q"][0], g["q"].astype(np.int64))
    assert abs(r["x_scale"][0] - g["x_scale"][0]) <= 1e-17
    assert np.array_equal(r["qw"], np.stack([g["qw0"], g["qw1"]]).astype(np.int64))
    assert np.allclose(r["w_scale"], g["ws"], rtol=1e-15, atol=0)
    assert np.array_equal(r["acc"][0], g["acc"].astype(np.int64))
    assert np.allclose(r["y"][0], g["out"], rtol=1e-14, atol=0)
    # s_t invariance carries over to the 8-bit quantizer
    r2 = w4a8_linear(x, w, b, s_t=2.0)
    assert np.array_equal(r2["q"], r["q"]) and abs(r2["x_scale"][0] - r["x_scale"][0]) <= 1e-17


def check_w4a8_error_bound(w4a8_linear, fwht, seed=60):
    """|y - x W'^T| is bounded by the two rounding errors: per element
    |y_k - Delta_x q_k| <= Delta_x / 2 and |w'_nk - Delta_w qw_nk| <= Delta_w / 2,
    so |err_in| <= sum_k (Delta_x/2 |w'_nk| + |x'_k| Delta_w/2 + Delta_x Delta_w / 4).
    An 8-bit activation must also beat the 4-bit one on the same inputs."""
    rng = np.random.default_rng(seed)
    M, N, K, b = 8, 16, 256, 64
    x = rng.standard_normal((M, K))
    w = rng.standard_normal((N, K)) * 0.1
    r = w4a8_linear(x, w, b)
    xp, wp = fwht(x, b), fwht(w, b)
    exact = xp @ wp.T
    dx, dw = r["x_scale"][:, None], r["w_scale"][None, :]
    bound = (dx / 2) * np.abs(wp).sum(1)[None, :] + (dw / 2) * np.abs(xp).sum(1)[:, None] + K * dx * dw / 4
    assert np.all(np.abs(r["y"] - exact) <= bound * (1 + 1e-12))
    assert np.abs(r["q"]).max() == 127


# --------------------------------------------------------------------------
# DiT block composition (two tiny blocks worked by hand, every quantization
# exact; tests/golden/dit_block_pi.txt and dit_block_gr00t.txt)
# --------------------------------------------------------------------------

def _tiny_dit_cfg(arch):
    from types import SimpleNamespace
    return SimpleNamespace(arch=arch, hidden=4, mlp=4, n_heads=1, head_dim=4, steps=1)


def _mat(v, cols):
    return np.asarray(v, dtype=np.float64).reshape(-1, cols)


def _check_named(out, g, prefix, names, tag):
    for nm in names:
        exp = _mat(g[prefix + nm], len(out[nm][0]) if np.ndim(out[nm]) == 2 else 1)
        got = np.asarray(out[nm], dtype=np.float64).reshape(exp.shape)
        assert np.allclose(got, exp, rtol=1e-12, atol=1e-12), (tag, nm, got, exp)


def check_dit_block_pi(block_trace, quantize_block_weights):
    g = load_golden_rows("dit_block_pi.txt")
    cfg = _tiny_dit_cfg("pi")
    blk = {"g1": g["g1"], "g2": g["g2"], "wqkv": _mat(g["wqkv"], 4), "wo": _mat(g["wo"], 4),
           "wgu": _mat(g["wgu"], 4), "wd": _mat(g["wd"], 4)}
    w = {"blocks": [blk]}
    mod = [[{k: g[k] for k in ("sc1", "sh1", "gt1", "sc2", "sh2", "gt2")}]]
    s_table = g["s"].reshape(1, 1, 4)
    prefix = (g["kp"].reshape(1, 1, 2, 4), g["vp"].reshape(1, 1, 2, 4))
    qb = quantize_block_weights(cfg, w["blocks"])
    out = block_trace(cfg, w, qb, mod, s_table, _mat(g["r"], 4), 0, 0, 1, 1, prefix=prefix)
    _check_named(out, g, "", ("h1", "qkv", "attn", "r1", "h2", "gate_up", "act", "r_out"), "pi")


def check_dit_block_gr00t(block_trace, quantize_block_weights, cond_kv):
    g = load_golden_rows("dit_block_gr00t.txt")
    cfg = _tiny_dit_cfg("gr00t")
    blocks, mod = [], []
    for l, lin in ((0, ("wq", "wkv", "wo", "wff0", "wff2")), (1, ("wqkv", "wo", "wff0", "wff2"))):
        p = f"b{l}_"
        blk = {"g1": g[p + "g1"], "g3": g[p + "g3"], "beta3": g[p + "beta3"]}
        for nm in lin:
            blk[nm] = _mat(g[p + nm], 4)
        blocks.append(blk)
        mod.append([{"sc1": g[p + "sc1"], "sh1": g[p + "sh1"]}])
    w = {"blocks": blocks}
    s_table = np.stack([g["s"], g["s"][::-1]]).reshape(2, 1, 4)
    qb = quantize_block_weights(cfg, blocks)
    ckv = cond_kv(cfg, qb, g["cond"].reshape(2, 2, 4))
    assert np.allclose(ckv[0].reshape(-1), g["ckv"], rtol=0, atol=1e-12), ckv[0]
    for l, site0 in ((0, "q"), (1, "qkv")):
        out = block_trace(cfg, w, qb, mod, s_table, _mat(g[f"b{l}_r"], 4), l, 0, 2, 1, ckv=ckv)
        _check_named(out, g, f"b{l}_", ("h1", site0, "attn", "r1", "h2", "gate_up", "act", "r_out"),
                     f"gr00t block {l}")
