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

def check_quantizer(quantize_sym, seed=4):
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((64, 256)) * rng.uniform(0.01, 100, size=(64, 1))
    q, d, _ = quantize_sym(z)
    # Error bound |z - Delta q| <= Delta/2 (absmax scaling never clips).
    err = np.abs(z - d[:, None] * q)
    assert np.all(err <= d[:, None] / 2 * (1 + 1e-12))
    # The absmax element maps to +-7, and -8 never appears.
    idx = np.argmax(np.abs(z), axis=1)
    assert np.array_equal(np.abs(q[np.arange(64), idx]), np.full(64, 7))
    assert q.min() >= -7 and q.max() <= 7
    assert np.allclose(d, np.max(np.abs(z), axis=1) / 7, rtol=1e-15, atol=0)
    # Zero row -> zero codes and zero scale.
    q0, d0, _ = quantize_sym(np.zeros((2, 16)))
    assert np.all(q0 == 0) and np.all(d0 == 0)
    # All-equal-magnitude row -> every code +-7.
    s = np.sign(rng.standard_normal((1, 32))) * 2.5
    qs, _, _ = quantize_sym(s)
    assert np.array_equal(qs, (7 * np.sign(s)).astype(np.int64))


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
