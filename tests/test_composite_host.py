"""Host-side preparation of the full composite rotation against the oracle
(CPU only): zigzag permutation, fp16 block matrices, folded weight codes, and
argument validation of the online call."""
import ctypes as C

import numpy as np

import paper_2605_28803_amd as oq
from paper_2605_28803_amd import _lib
from oracle import composite
from tests import oracle_pins as P
from tests import parity

SHAPE, NULL, ALIGN, ARG, OK = -2, -1, -3, -7, 0
P16 = C.c_void_p(0x10000)
P4 = C.c_void_p(0x10004)


def test_zigzag_matches_oracle():
    g = P.load_golden_rows("zigzag_example.txt")
    assert np.array_equal(oq.zigzag_permutation_host(g["energy"], 4), g["perm"].astype(np.int32))
    rng = np.random.default_rng(40)
    for K, c in ((256, 64), (1536, 64), (4096, 64), (96, 32)):
        e = rng.exponential(size=K)
        e[rng.choice(K, 7, replace=False)] = e[3]
        assert np.array_equal(oq.zigzag_permutation_host(e, c), composite.zigzag_permutation(e, K // c))


def _orthogonal(rng, c, nb):
    return np.stack([P.random_orthogonal(rng, c) for _ in range(nb)])


def test_block_rotations_match_oracle_rounded():
    rng = np.random.default_rng(41)
    u = _orthogonal(rng, 64, 6)
    rt = oq.block_rotations_host(u)  # uint16, column-major blocks
    ref = composite.block_rotations(u).astype(np.float16)
    got = np.transpose(rt, (0, 2, 1)).view(np.float16)
    diff = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    ulp = np.spacing(np.abs(ref)).astype(np.float64)
    # fp64 sums in a different order may round to the neighbouring fp16 value
    # only when the exact value sits on a rounding boundary
    assert np.all(diff <= ulp)
    assert np.count_nonzero(diff) <= 2


def test_weight_fold_matches_oracle():
    rng = np.random.default_rng(42)
    N, K, c = 96, 1024, 64
    w = rng.standard_normal((N, K)) * 0.02
    w[:, rng.choice(K, 6, replace=False)] *= 40
    perm = composite.zigzag_permutation(composite.channel_energy(w), K // c)
    u, _ = composite.block_svd_factors(w, perm, c)
    r16 = composite.block_rotations(u).astype(np.float16)
    rt = np.ascontiguousarray(np.transpose(r16, (0, 2, 1))).view(np.uint16)
    wq, ws = oq.quantize_weights_composite_host(w, perm.astype(np.int32), rt)
    qo, wso, ro = composite.fold_weights_composite(w, perm, r16.astype(np.float64))
    qg = parity.unpack_int4(wq)
    mism = qg != qo
    # both sides are float64; a code can differ only on an exact rounding tie
    assert np.count_nonzero(mism) <= 2
    assert np.all(np.abs(parity.dist_to_boundary(ro[mism])) < 1e-9)
    assert np.allclose(ws, wso.astype(np.float32), rtol=1e-7)


def test_composite_call_rejects_bad_arguments():
    lib = _lib.load()
    f = lib.oq_rotate_quantize_act_composite
    assert f(P16, 4, 96, 96, P16, P16, None, 0, P16, P16, None) == SHAPE    # K % 64
    assert f(P16, 4, 32768, 32768, P16, P16, None, 0, P16, P16, None) == SHAPE
    assert f(P16, 4, 128, 64, P16, P16, None, 0, P16, P16, None) == SHAPE   # ldx < K
    assert f(P16, 4, 128, 132, P16, P16, None, 0, P16, P16, None) == ALIGN  # ldx % 8
    # perm NULL is valid (the input already in the permuted order): it passes
    # the argument checks and stops only at the device check on a host
    # without a GPU
    assert f(P16, 4, 128, 128, None, P16, None, 0, P16, P16, None) not in (NULL, SHAPE, ALIGN, ARG, OK)
    assert f(P16, 4, 128, 128, P16, None, None, 0, P16, P16, None) == NULL  # Rt
    assert f(P16, 4, 128, 128, P4, P16, None, 0, P16, P16, None) == ALIGN
    assert f(P16, 4, 128, 128, P16, P16, None, -1, P16, P16, None) == ARG
    assert f(None, 0, 128, 128, None, None, None, 0, None, None, None) == OK
    z = lib.oq_zigzag_permutation_host
    assert z(None, 8, 4, P16) == NULL
    assert z(P16, 10, 4, P16) == SHAPE
    r = lib.oq_block_rotations_host
    assert r(P16, 96, 48, P16) == SHAPE
    wq = lib.oq_quantize_weights_composite_host
    bad = np.array([0, 1, 2, 9], dtype=np.int32)
    wd = np.zeros((1, 4)); rt = np.zeros((1, 4, 4), dtype=np.uint16)
    out = np.zeros(2, dtype=np.uint8); ws = np.zeros(1, dtype=np.float32)
    assert wq(wd.ctypes.data, 1, 4, 4, bad.ctypes.data, rt.ctypes.data, out.ctypes.data, ws.ctypes.data) == ARG


def test_prepare_calls_reject_bad_arguments():
    lib = _lib.load()
    e = lib.oq_channel_energy
    assert e(None, 4, 64, 64, P16, None) == NULL
    assert e(P16, 0, 64, 64, P16, None) == SHAPE
    assert e(P16, 4, 64, 32, P16, None) == SHAPE
    assert e(P16, 4, 64, 64, P4, None) == ALIGN                  # fp64 output 8-byte aligned
    z = lib.oq_zigzag_permutation
    assert z(P16, 96, 64, P16, None) == SHAPE                    # K % block
    assert z(P16, 1 << 17, 64, P16, None) == SHAPE               # K limit
    assert z(None, 128, 64, P16, None) == NULL
    s = lib.oq_block_svd
    assert s(P16, 8, 128, 128, P16, 32, P16, P16, None) == SHAPE  # block must be 64
    assert s(P16, 8, 96, 96, P16, 64, P16, P16, None) == SHAPE
    assert s(P16, 8, 128, 128, None, 64, P16, P16, None) == NULL
    assert s(P16, 8, 128, 128, P16, 64, P4, P16, None) == ALIGN
    r = lib.oq_block_rotations
    assert r(P16, 100, 64, P16, None) == SHAPE
    assert r(None, 128, 64, P16, None) == NULL
    ws = lib.oq_prepare_weights_workspace_bytes(1024)
    assert ws == 1024 * 66 * 8 and lib.oq_prepare_weights_workspace_bytes(0) == 0
    f = lib.oq_prepare_weights_composite
    assert f(P16, 8, 1024, 1024, P16, P16, P16, P16, P16, ws - 1, None) == SHAPE
    assert f(P16, 8, 1024, 1028, P16, P16, P16, P16, P16, ws, None) == ALIGN  # ldw % 8
    assert f(P16, 8, 1024, 1024, P16, P16, None, P16, P16, ws, None) == NULL
    assert f(P16, 8, 1000, 1000, P16, P16, P16, P16, P16, ws, None) == SHAPE  # K % 64
