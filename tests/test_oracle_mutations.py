"""Each pin must reject a plausible mistake planted in a copy of the oracle
(CPU only; the mistakes live in this file, the oracle is untouched)."""
import numpy as np
import pytest

from oracle import composite, hadamard, quant, linear
from oracle import dit as odit
from tests import oracle_pins as P


def fwht_unnormalized(x, b):
    return hadamard.fwht(x, b) * np.sqrt(float(b))


def fwht_sign_swapped(x, b):
    x = np.asarray(x, np.float64)
    K = x.shape[-1]
    y = x.reshape(-1, K // b, b).copy()
    h = 1
    while h < b:
        y = y.reshape(y.shape[0], K // b, b // (2 * h), 2, h)
        u, v = y[:, :, :, 0, :].copy(), y[:, :, :, 1, :].copy()
        y[:, :, :, 0, :] = u - v
        y[:, :, :, 1, :] = u + v
        h *= 2
    return y.reshape(x.shape) / np.sqrt(b)


def fwht_skip_last_stage(x, b):
    if b <= 1:
        return np.asarray(x, np.float64)
    return hadamard.fwht(x, b // 2) * np.sqrt((b // 2) / b)


def quant_qmax8(z):
    return quant.quantize_sym(z, qmax=8)


def quant_floor(z):
    q, d, r = quant.quantize_sym(z)
    return np.clip(np.floor(r), -7, 7).astype(np.int64), d, r


def rq_scale_not_divided(x, b, s_t=1.0):
    q, xs, r = quant.rotate_quantize_act(x, b, s_t)
    return q, xs * s_t, r


def gemm_not_transposed(q, qw):
    return (np.asarray(q) @ np.asarray(qw)).astype(np.int64)


def dequant_no_wscale(acc, xs, ws, bias=None):
    return linear.dequant(acc, xs, np.ones_like(np.asarray(ws, np.float64)), bias)


def sylvester_wrong_sign(n):
    h = hadamard.sylvester(n).copy()
    if n > 1:
        h[-1, -1] *= -1
    return h


def zigzag_ascending(energy, n_blocks):
    return composite.zigzag_permutation(-np.asarray(energy, np.float64), n_blocks)


def zigzag_round_robin(energy, n_blocks):
    e = np.asarray(energy, np.float64)
    K = e.shape[0]
    c = K // n_blocks
    order = sorted(range(K), key=lambda j: (-e[j], j))
    perm = np.empty(K, dtype=np.int64)
    for i, ch in enumerate(order):
        r, p = divmod(i, n_blocks)
        perm[p * c + r] = ch
    return perm


def svd_factor_transposed(w, perm, c):
    u, s = composite.block_svd_factors(w, perm, c)
    return np.transpose(u, (0, 2, 1)), s


def rotations_unnormalized(u):
    return composite.block_rotations(u) * np.sqrt(np.asarray(u).shape[-1])


def rotate_inverse_gather(x, perm, r):
    inv = np.empty_like(perm)
    inv[perm] = np.arange(len(perm))
    return composite.rotate_composite(x, inv, r)


def rotate_transposed_blocks(x, perm, r):
    return composite.rotate_composite(x, perm, np.transpose(np.asarray(r), (0, 2, 1)))


def rqc_scale_not_divided(x, perm, r, s_t=1.0):
    q, xs, ratio = composite.rotate_quantize_composite(x, perm, r, s_t)
    return q, xs * s_t, ratio


@pytest.mark.parametrize("check,impl", [
    (P.check_zigzag, zigzag_ascending),
    (P.check_zigzag, zigzag_round_robin),
    (P.check_block_svd, svd_factor_transposed),
    (P.check_block_rotations, rotations_unnormalized),
])
def test_composite_pin_rejects_mutant(check, impl):
    with pytest.raises((AssertionError, ValueError)):
        check(impl)


def test_rotate_composite_pin_rejects_mutants():
    for impl in (rotate_inverse_gather, rotate_transposed_blocks):
        with pytest.raises(AssertionError):
            P.check_rotate_composite(impl, composite.block_rotations, hadamard.fwht)
    with pytest.raises(AssertionError):
        P.check_rotate_quantize_composite(rqc_scale_not_divided, quant.rotate_quantize_act)


@pytest.mark.parametrize("check,impl", [
    (P.check_sylvester, sylvester_wrong_sign),
    (P.check_fwht_dense, fwht_unnormalized),
    (P.check_fwht_dense, fwht_sign_swapped),
    (P.check_fwht_dense, fwht_skip_last_stage),
    (P.check_fwht_closed_forms, fwht_unnormalized),
    (P.check_quantizer, quant_qmax8),
    (P.check_quantizer, quant_floor),
    (P.check_st_invariance, rq_scale_not_divided),
    (P.check_int_gemm, gemm_not_transposed),
    (P.check_dequant, dequant_no_wscale),
])
def test_pin_rejects_mutant(check, impl):
    with pytest.raises((AssertionError, ValueError)):
        check(impl)


def test_worked_example_rejects_qmax8():
    def rq(x, b, s_t=1.0):
        y = hadamard.fwht(x, b) * s_t
        q, d, r = quant.quantize_sym(y, qmax=8)
        return q, d / s_t, r
    with pytest.raises(AssertionError):
        P.check_worked_example_activation(rq)


# --------------------------------------------------------------------------
# DiT block composition: each mutant is the oracle's block with one planted
# misreading (of the modulation, a gate, the prefix keys, gate against up,
# the conditioning tokens, the LayerNorm affine) or one misplaced operation.
# --------------------------------------------------------------------------

def _with_mod(fn):
    def mutant(cfg, w, qb, mod, s_table, r, l, t, B, S, **kw):
        mm = [[dict(x) for x in row] for row in mod]
        fn(mm[l][t])
        return odit.block_trace(cfg, w, qb, mm, s_table, r, l, t, B, S, **kw)
    return mutant


def _swap(a, b):
    def f(m):
        m[a], m[b] = m[b], m[a]
    return f


def _ones(name):
    def f(m):
        m[name] = np.ones_like(m[name])
    return f


def block_no_prefix(cfg, w, qb, mod, s_table, r, l, t, B, S, prefix=None, **kw):
    kp, vp = prefix
    return odit.block_trace(cfg, w, qb, mod, s_table, r, l, t, B, S, prefix=(kp[:, :, :0], vp[:, :, :0]), **kw)


def block_gate_up_swapped(cfg, w, qb, mod, s_table, r, l, t, B, S, **kw):
    F = cfg.mlp
    qq = [dict(x) for x in qb]
    qw, ws = qq[l]["wgu"]
    order = np.r_[F:2 * F, 0:F]
    qq[l]["wgu"] = (qw[order], ws[order])
    return odit.block_trace(cfg, w, qq, mod, s_table, r, l, t, B, S, **kw)


def block_pi_norm2_on_block_input(cfg, w, qb, mod, s_table, r, l, t, B, S, prefix=None, **kw):
    """The second norm reads the block's input residual instead of the residual
    after the attention branch."""
    out = odit.block_trace(cfg, w, qb, mod, s_table, r, l, t, B, S, prefix=prefix)
    blk, m = w["blocks"][l], mod[l][t]
    h2 = odit.f16(odit.rms_norm(r) * blk["g2"] * (1.0 + m["sc2"]) + m["sh2"])
    return odit.block_trace(cfg, w, qb, mod, s_table, r, l, t, B, S, prefix=prefix,
                            forced={"h2": h2, "attn": out["attn"]})


def block_gr00t_cond_of_sample0(cfg, w, qb, mod, s_table, r, l, t, B, S, ckv=None, **kw):
    c = {k: np.repeat(v[:1], v.shape[0], axis=0) for k, v in ckv.items()}
    return odit.block_trace(cfg, w, qb, mod, s_table, r, l, t, B, S, ckv=c, **kw)


def block_gr00t_cond_k_v_swapped(cfg, w, qb, mod, s_table, r, l, t, B, S, ckv=None, **kw):
    D = cfg.hidden
    c = {k: np.concatenate([v[..., D:], v[..., :D]], axis=-1) for k, v in ckv.items()}
    return odit.block_trace(cfg, w, qb, mod, s_table, r, l, t, B, S, ckv=c, **kw)


def block_gr00t_attention_across_batch(cfg, w, qb, mod, s_table, r, l, t, B, S, **kw):
    if l % 2 == 0:
        return odit.block_trace(cfg, w, qb, mod, s_table, r, l, t, B, S, **kw)
    return odit.block_trace(cfg, w, qb, mod, s_table, r, l, t, 1, B * S, **kw)


def block_gr00t_ln3_affine_swapped(cfg, w, qb, mod, s_table, r, l, t, B, S, **kw):
    ww = {"blocks": [dict(b) for b in w["blocks"]]}
    b = ww["blocks"][l]
    b["g3"], b["beta3"] = b["beta3"], b["g3"]
    return odit.block_trace(cfg, ww, qb, mod, s_table, r, l, t, B, S, **kw)


@pytest.mark.parametrize("impl", [
    _with_mod(_swap("sc1", "sh1")),
    _with_mod(_swap("sc2", "sh2")),
    _with_mod(_ones("gt1")),
    _with_mod(_ones("gt2")),
    _with_mod(_swap("gt1", "gt2")),
    block_no_prefix,
    block_gate_up_swapped,
    block_pi_norm2_on_block_input,
], ids=["sc1_sh1", "sc2_sh2", "no_gt1", "no_gt2", "gates_swapped", "no_prefix", "gate_up_swapped",
        "norm2_on_block_input"])
def test_dit_block_pi_pin_rejects_mutant(impl):
    with pytest.raises(AssertionError):
        P.check_dit_block_pi(impl, odit.quantize_block_weights)


@pytest.mark.parametrize("impl", [
    _with_mod(_swap("sc1", "sh1")),
    block_gr00t_cond_of_sample0,
    block_gr00t_cond_k_v_swapped,
    block_gr00t_attention_across_batch,
    block_gr00t_ln3_affine_swapped,
], ids=["sc1_sh1", "cond_of_sample0", "cond_k_v_swapped", "attention_across_batch", "ln3_affine_swapped"])
def test_dit_block_gr00t_pin_rejects_mutant(impl):
    with pytest.raises(AssertionError):
        P.check_dit_block_gr00t(impl, odit.quantize_block_weights, odit.cond_kv)
