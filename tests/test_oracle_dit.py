"""DiT oracle pieces against library routines and closed forms (CPU only)."""
import numpy as np
import torch
import torch.nn.functional as Fn

from oracle import dit, quant
from tests import oracle_pins as P
from workloads import configs, dit_inputs


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))


def test_f16_rounding_is_nearest():
    """f16() returns the nearest fp16 value (ties to even), checked against both
    fp16 neighbours of the result.  (torch's float64 -> half goes through
    float32 and can double-round, so it is not used as the reference.)"""
    x = np.random.default_rng(0).standard_normal(10000) * 100
    r = dit.f16(x)
    h = r.astype(np.float16)
    up = np.nextafter(h, np.float16(np.inf)).astype(np.float64)
    dn = np.nextafter(h, np.float16(-np.inf)).astype(np.float64)
    e = np.abs(x - r)
    assert np.all(e <= np.abs(x - up)) and np.all(e <= np.abs(x - dn))
    ties = (e == np.abs(x - up)) | (e == np.abs(x - dn))
    assert np.all((h[ties].view(np.uint16) & 1) == 0)


def test_rms_norm_library_and_closed_form():
    x = np.random.default_rng(1).standard_normal((7, 1024)) * 3
    ref = Fn.rms_norm(_t(x), (1024,), eps=dit.EPS).numpy()
    assert np.allclose(dit.rms_norm(x), ref, rtol=1e-13, atol=1e-13)
    c = np.full((1, 64), -2.0)
    assert np.allclose(dit.rms_norm(c), -2.0 / np.sqrt(4.0 + dit.EPS))


def test_layer_norm_library_and_closed_form():
    x = np.random.default_rng(2).standard_normal((7, 1536)) * 3 + 1
    ref = Fn.layer_norm(_t(x), (1536,), eps=dit.EPS).numpy()
    assert np.allclose(dit.layer_norm(x), ref, rtol=1e-12, atol=1e-12)
    assert np.allclose(dit.layer_norm(np.full((1, 8), 5.0)), 0.0)


def test_gelu_tanh_library():
    x = np.linspace(-12, 12, 4001)
    ref = Fn.gelu(_t(x), approximate="tanh").numpy()
    assert np.allclose(dit.gelu_tanh(x), ref, rtol=1e-14, atol=1e-15)
    assert dit.gelu_tanh(np.array([0.0]))[0] == 0.0


def test_attention_library_and_closed_forms():
    rng = np.random.default_rng(3)
    S, T, H, hd = 5, 37, 4, 16
    q = rng.standard_normal((S, H * hd))
    k = rng.standard_normal((T, H * hd))
    v = rng.standard_normal((T, H * hd))
    out = dit.attention(q, k, v, H)
    qt = _t(q).reshape(S, H, hd).transpose(0, 1)
    kt = _t(k).reshape(T, H, hd).transpose(0, 1)
    vt = _t(v).reshape(T, H, hd).transpose(0, 1)
    ref = Fn.scaled_dot_product_attention(qt, kt, vt).transpose(0, 1).reshape(S, H * hd).numpy()
    assert np.allclose(out, ref, rtol=1e-12, atol=1e-12)
    # All keys equal -> uniform weights -> mean of the values.
    k_eq = np.repeat(k[:1], T, axis=0)
    assert np.allclose(dit.attention(q, k_eq, v, H), np.repeat(v.mean(0, keepdims=True), S, 0))
    # One key -> its value.
    assert np.allclose(dit.attention(q, k[:1], v[:1], H), np.repeat(v[:1], S, 0))


def _zero_block_weights(inp):
    for blk in inp["w"]["blocks"]:
        for name in list(blk):
            if name.startswith("w"):
                blk[name] = np.zeros_like(blk[name])


def test_step_skeleton_with_zero_block_weights():
    """With every quantized weight zero the blocks add nothing (zero rows
    quantize to zero codes), so one step reduces to in-projection, final norm,
    out-projection and the Euler update, recomputed here with torch."""
    for cfg in (configs.DIT_PI, configs.DIT_GR00T):
        inp = dit_inputs.make_dit_inputs(cfg, n_blocks=2, batch=2)
        _zero_block_weights(inp)
        w = inp["w"]
        qb = dit.quantize_block_weights(cfg, w["blocks"])
        ckv = dit.cond_kv(cfg, qb, inp["cond"]) if cfg.arch == "gr00t" else None
        prefix = (inp["kp"], inp["vp"]) if cfg.arch == "pi" else None
        x1 = dit.step(cfg, w, qb, inp["mod"], inp["s_table"], inp["x0"], 0, prefix=prefix, ckv=ckv)
        x = _t(inp["x0"]).reshape(-1, cfg.action_dim)
        r = x @ _t(w["w_in"]).T + _t(w["b_in"])
        D = cfg.hidden
        n = Fn.rms_norm(r, (D,), eps=dit.EPS) if cfg.arch == "pi" else Fn.layer_norm(r, (D,), eps=dit.EPS)
        hf = _t((n * _t(w["g_f"])).numpy().astype(np.float16).astype(np.float64))
        v = hf @ _t(w["w_out"]).T + _t(w["b_out"])
        dt = (-1.0 if cfg.arch == "pi" else 1.0) / cfg.steps
        ref = (x + dt * v).numpy().reshape(x1.shape)
        assert np.allclose(x1, ref, rtol=1e-12, atol=1e-12), cfg.name


def test_block_residual_uses_every_linear():
    """A non-zero block changes the residual; zeroing any one quantized weight
    changes the result (no linear is silently skipped)."""
    cfg = configs.DIT_PI
    inp = dit_inputs.make_dit_inputs(cfg, n_blocks=1)
    w = inp["w"]
    prefix = (inp["kp"], inp["vp"])

    def run(blocks):
        ww = dict(w)
        ww["blocks"] = blocks
        qb = dit.quantize_block_weights(cfg, blocks)
        tr = []
        dit.step(cfg, ww, qb, inp["mod"], inp["s_table"], inp["x0"], 0, prefix=prefix, trace=tr)
        return tr[-1]

    base = run(w["blocks"])
    for name in ("wqkv", "wo", "wgu", "wd"):
        blk = dict(w["blocks"][0])
        blk[name] = np.zeros_like(blk[name])
        assert not np.allclose(run([blk]), base), name


def test_gr00t_blocks_use_every_linear():
    """Both GR00T block kinds (cross-attention with the conditioning k|v linear,
    self-attention): zeroing any one quantized weight changes the residual.
    The blocks are quantized once; a zeroed weight is zero codes and a zero
    scale (what the quantizer gives for an all-zero row)."""
    cfg = configs.DIT_GR00T
    inp = dit_inputs.make_dit_inputs(cfg, n_blocks=2, batch=2)
    w = inp["w"]
    qb0 = dit.quantize_block_weights(cfg, w["blocks"])
    assert np.all(quant.quantize_sym(np.zeros((3, 64)))[0] == 0)

    def run(qb):
        ckv = dit.cond_kv(cfg, qb, inp["cond"])
        tr = []
        dit.step(cfg, w, qb, inp["mod"], inp["s_table"], inp["x0"], 0, ckv=ckv, trace=tr)
        return tr

    base = run(qb0)
    for l, names in ((0, ("wq", "wkv", "wo", "wff0", "wff2")), (1, ("wqkv", "wo", "wff0", "wff2"))):
        for name in names:
            qb = [dict(b) for b in qb0]
            qw, ws = qb[l][name]
            qb[l][name] = (np.zeros_like(qw), np.zeros_like(ws))
            assert not np.allclose(run(qb)[l], base[l]), (l, name)


def test_step_scale_changes_only_boundary_codes():
    """eq:perstep_scale reading: s_t multiplies before the per-token quantizer and
    is divided back out, so the block output does not depend on s_t beyond
    float64 rounding at code boundaries."""
    x = np.random.default_rng(4).standard_normal((50, 4096)).astype(np.float16).astype(np.float64)
    q1, xs1, _ = quant.rotate_quantize_act(x, 4096, 1.0)
    q2, xs2, _ = quant.rotate_quantize_act(x, 4096, 3.25)
    assert np.mean(q1 != q2) < 1e-5
    assert np.allclose(xs1, xs2, rtol=1e-14)


def test_block_composition_golden_pi():
    """A tiny Pi-style block worked by hand (every quantization exact)."""
    P.check_dit_block_pi(dit.block_trace, dit.quantize_block_weights)


def test_block_composition_golden_gr00t():
    """Tiny GR00T-style cross- and self-attention blocks worked by hand."""
    P.check_dit_block_gr00t(dit.block_trace, dit.quantize_block_weights, dit.cond_kv)


def test_block_is_block_trace_output():
    cfg = configs.DIT_PI
    inp = dit_inputs.make_dit_inputs(cfg, n_blocks=1)
    w = inp["w"]
    qb = dit.quantize_block_weights(cfg, w["blocks"])
    r = dit.in_projection(w, inp["x0"])
    a = dit.block(cfg, w, qb, inp["mod"], inp["s_table"], r, 0, 2, 1, cfg.tokens, prefix=(inp["kp"], inp["vp"]))
    tr = dit.block_trace(cfg, w, qb, inp["mod"], inp["s_table"], r, 0, 2, 1, cfg.tokens,
                         prefix=(inp["kp"], inp["vp"]))
    assert np.array_equal(a, tr["r_out"])
    # Forcing every value with the oracle's own changes nothing.
    forced = {k: tr[k] for k in ("h1", "qkv", "attn", "h2", "gate_up", "act")}
    forced.update({f"codes{i}": tr[f"codes{i}"][:2] for i in range(4)})
    tf = dit.block_trace(cfg, w, qb, inp["mod"], inp["s_table"], r, 0, 2, 1, cfg.tokens,
                         prefix=(inp["kp"], inp["vp"]), forced=forced)
    assert np.array_equal(tf["r_out"], a)


def test_unquantized_mode_on_the_golden_blocks():
    """Every quantization of the hand-worked blocks is exact, so the oracle's
    unquantized mode (plain float64 products) must give the same numbers."""
    from functools import partial
    P.check_dit_block_pi(partial(dit.block_trace, unquantized=True), dit.quantize_block_weights)
    P.check_dit_block_gr00t(partial(dit.block_trace, unquantized=True), dit.quantize_block_weights, dit.cond_kv)


def test_unquantized_conditioning_kv_is_the_plain_product():
    cfg = configs.DIT_GR00T
    inp = dit_inputs.make_dit_inputs(cfg, n_blocks=2, batch=2)
    ckv = dit.cond_kv_unquantized(cfg, inp["w"], inp["cond"])
    ref = torch.einsum("bpd,nd->bpn", _t(inp["cond"]), _t(inp["w"]["blocks"][0]["wkv"])).numpy()
    assert np.allclose(ckv[0], dit.f16(ref), rtol=0, atol=1e-3)
    assert set(ckv) == {0}
