"""DiT action-head denoising step, oracle side (test infrastructure only).

The paper quantizes every linear of the DiT action head of Pi-0.5 and
GR00T-N1.5 to W4A4, with RTN weights and the per-step activation scale
(Experimental Settings, Implementation Details), runs T Euler denoising steps
(same paragraph) and describes the GR00T block as AdaLayerNorm -> attention
q/k/v -> ... -> LayerNorm -> ff.net[0] -> GELU -> ff.net[2] (Appendix,
"Necessity of Per-Step Activation Scaling for DiT").  The paper does not give
the block equations; the readings used here are:

"pi" block (Pi-0.5 action expert):
    h   = fp16(rms(r) * g1 * (1 + sc1_t) + sh1_t)
    qkv = fp16(W4A4(h; Wqkv, s[l,t,0]))                   q | k | v along N
    o   = fp16(attention(q, [Kp ; k], [Vp ; v]))          prefix keys first
    r  += gt1_t * W4A4(o; Wo, s[l,t,1])
    h2  = fp16(rms(r) * g2 * (1 + sc2_t) + sh2_t)
    gu  = fp16(W4A4(h2; Wgu, s[l,t,2]))                   gate | up along N
    a   = fp16(gelu_tanh(gate) * up)
    r  += gt2_t * W4A4(a; Wd, s[l,t,3])
"gr00t" block (GR00T-N1.5 DiT):
    h   = fp16(ln(r) * g1 * (1 + sc1_t) + sh1_t)          AdaLayerNorm
    even blocks: q = fp16(W4A4(h; Wq, s[l,t,0])), k|v = fp16(W4A4(cond; Wkv, 1))
                 computed once per denoising call (cond does not depend on t)
    odd blocks:  q|k|v = fp16(W4A4(h; Wqkv, s[l,t,0])), self-attention
    o   = fp16(attention per sample)
    r  += W4A4(o; Wo, s[l,t,1])
    h3  = fp16(ln(r) * g3 + beta3)                         plain LayerNorm
    f   = fp16(gelu_tanh(W4A4(h3; Wff0, s[l,t,2])))
    r  += W4A4(f; Wff2, s[l,t,3])
Step (both): r = x_t . W_in^T + b_in ; blocks ; v = fp16(norm(r) * g_f) .
W_out^T + b_out ; x_{t+1} = x_t + dt * v, dt = -1/T (pi: tau 1 -> 0) or +1/T
(gr00t: tau 0 -> 1).

rms(r) = r / sqrt(mean(r^2) + 1e-6); ln(r) = (r - mean) / sqrt(var + 1e-6);
attention = softmax(q k^T / sqrt(head_dim)) v per head; gelu_tanh(x) =
x/2 (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3))).  The residual r and the action
state x are float64 (the HIP path keeps them in fp32); every tensor that is an
input or output of a quantized linear is rounded to fp16 where "fp16(...)" is
written.  The Hadamard block of a linear is the largest power of two dividing
its input size (the block-wise form of eq:blockdiag).

Parity: the norms, the attention and the activation are pinned by closed
forms and library routines in the tests.  The composition of a block (where
the modulation scale, shift and gates act, which residual branch each gate
scales, the prefix keys ahead of the own keys, per-sample attention, the
conditioning k|v of the cross-attention blocks, gate against up) is pinned by
two tiny blocks worked by hand (tests/golden/dit_block_pi.txt,
dit_block_gr00t.txt) whose every quantization is exact, so their outputs are
plain numbers; planted mistakes in each of those places fail that pin.
"""
from __future__ import annotations

import numpy as np

from .linear import dequant, int_gemm, w4a4_linear
from .quant import quantize_weights, rotate_quantize_act, rotate_quantize_static

EPS = 1e-6


def f16(x):
    """Round to the nearest fp16 value (ties to even) and return float64."""
    return np.asarray(x, dtype=np.float64).astype(np.float16).astype(np.float64)


def rms_norm(r: np.ndarray) -> np.ndarray:
    r = np.asarray(r, dtype=np.float64)
    return r / np.sqrt(np.mean(r * r, axis=-1, keepdims=True) + EPS)


def layer_norm(r: np.ndarray) -> np.ndarray:
    r = np.asarray(r, dtype=np.float64)
    mu = np.mean(r, axis=-1, keepdims=True)
    var = np.mean((r - mu) ** 2, axis=-1, keepdims=True)
    return (r - mu) / np.sqrt(var + EPS)


def gelu_tanh(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    return 0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * x ** 3)))


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_heads: int) -> np.ndarray:
    """q [S, H*hd], k/v [T, H*hd] -> [S, H*hd]; softmax over the T keys per head."""
    S = q.shape[0]
    hd = q.shape[1] // n_heads
    out = np.empty((S, n_heads * hd))
    for h in range(n_heads):
        sl = slice(h * hd, (h + 1) * hd)
        s = q[:, sl] @ k[:, sl].T / np.sqrt(float(hd))
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, sl] = p @ v[:, sl]
    return out


def hadamard_block(n: int) -> int:
    return n & (-n)


def quantize_block_weights(cfg, blocks):
    """Offline: quantize every W4A4 weight of every block (dict name -> (qw, ws))."""
    D, F = cfg.hidden, cfg.mlp
    out = []
    for blk in blocks:
        qb = {}
        for name, w in blk.items():
            if not name.startswith("w"):
                continue
            K = w.shape[1]
            qw, ws, _ = quantize_weights(w, hadamard_block(K))
            qb[name] = (qw, ws)
        out.append(qb)
    del D, F
    return out


def _lin(x, qweights, name, s):
    qw, ws = qweights[name]
    b = hadamard_block(x.shape[1])
    return w4a4_linear(x, None, b, s, weights=(qw, ws))["y"]


def cond_kv(cfg, qblocks, cond):
    """gr00t: per even block, k|v of the conditioning tokens, [B, P, 2D] fp16 values."""
    out = {}
    B, P, D = cond.shape
    for l in range(len(qblocks)):
        if cfg.arch == "gr00t" and l % 2 == 0:
            kv = f16(_lin(cond.reshape(B * P, D), qblocks[l], "wkv", 1.0))
            out[l] = kv.reshape(B, P, 2 * D)
    return out


def block_trace(cfg, w, qblocks, mod, s_table, r, l, t, B, S, prefix=None, ckv=None, forced=None,
                static=None, unquantized=False):
    """Block l at step t on the residual r [B*S, D] (float64), every
    intermediate returned in a dict.

    Names: "h1" (first norm output), "qkv" (pi and odd gr00t blocks) or "q"
    (even gr00t blocks), "attn", "r1" (residual after the attention branch),
    "h2" (second norm output), "gate_up" (pi: [gate | up]; gr00t: the ff0
    output before the GELU), "act", "r_out"; for each quantization site i
    (0: q|k|v input, 1: o input, 2: gate|up / ff0 input, 3: down / ff2 input)
    "codes{i}" = (q, x_scale, ratio) and "y{i}" = the linear's output before
    fp16 rounding or the residual update.

    forced (teacher forcing): a dict that may hold values another
    implementation produced under the names "h1", "qkv", "q", "attn", "h2",
    "gate_up", "act" and "codes{i}" = (q, x_scale).  A forced value is what
    everything downstream of it uses; under its own name the result keeps
    the oracle's value computed from the (forced) inputs upstream of it.  So
    each operation is evaluated on the other implementation's own input.

    static: None (per-token quantizer with the scalar step s_table[l, t, i])
    or (delta, qweights_t): the per-channel static steps delta[i] of the four
    sites at (l, t) and the weights folded with them, a dict like qblocks[l]
    (eq:perstep_scale with the per-channel table; token scale 1).

    unquantized: every linear is the plain float64 product x W^T with the
    block's weights as given (no rotation, no codes: the model the
    quantization approximates); qblocks is then unused."""
    D, H, F = cfg.hidden, cfg.n_heads, cfg.mlp
    blk, m = w["blocks"][l], mod[l][t]
    st = s_table[l, t]
    fz = forced or {}
    out = {}

    def tf(name, own):
        out[name] = own
        v = fz.get(name)
        return own if v is None else np.asarray(v, dtype=np.float64)

    def site(i, x, name):
        if unquantized:
            y = x @ np.asarray(w["blocks"][l][name], dtype=np.float64).T
            out[f"y{i}"] = y
            return y
        b = hadamard_block(x.shape[1])
        if static is None:
            q, xs, ratio = rotate_quantize_act(x, b, st[i])
            qw, ws = qblocks[l][name]
        else:
            q, xs, ratio = rotate_quantize_static(x, b, static[0][i])
            qw, ws = static[1][name]
        out[f"codes{i}"] = (q, xs, ratio)
        fq = fz.get(f"codes{i}")
        if fq is not None:
            q, xs = fq
        y = dequant(int_gemm(q, qw), xs, ws)
        out[f"y{i}"] = y
        return y

    if cfg.arch == "pi":
        h = tf("h1", f16(rms_norm(r) * blk["g1"] * (1.0 + m["sc1"]) + m["sh1"]))
        qkv = tf("qkv", f16(site(0, h, "wqkv")))
        o = np.empty((B * S, D))
        Kp, Vp = prefix
        for b in range(B):
            rows = slice(b * S, (b + 1) * S)
            kk = np.concatenate([Kp[l, b], qkv[rows, D:2 * D]], axis=0)
            vv = np.concatenate([Vp[l, b], qkv[rows, 2 * D:]], axis=0)
            o[rows] = attention(qkv[rows, :D], kk, vv, H)
        o = tf("attn", f16(o))
        r = r + m["gt1"] * site(1, o, "wo")
        out["r1"] = r
        h2 = tf("h2", f16(rms_norm(r) * blk["g2"] * (1.0 + m["sc2"]) + m["sh2"]))
        gu = tf("gate_up", f16(site(2, h2, "wgu")))
        a = tf("act", f16(gelu_tanh(gu[:, :F]) * gu[:, F:]))
        out["r_out"] = r + m["gt2"] * site(3, a, "wd")
        return out
    if cfg.arch == "gr00t":
        h = tf("h1", f16(layer_norm(r) * blk["g1"] * (1.0 + m["sc1"]) + m["sh1"]))
        o = np.empty((B * S, D))
        if l % 2 == 0:
            q = tf("q", f16(site(0, h, "wq")))
            kv = ckv[l]
            for b in range(B):
                rows = slice(b * S, (b + 1) * S)
                o[rows] = attention(q[rows], kv[b, :, :D], kv[b, :, D:], H)
        else:
            qkv = tf("qkv", f16(site(0, h, "wqkv")))
            for b in range(B):
                rows = slice(b * S, (b + 1) * S)
                o[rows] = attention(qkv[rows, :D], qkv[rows, D:2 * D], qkv[rows, 2 * D:], H)
        o = tf("attn", f16(o))
        r = r + site(1, o, "wo")
        out["r1"] = r
        h3 = tf("h2", f16(layer_norm(r) * blk["g3"] + blk["beta3"]))
        ff = tf("gate_up", f16(site(2, h3, "wff0")))
        f = tf("act", f16(gelu_tanh(ff)))
        out["r_out"] = r + site(3, f, "wff2")
        return out
    raise ValueError(cfg.arch)


def block(cfg, w, qblocks, mod, s_table, r, l, t, B, S, prefix=None, ckv=None, unquantized=False):
    """Block l at step t on the residual r [B*S, D] (float64); returns the new residual."""
    return block_trace(cfg, w, qblocks, mod, s_table, r, l, t, B, S, prefix=prefix, ckv=ckv,
                       unquantized=unquantized)["r_out"]


def cond_kv_unquantized(cfg, w, cond):
    """gr00t: cond_kv with the k|v linear as the plain product (fp16 values)."""
    out = {}
    B, P, D = cond.shape
    for l, blk in enumerate(w["blocks"]):
        if cfg.arch == "gr00t" and l % 2 == 0:
            kv = f16(cond.reshape(B * P, D) @ np.asarray(blk["wkv"], dtype=np.float64).T)
            out[l] = kv.reshape(B, P, 2 * D)
    return out


def in_projection(w, x_t):
    """r = x_t . W_in^T + b_in for x_t [B, S, A] -> [B*S, D]."""
    B, S, A = x_t.shape
    return x_t.reshape(B * S, A) @ np.asarray(w["w_in"], np.float64).T + w["b_in"][None, :]


def step(cfg, w, qblocks, mod, s_table, x_t, t, prefix=None, ckv=None, trace=None, unquantized=False):
    """One Euler denoising step.  x_t [B, S, A] float64 -> x_{t+1}.

    w: dict with w_in [D, A], b_in [D], w_out [A, D], b_out [A], g_f [D] and
    blocks: list of per-block dicts (gains g1/g2 or g1/g3/beta3).
    qblocks: output of quantize_block_weights.  mod[l][t]: dict of the per-step
    modulation vectors.  s_table [L, T, 4].  prefix: pi, (Kp, Vp) each
    [L, B, P, D]; ckv: gr00t, output of cond_kv.  trace: optional list that
    receives the residual after each block.  unquantized: every block
    linear as the plain float64 product (see block_trace).
    """
    B, S, A = x_t.shape
    r = in_projection(w, x_t)
    for l in range(len(w["blocks"])):
        r = block(cfg, w, qblocks, mod, s_table, r, l, t, B, S, prefix=prefix, ckv=ckv, unquantized=unquantized)
        if trace is not None:
            trace.append(r.copy())
    norm = rms_norm if cfg.arch == "pi" else layer_norm
    hf = f16(norm(r) * w["g_f"])
    v = hf @ np.asarray(w["w_out"], np.float64).T + w["b_out"][None, :]
    dt = (-1.0 if cfg.arch == "pi" else 1.0) / cfg.steps
    return x_t + dt * v.reshape(B, S, A)


def denoise(cfg, w, mod, s_table, x0, prefix=None, cond=None, n_steps=None, unquantized=False):
    """Full Euler loop from x0 over n_steps (default cfg.steps); unquantized:
    the same loop with every block linear as the plain float64 product."""
    if unquantized:
        qblocks = None
        ckv = cond_kv_unquantized(cfg, w, cond) if cfg.arch == "gr00t" else None
    else:
        qblocks = quantize_block_weights(cfg, w["blocks"])
        ckv = cond_kv(cfg, qblocks, cond) if cfg.arch == "gr00t" else None
    x = np.asarray(x0, dtype=np.float64)
    for t in range(cfg.steps if n_steps is None else n_steps):
        x = step(cfg, w, qblocks, mod, s_table, x, t, prefix=prefix, ckv=ckv, unquantized=unquantized)
    return x
