"""Seeded DiT inputs: weights (already in the rotated-input basis, i.e. the
SVD factor folded offline), norm gains with outlier channels, per-step
modulation, prefix / conditioning tokens, the per-step scale table and the
initial noise.  Random numbers only; every value is fp16-representable where
the HIP path consumes fp16."""
from __future__ import annotations

import numpy as np

from .generators import gaussian, outlier_channels, log_uniform


def _f16(a):
    return np.asarray(a, np.float64).astype(np.float16).astype(np.float64)


def make_dit_inputs(cfg, n_blocks=None, batch=None):
    L = cfg.n_blocks if n_blocks is None else n_blocks
    B = cfg.batch if batch is None else batch
    D, F, A, S, P, T = cfg.hidden, cfg.mlp, cfg.action_dim, cfg.tokens, cfg.prefix, cfg.steps
    sd = cfg.seed
    n_out = int(round(cfg.outlier_frac * D))

    def gain(name):
        g = 1.0 + gaussian(sd, name, (D,), 0.05)
        g[outlier_channels(sd, name, D, n_out)] *= cfg.outlier_factor
        return _f16(g)

    w = {
        "w_in": _f16(gaussian(sd, "w_in", (D, A), 1.0 / np.sqrt(A))),
        "b_in": _f16(gaussian(sd, "b_in", (D,), 0.02)),
        "w_out": _f16(gaussian(sd, "w_out", (A, D), cfg.w_std)),
        "b_out": _f16(gaussian(sd, "b_out", (A,), 0.02)),
        "g_f": _f16(1.0 + gaussian(sd, "g_f", (D,), 0.05)),
        "blocks": [],
    }
    for l in range(L):
        p = f"blk{l}/"
        blk = {}
        if cfg.arch == "pi":
            blk["g1"] = gain(p + "g1")
            blk["g2"] = gain(p + "g2")
            blk["wqkv"] = _f16(gaussian(sd, p + "wqkv", (3 * D, D), cfg.w_std))
            blk["wo"] = _f16(gaussian(sd, p + "wo", (D, D), cfg.w_std))
            blk["wgu"] = _f16(gaussian(sd, p + "wgu", (2 * F, D), cfg.w_std))
            blk["wd"] = _f16(gaussian(sd, p + "wd", (D, F), cfg.w_std))
        else:
            blk["g1"] = gain(p + "g1")
            blk["g3"] = gain(p + "g3")
            blk["beta3"] = _f16(gaussian(sd, p + "beta3", (D,), 0.02))
            if l % 2 == 0:
                blk["wq"] = _f16(gaussian(sd, p + "wq", (D, D), cfg.w_std))
                blk["wkv"] = _f16(gaussian(sd, p + "wkv", (2 * D, D), cfg.w_std))
            else:
                blk["wqkv"] = _f16(gaussian(sd, p + "wqkv", (3 * D, D), cfg.w_std))
            blk["wo"] = _f16(gaussian(sd, p + "wo", (D, D), cfg.w_std))
            blk["wff0"] = _f16(gaussian(sd, p + "wff0", (F, D), cfg.w_std))
            blk["wff2"] = _f16(gaussian(sd, p + "wff2", (D, F), cfg.w_std))
        w["blocks"].append(blk)

    names = ("sc1", "sh1", "gt1", "sc2", "sh2", "gt2") if cfg.arch == "pi" else ("sc1", "sh1")
    mod = []
    for l in range(L):
        per_t = []
        for t in range(T):
            m = {}
            for nm in names:
                mean = 1.0 if nm.startswith("gt") else 0.0
                m[nm] = _f16(gaussian(sd, f"mod{l}/{t}/{nm}", (D,), 0.1, mean))
            per_t.append(m)
        mod.append(per_t)

    s_table = log_uniform(sd, "s_table", (L, T, 4), cfg.s_lo, cfg.s_hi).astype(np.float32).astype(np.float64)
    x0 = gaussian(sd, "x0", (B, S, A)).astype(np.float32).astype(np.float64)

    out = {"w": w, "mod": mod, "s_table": s_table, "x0": x0, "n_blocks": L, "batch": B}
    if cfg.arch == "pi":
        out["kp"] = _f16(gaussian(sd, "kp", (L, B, P, D)))
        out["vp"] = _f16(gaussian(sd, "vp", (L, B, P, D)))
    else:
        c = gaussian(sd, "cond", (B, P, D))
        c[..., outlier_channels(sd, "cond", D, n_out)] *= cfg.outlier_factor
        out["cond"] = _f16(c)
    return out
