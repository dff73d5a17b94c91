"""Teacher-forced check of one DiT block run by the library against the
oracle's block (test code; shares nothing with the HIP path).

The library runs block l of step t on a residual; its fp16 site values
(norm outputs, linear outputs, attention output, activation), the codes its
fused producers wrote for each of the four quantization sites
(oq_dit_run_block_until) and the block's output residual are read back.
oracle.dit.block_trace is then run on the same residual with every one of
those values forced, so each of its operations is evaluated on the
library's own input of that operation, and its results are compared:
  * glue outputs (norms, attention, linear outputs in fp16, activation):
    relative L2 <= 2e-3;
  * codes of each site: the boundary rule of tests/parity.py against the
    oracle's codes of the library's fp16 site input;
  * the residual update: relative L2 <= 2e-3 (the oracle's linears take the
    library's codes, so identical integer products feed both).
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import dit as odit
from tests import parity

DEV = torch.device("cuda:0")
SITE_INPUT = ("h1", "attn", "h2", "act")


def gpu_weights(model, l):
    """The library's quantized weights of block l (codes and scales) as the
    oracle's qblocks entry."""
    return {nm: (parity.unpack_int4(Wq.cpu().numpy()), ws.cpu().numpy().astype(np.float64))
            for nm, (Wq, ws) in model.qweights[l].items()}


def static_weights(model, l, t):
    """The library's step-folded weights of (block l, step t) by weight name."""
    names = model.SITE_WEIGHTS[model.arch]
    out = {}
    for i in range(4):
        Wq, ws = model.static_weight(l, t, i)
        q = (parity.unpack_int4(Wq.cpu().numpy()), ws.cpu().numpy().astype(np.float64))
        for nm in names[i]:
            out[nm] = q
    return out


def run_gpu_block(model, l, t, r_in):
    """Codes of the four sites (a run stopped after each producer), then the
    whole block: (intermediates, [(q, x_scale)] * 4, r_out float64)."""
    Ks = model.site_dims()[0]
    codes = []
    for site in range(4):
        r = torch.from_numpy(np.ascontiguousarray(r_in, dtype=np.float32)).to(DEV)
        model.run_block_until(l, t, r, site)
        codes.append(model.site_codes(Ks[site]))
    r = torch.from_numpy(np.ascontiguousarray(r_in, dtype=np.float32)).to(DEV)
    model.run_block(l, t, r)
    torch.cuda.synchronize()
    return model.intermediates(), codes, r.cpu().numpy().astype(np.float64)


def check_block(cfg, inp, model, l, t, r_in, static_delta=None):
    """Returns (errors by name, code mismatches, r_out of the library).
    static_delta: the four step rows of (l, t) in the static mode (None:
    per-token quantizer)."""
    D = cfg.hidden
    B, S = inp["batch"], cfg.tokens
    it, codes, r_out = run_gpu_block(model, l, t, r_in)
    r = np.asarray(r_in, dtype=np.float32).astype(np.float64)
    gr = cfg.arch == "gr00t"
    site0 = "q" if gr and l % 2 == 0 else "qkv"
    # gr00t: the ff0 linear applies the GELU in its epilogue, so its fp16
    # output before the activation is not kept; act is checked instead.
    names = ("h1", site0, "attn", "h2", "act") if gr else ("h1", site0, "attn", "h2", "gate_up", "act")
    forced = {nm: it[nm] for nm in names}
    for i in range(4):
        forced[f"codes{i}"] = codes[i]
    qb = {l: gpu_weights(model, l)}
    kw = {}
    if gr:
        P = cfg.prefix
        if l % 2 == 0:
            kw["ckv"] = {l: model.cond_kv_block(l).reshape(B, P, 2 * D)}
    else:
        kw["prefix"] = (inp["kp"], inp["vp"])
    static = None
    if static_delta is not None:
        static = (static_delta, static_weights(model, l, t))
    tr = odit.block_trace(cfg, inp["w"], qb, inp["mod"], inp["s_table"], r, l, t, B, S, forced=forced,
                          static=static, **kw)
    errs = {nm: parity.rel_l2(it[nm], tr[nm]) for nm in names}
    n_mis = 0
    for i in range(4):
        x = it[SITE_INPUT[i]]
        K = x.shape[1]
        b = K & -K
        q_o, xs_o, r_o = tr[f"codes{i}"]
        q_g, xs_g = codes[i]
        if static is None:
            tau = parity.tau_rows(x, b)
            assert np.allclose(xs_g, xs_o, rtol=1e-5, atol=0), (l, t, i)
        else:
            tau = parity.tau_static(x, b, static_delta[i], r_o)
            assert np.array_equal(xs_g, np.ones_like(xs_g)), (l, t, i)
        n, _ = parity.check_codes(q_g, q_o, r_o, tau)
        n_mis += n
    errs["update"] = parity.rel_l2(r_out - r, tr["r_out"] - r)
    return errs, n_mis, r_out


def assert_block(cfg, inp, model, l, t, r_in, tag="", static_delta=None):
    errs, n_mis, r_out = check_block(cfg, inp, model, l, t, r_in, static_delta=static_delta)
    print(f"{tag}block {l} step {t}: code mismatches {n_mis}; " +
          ", ".join(f"{k} {v:.2e}" for k, v in errs.items()), flush=True)
    for k, v in errs.items():
        assert v <= parity.REL_L2_OUT, (l, t, k, v)
    return r_out


def assert_in_projection(inp, model, tag=""):
    """The library's action in-projection (oq_dit_in_projection) against the
    oracle's r = x W_in^T + b_in, a float64 product of the same fp16 weights and
    fp32 actions.  Each library output is an fp32 fma chain over the A action
    channels and then the bias addition, A + 1 roundings, so the standard bound
    for a recursive sum holds: |r - r_exact| <= gamma_{A+1} (sum_a |x_a w_a| +
    |b|) with gamma_n = n u / (1 - n u), u = 2^-24."""
    x = np.ascontiguousarray(inp["x0"], dtype=np.float32)
    M, D = model.M, model.cfg_c.hidden
    r = torch.empty((M, D), dtype=torch.float32, device=DEV)
    model.in_projection(torch.from_numpy(x).to(DEV), r)
    torch.cuda.synchronize()
    got = r.cpu().numpy().astype(np.float64)
    x64 = x.astype(np.float64)
    want = odit.in_projection(inp["w"], x64)
    A = x.shape[-1]
    mag = (np.abs(x64.reshape(M, A)) @ np.abs(np.asarray(inp["w"]["w_in"], np.float64)).T
           + np.abs(np.asarray(inp["w"]["b_in"], np.float64))[None, :])
    n, u = A + 1, 2.0 ** -24
    err = np.abs(got - want)
    bound = n * u / (1 - n * u) * mag
    print(f"{tag}in-projection M={M} D={D} A={A}: max |err| / bound {float(np.max(err / bound)):.3f}", flush=True)
    assert np.all(err <= bound)
