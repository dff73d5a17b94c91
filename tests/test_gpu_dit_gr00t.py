"""GR00T-shaped DiT denoising step against the oracle (GPU).

Batched action head: hidden 1536, MLP 6144 (non-gated GELU), 32 heads x 48,
16 action tokens per sample, cross-attention to 300 conditioning tokens on
even blocks and self-attention on odd blocks, AdaLayerNorm / LayerNorm,
Hadamard blocks 512 (K = 1536) and 2048 (K = 6144).  Parity per quantization
site with teacher forcing, as for the Pi-0.5-shaped head: every linear, the
conditioning k|v linear and every glue operation is checked against the oracle
fed the GPU's own fp16 input of that operation; a step whose blocks are the
identity is compared with the oracle step directly."""
import numpy as np
import pytest
import torch

import paper_2605_28803_amd as oq
from oracle import dit as odit
from oracle import linear as olin
from oracle import quant as oquant
from tests import parity
from workloads import configs, dit_inputs

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
CFG = configs.DIT_GR00T


def _setup(n_blocks, batch, zero_blocks=False):
    inp = dit_inputs.make_dit_inputs(CFG, n_blocks=n_blocks, batch=batch)
    if zero_blocks:
        for blk in inp["w"]["blocks"]:
            for name in list(blk):
                if name.startswith("w"):
                    blk[name] = np.zeros_like(blk[name])
    return inp, oq.DiT(CFG, inp, device="cuda:0")


def _site(x_gpu, s, qw, ws, tag):
    """Code check of one linear input (the library's kernel on the GPU's
    fp16 input against the oracle); returns the oracle's output computed from
    the GPU's codes and scales."""
    K = x_gpu.shape[1]
    b = K & -K
    X = torch.from_numpy(x_gpu.astype(np.float16)).to(DEV)
    Xq, xs = oq.rotate_quantize_act(X, b, s_table=np.array([s], np.float32), t=0)
    torch.cuda.synchronize()
    q_g, xs_g = parity.unpack_int4(Xq.cpu().numpy()), xs.cpu().numpy().astype(np.float64)
    q_o, xs_o, r_o = oquant.rotate_quantize_act(x_gpu, b, float(np.float32(s)))
    n_mis, _ = parity.check_codes(q_g, q_o, r_o, parity.tau_rows(x_gpu, b))
    assert np.allclose(xs_g, xs_o, rtol=1e-5), tag
    return olin.dequant(olin.int_gemm(q_g, qw), xs_g, ws), n_mis


def _weights(model, l):
    return {nm: (parity.unpack_int4(Wq.cpu().numpy()), ws.cpu().numpy().astype(np.float64))
            for nm, (Wq, ws) in model.qweights[l].items()}


def _check_block(inp, model, l, t, r_in, check_cond=True):
    D, H = CFG.hidden, CFG.n_heads
    B, S, P = inp["batch"], CFG.tokens, CFG.prefix
    blk, m, st = inp["w"]["blocks"][l], inp["mod"][l][t], inp["s_table"][l, t]
    r_t = torch.from_numpy(r_in.astype(np.float32)).to(DEV)
    model.run_block(l, t, r_t)
    torch.cuda.synchronize()
    r_out = r_t.cpu().numpy().astype(np.float64)
    it = model.intermediates()
    W = _weights(model, l)
    r = r_in.astype(np.float32).astype(np.float64)
    errs, n_mis = {}, 0
    h1 = odit.f16(odit.layer_norm(r) * blk["g1"] * (1.0 + m["sc1"]) + m["sh1"])
    errs["h1"] = parity.rel_l2(it["h1"], h1)
    att = np.empty((B * S, D))
    if l % 2 == 0:
        y, n = _site(it["h1"], st[0], *W["wq"], "q")
        n_mis += n
        errs["q"] = parity.rel_l2(it["q"], odit.f16(y))
        kv = it["cond_kv"][l // 2]
        if check_cond:
            ykv, n = _site(inp["cond"].reshape(B * P, D), 1.0, *W["wkv"], "cond_kv")
            n_mis += n
            errs["cond_kv"] = parity.rel_l2(kv, odit.f16(ykv))
        for b in range(B):
            rows = slice(b * S, (b + 1) * S)
            kb = kv[b * P:(b + 1) * P]
            att[rows] = odit.attention(it["q"][rows], kb[:, :D], kb[:, D:], H)
    else:
        y, n = _site(it["h1"], st[0], *W["wqkv"], "qkv")
        n_mis += n
        errs["qkv"] = parity.rel_l2(it["qkv"], odit.f16(y))
        qkv = it["qkv"]
        for b in range(B):
            rows = slice(b * S, (b + 1) * S)
            att[rows] = odit.attention(qkv[rows, :D], qkv[rows, D:2 * D], qkv[rows, 2 * D:], H)
    errs["attn"] = parity.rel_l2(it["attn"], odit.f16(att))
    y_o, n = _site(it["attn"], st[1], *W["wo"], "o")
    n_mis += n
    r1 = r + y_o
    h2 = odit.f16(odit.layer_norm(r1) * blk["g3"] + blk["beta3"])
    errs["h2"] = parity.rel_l2(it["h2"], h2)
    y_f, n = _site(it["h2"], st[2], *W["wff0"], "ff0")
    n_mis += n
    errs["ff0"] = parity.rel_l2(it["gate_up"], odit.f16(y_f))
    errs["act"] = parity.rel_l2(it["act"], odit.f16(odit.gelu_tanh(it["gate_up"])))
    y_d, n = _site(it["act"], st[3], *W["wff2"], "ff2")
    n_mis += n
    r2 = r1 + y_d
    errs["update"] = parity.rel_l2(r_out - r, r2 - r)
    return errs, n_mis, r_out


def test_blocks_teacher_forced_gr00t():
    inp, model = _setup(n_blocks=2, batch=4)
    r0 = odit.in_projection(inp["w"], inp["x0"])
    for t in (0, 3):
        rr = r0
        for l in range(2):
            errs, n_mis, rr = _check_block(inp, model, l, t, rr, check_cond=(t == 0))
            print(f"gr00t block {l} step {t}: code mismatches {n_mis}; " +
                  ", ".join(f"{k} {v:.2e}" for k, v in errs.items()), flush=True)
            for k, v in errs.items():
                assert v <= parity.REL_L2_OUT, (l, t, k, v)


def test_full_size_sampled_blocks_gr00t():
    """All 16 blocks at batch 64 (M = 1024, 19200 conditioning rows) run on the
    GPU as a teacher-forced chain; a cross-attention block (0), a
    self-attention block (1) and the last block are checked site by site."""
    inp = dit_inputs.make_dit_inputs(CFG)
    model = oq.DiT(CFG, inp, device="cuda:0")
    t = 2
    r = torch.from_numpy(odit.in_projection(inp["w"], inp["x0"]).astype(np.float32)).to(DEV)
    for l in range(CFG.n_blocks):
        if l in (0, 1, CFG.n_blocks - 1):
            errs, n_mis, r_next = _check_block(inp, model, l, t, r.cpu().numpy().astype(np.float64),
                                               check_cond=(l == 0))
            print(f"gr00t full-size block {l}: code mismatches {n_mis}; " +
                  ", ".join(f"{k} {v:.2e}" for k, v in errs.items()), flush=True)
            for k, v in errs.items():
                assert v <= parity.REL_L2_OUT, (l, k, v)
            r = torch.from_numpy(r_next.astype(np.float32)).to(DEV)
        else:
            model.run_block(l, t, r)
    assert torch.isfinite(r).all().item()


def test_step_with_identity_blocks_matches_oracle_gr00t():
    """Zero block weights make every block the identity, so the step is the
    in-projection, the final LayerNorm, the out-projection and the Euler
    update (dt = +1/T), compared with the oracle step directly."""
    inp, model = _setup(n_blocks=2, batch=4, zero_blocks=True)
    x0 = inp["x0"].astype(np.float32)
    qb = odit.quantize_block_weights(CFG, inp["w"]["blocks"])
    ckv = odit.cond_kv(CFG, qb, inp["cond"])
    for t in (0, 3):
        x = torch.from_numpy(x0).to(DEV)
        model.step(x, t)
        torch.cuda.synchronize()
        ref = odit.step(CFG, inp["w"], qb, inp["mod"], inp["s_table"], x0.astype(np.float64), t, ckv=ckv)
        e = parity.rel_l2(x.cpu().numpy() - x0, ref - x0)
        print(f"gr00t identity-block step {t}: rel_l2 {e:.2e}")
        assert e <= parity.REL_L2_OUT


def test_final_stage_and_end_to_end_gr00t():
    inp, model = _setup(n_blocks=2, batch=4)
    x0 = inp["x0"].astype(np.float32)
    t = 1
    x = torch.from_numpy(x0).to(DEV)
    model.step(x, t)
    torch.cuda.synchronize()
    x1 = x.cpu().numpy().astype(np.float64)
    r = model.intermediates()["resid"]
    w = inp["w"]
    hf = odit.f16(odit.layer_norm(r) * w["g_f"])
    v = hf @ w["w_out"].T + w["b_out"][None, :]
    ref_final = x0.astype(np.float64) + (1.0 / CFG.steps) * v.reshape(x0.shape)
    e = parity.rel_l2(x1 - x0, ref_final - x0)
    print(f"gr00t final stage rel_l2 {e:.2e}")
    assert e <= parity.REL_L2_OUT
    qb = odit.quantize_block_weights(CFG, inp["w"]["blocks"])
    ckv = odit.cond_kv(CFG, qb, inp["cond"])
    ref = odit.step(CFG, inp["w"], qb, inp["mod"], inp["s_table"], x0.astype(np.float64), t, ckv=ckv)
    print(f"gr00t end-to-end step rel_l2 vs independent oracle {parity.rel_l2(x1 - x0, ref - x0):.2e}")
    assert np.all(np.isfinite(x1))


def test_denoise_equals_repeated_steps_gr00t():
    inp, model = _setup(n_blocks=2, batch=2)
    x0 = torch.from_numpy(inp["x0"].astype(np.float32)).to(DEV)
    a = x0.clone()
    model.denoise(a, CFG.steps)
    b = x0.clone()
    for t in range(CFG.steps):
        model.step(b, t)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
