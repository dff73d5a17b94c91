"""GR00T-shaped DiT denoising step against the oracle (GPU).

Batched action head: hidden 1536, MLP 6144 (non-gated GELU), 32 heads x 48,
16 action tokens per sample, cross-attention to 300 conditioning tokens on
even blocks and self-attention on odd blocks, AdaLayerNorm / LayerNorm,
Hadamard blocks 512 (K = 1536) and 2048 (K = 6144).  Parity per quantization
site with teacher forcing, as for the Pi-0.5-shaped head (the oracle's
block_trace with every GPU site value forced, tests/dit_parity.py): every
linear, the conditioning k|v linear and every glue operation is checked
against the oracle fed the GPU's own fp16 input of that operation; a step whose blocks are the
identity is compared with the oracle step directly."""
import numpy as np
import pytest
import torch

import paper_2605_28803_amd as oq
from oracle import dit as odit
from oracle import linear as olin
from oracle import quant as oquant
from tests import dit_parity, parity
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


def _check_cond(inp, model):
    """The conditioning k|v of each cross-attention block: the library's
    codes of the conditioning rows (the same rotate-quantize kernel its
    set_condition runs) against the oracle's, and its fp16 k|v against the
    oracle's product of those codes with the block's k|v weight."""
    D, B, P = CFG.hidden, inp["batch"], CFG.prefix
    x = inp["cond"].reshape(B * P, D)
    b = D & -D
    Xq, xs = oq.rotate_quantize_act(torch.from_numpy(x.astype(np.float16)).to(DEV), b)
    torch.cuda.synchronize()
    q_g, xs_g = parity.unpack_int4(Xq.cpu().numpy()), xs.cpu().numpy().astype(np.float64)
    q_o, xs_o, r_o = oquant.rotate_quantize_act(x, b, 1.0)
    parity.check_codes(q_g, q_o, r_o, parity.tau_rows(x, b))
    assert np.allclose(xs_g, xs_o, rtol=1e-5)
    for l in range(0, inp["n_blocks"], 2):
        qw, ws = dit_parity.gpu_weights(model, l)["wkv"]
        ref = odit.f16(olin.dequant(olin.int_gemm(q_g, qw), xs_g, ws))
        e = parity.rel_l2(model.cond_kv_block(l), ref)
        print(f"gr00t conditioning k|v of block {l}: rel_l2 {e:.2e}", flush=True)
        assert e <= parity.REL_L2_OUT


def test_blocks_teacher_forced_gr00t():
    inp, model = _setup(n_blocks=2, batch=4)
    _check_cond(inp, model)
    dit_parity.assert_in_projection(inp, model, "gr00t ")
    r0 = odit.in_projection(inp["w"], inp["x0"])
    for t in (0, 3):
        rr = r0
        for l in range(2):
            rr = dit_parity.assert_block(CFG, inp, model, l, t, rr, tag="gr00t ")


def test_full_size_sampled_blocks_gr00t():
    """All 16 blocks at batch 64 (M = 1024, 19200 conditioning rows) run on the
    GPU as a teacher-forced chain; a cross-attention block (0), a
    self-attention block (1) and the last block are checked site by site."""
    inp = dit_inputs.make_dit_inputs(CFG)
    model = oq.DiT(CFG, inp, device="cuda:0")
    dit_parity.assert_in_projection(inp, model, "gr00t full size ")
    t = 2
    r = torch.from_numpy(odit.in_projection(inp["w"], inp["x0"]).astype(np.float32)).to(DEV)
    for l in range(CFG.n_blocks):
        if l in (0, 1, CFG.n_blocks - 1):
            r_next = dit_parity.assert_block(CFG, inp, model, l, t, r.cpu().numpy().astype(np.float64),
                                             tag="gr00t full-size ")
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
