"""The DiT driver at shapes beyond the two configured workloads (GPU).

The Pi-0.5 architecture (Section 5's setting, every block linear W4A4) with
  * six samples (300 action rows): token codes in the row layout, the
    generic norm, merge and GELU producers (more than 256 rows), the tiled
    GEMM kernels, four rows per final-stage workgroup;
  * a wider model (hidden 2048, 16 heads of 128, 48 action channels, 20
    tokens, 100 prefix keys): the generic producers on 2048-channel rows, the
    merge of two key splits, the final stage's streamed weights (more than
    32 action channels), the in-projection on its own;
  * one block with 24 and with 12 action channels: the in-projection's
    preloaded 24-channel rows kernel (oq_dit_in_projection) beside the step's
    fused in-projection, and the per-channel sums of both when the action
    width is not a multiple of 8.
For each: teacher-forced block parity against the oracle at the bounds of
the configured shapes, the final stage against its definition, and the timed
step (graph replay) bit-equal to the step rebuilt from its parts."""
import dataclasses

import numpy as np
import pytest
import torch

import paper_2605_28803_amd as oq
from oracle import dit as odit
from tests import dit_parity, parity
from workloads import configs, dit_inputs

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")

SHAPES = {
    "pi_batch6": dataclasses.replace(configs.DIT_PI, name="pi_batch6", n_blocks=2, batch=6, steps=3),
    "pi_wide": dataclasses.replace(configs.DIT_PI, name="pi_wide", n_blocks=2, hidden=2048, n_heads=16,
                                   head_dim=128, tokens=20, prefix=100, steps=3, action_dim=48),
    "pi_a24": dataclasses.replace(configs.DIT_PI, name="pi_a24", n_blocks=1, prefix=64, steps=3, action_dim=24),
    "pi_a12": dataclasses.replace(configs.DIT_PI, name="pi_a12", n_blocks=1, prefix=64, steps=3, action_dim=12),
}


@pytest.fixture(scope="module", params=sorted(SHAPES))
def shape(request):
    cfg = SHAPES[request.param]
    inp = dit_inputs.make_dit_inputs(cfg, n_blocks=cfg.n_blocks)
    model = oq.DiT(cfg, inp, device="cuda:0")
    yield request.param, cfg, inp, model
    model.close()


def test_blocks_teacher_forced(shape):
    name, cfg, inp, model = shape
    r0 = odit.in_projection(inp["w"], inp["x0"])
    for t in (0, 2):
        rr = r0
        for l in range(inp["n_blocks"]):
            rr = dit_parity.assert_block(cfg, inp, model, l, t, rr)
    print(f"{name}: blocks within the per-site bounds", flush=True)


def test_in_projection(shape):
    name, cfg, inp, model = shape
    dit_parity.assert_in_projection(inp, model, f"{name} ")


def test_final_stage(shape):
    name, cfg, inp, model = shape
    x0 = inp["x0"].astype(np.float32)
    x = torch.from_numpy(x0).to(DEV)
    model.step(x, 1)
    torch.cuda.synchronize()
    x1 = x.cpu().numpy().astype(np.float64)
    r = model.intermediates()["resid"]
    w = inp["w"]
    hf = odit.f16(odit.rms_norm(r) * w["g_f"])
    v = hf @ w["w_out"].T + w["b_out"][None, :]
    ref = x0.astype(np.float64) + (-1.0 / cfg.steps) * v.reshape(x0.shape)
    e = parity.rel_l2(x1 - x0, ref - x0)
    print(f"{name}: final stage rel_l2 {e:.2e}", flush=True)
    assert e <= parity.REL_L2_OUT


def test_step_equals_block_chain(shape):
    name, cfg, inp, model = shape
    x0 = torch.from_numpy(inp["x0"].astype(np.float32)).to(DEV)
    t = 1
    xs = x0.clone()
    model.step(xs, t)
    torch.cuda.synchronize()
    r_step = model.step_residual()
    xc = x0.clone()
    r = torch.empty((model.M, model.cfg_c.hidden), dtype=torch.float32, device=DEV)
    model.in_projection(xc, r)
    for l in range(model.cfg_c.n_blocks):
        model.run_block(l, t, r)
    model.final_stage(r, xc)
    torch.cuda.synchronize()
    assert torch.equal(xs, xc), name
    assert np.array_equal(r_step, r.cpu().numpy().astype(np.float64)), name
