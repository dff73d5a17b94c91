"""The timed DiT path against the per-block path it is built from (GPU).

oq_dit_step / oq_dit_denoise run whole steps as replays of a captured HIP
graph, with the fused producers writing only codes.  The per-site parity
tests check oq_dit_run_block against the oracle.  Here a step rebuilt from
its parts on the same handle -- oq_dit_in_projection, oq_dit_run_block for
every block, oq_dit_final_stage -- must give the same x_{t+1} and the same
residual after the last block, bit for bit; likewise the whole denoising loop.
Both DiT shapes at full size, with the graph and without it
(OQ_DIT_NO_GRAPH=1 at creation), in the per-token mode and in the static
per-step mode (per-(layer, step, channel) table of eq:perstep_scale)."""
import os

import numpy as np
import pytest
import torch

import paper_2605_28803_amd as oq
from workloads import configs, dit_inputs
from workloads import generators as G

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _handle(cfg, inp, graph):
    old = os.environ.get("OQ_DIT_NO_GRAPH")
    os.environ["OQ_DIT_NO_GRAPH"] = "0" if graph else "1"
    try:
        return oq.DiT(cfg, inp, device="cuda:0")
    finally:
        if old is None:
            del os.environ["OQ_DIT_NO_GRAPH"]
        else:
            os.environ["OQ_DIT_NO_GRAPH"] = old


def _chain(model, x0, ts):
    """Steps rebuilt from the parts: (x after the steps, residual after the
    last block of the last step)."""
    L = model.cfg_c.n_blocks
    x = x0.clone()
    r = torch.empty((model.M, model.cfg_c.hidden), dtype=torch.float32, device=DEV)
    for t in ts:
        model.in_projection(x, r)
        for l in range(L):
            model.run_block(l, t, r)
        model.final_stage(r, x)
    torch.cuda.synchronize()
    return x, r.cpu().numpy().astype(np.float64)


def _check(model, inp, steps, tag):
    T = model.cfg_c.steps
    x0 = torch.from_numpy(inp["x0"].astype(np.float32)).to(DEV)
    for t in steps:
        xs = x0.clone()
        model.step(xs, t)
        torch.cuda.synchronize()
        r_step = model.step_residual()
        xc, rc = _chain(model, x0, [t])
        print(f"{tag} step {t}: max |x_step - x_chain| = {(xs - xc).abs().max().item():.3e}", flush=True)
        assert torch.equal(xs, xc), (tag, t)
        assert np.array_equal(r_step, rc), (tag, t)
        # a second replay of the same step gives the same result again
        xs2 = x0.clone()
        model.step(xs2, t)
        torch.cuda.synchronize()
        assert torch.equal(xs2, xs), (tag, t)
    xd = x0.clone()
    model.denoise(xd, T)
    torch.cuda.synchronize()
    xc, rc = _chain(model, x0, range(T))
    assert torch.equal(xd, xc), tag
    assert np.array_equal(model.step_residual(), rc), tag
    print(f"{tag} denoise over {T} steps: bit-equal", flush=True)


@pytest.fixture(scope="module")
def pi_inputs():
    return dit_inputs.make_dit_inputs(configs.DIT_PI)


@pytest.fixture(scope="module")
def gr00t_inputs():
    return dit_inputs.make_dit_inputs(configs.DIT_GR00T)


@pytest.mark.parametrize("graph", [True, False], ids=["graph", "no_graph"])
def test_step_equals_block_chain_pi(pi_inputs, graph):
    cfg = configs.DIT_PI
    print(f"pi full size, graph={graph}", flush=True)
    model = _handle(cfg, pi_inputs, graph)
    _check(model, pi_inputs, (0, cfg.steps - 1), f"pi graph={graph}")
    model.close()


@pytest.mark.parametrize("graph", [True, False], ids=["graph", "no_graph"])
def test_step_equals_block_chain_gr00t(gr00t_inputs, graph):
    cfg = configs.DIT_GR00T
    print(f"gr00t full size (batch 64), graph={graph}", flush=True)
    model = _handle(cfg, gr00t_inputs, graph)
    _check(model, gr00t_inputs, (0, cfg.steps - 1), f"gr00t graph={graph}")
    model.close()


def _static(model, inp, n_traj):
    shape = inp["x0"].shape
    x0s = [torch.from_numpy(G.gaussian(900 + j, "calib/x0", shape).astype(np.float32)).to(DEV) for j in range(n_traj)]
    table = model.calibrate_static_steps(x0s)
    model.set_static_steps(inp, table)
    return table


@pytest.mark.parametrize("graph", [True, False], ids=["graph", "no_graph"])
def test_static_step_equals_block_chain_pi(pi_inputs, graph):
    cfg = configs.DIT_PI
    print(f"pi full size static steps, graph={graph}", flush=True)
    model = _handle(cfg, pi_inputs, graph)
    table = _static(model, pi_inputs, 2)
    _check(model, pi_inputs, (0, cfg.steps - 1), f"pi static graph={graph}")
    del table
    model.close()


def test_static_step_equals_block_chain_gr00t():
    cfg = configs.DIT_GR00T
    inp = dit_inputs.make_dit_inputs(cfg, batch=8)
    print("gr00t 16 blocks batch 8 static steps", flush=True)
    model = _handle(cfg, inp, True)
    table = _static(model, inp, 1)
    _check(model, inp, (0, cfg.steps - 1), "gr00t static")
    del table
    model.close()
