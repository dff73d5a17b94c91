"""Codes written by the DiT driver's fused producers against the oracle (GPU).

Each quantized linear input of a block is produced by a kernel that writes the
fp16 row and quantizes the same values (norm, attention combine, GELU).  The
driver is stopped right after each producer (oq_dit_run_block_until); the
site's codes and token scales are read back from the workspace (tiled layout
for the Pi-0.5 shape, M = 50; row layout for the GR00T shape, M = 1024 at
batch 64, or M = 32 at the batch 2 used here, tiled) and checked against the
oracle's rotate-quantize of the GPU's own fp16 input of that site: codes by
the boundary rule (at most 1e-4 of the elements differ, each by one step,
each within the fp32 error bound of a half integer), token scales to 1e-5."""
import numpy as np
import pytest
import torch

from oracle import dit as odit
from oracle import quant as oquant
from tests import parity
from workloads import configs, dit_inputs
import paper_2605_28803_amd as oq

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
SITE_INPUT = {0: "h1", 1: "attn", 2: "h2", 3: "act"}


def _check_sites(cfg, inp, model, blocks, steps):
    D, F = cfg.hidden, cfg.mlp
    r0 = odit.in_projection(inp["w"], inp["x0"]).astype(np.float32)
    for l in blocks:
        for t in steps:
            for site in range(4):
                r = torch.from_numpy(r0.copy()).to(DEV)
                model.run_block_until(l, t, r, site)
                torch.cuda.synchronize()
                K = F if site == 3 else D
                x = model.intermediates()[SITE_INPUT[site]][:, :K]
                q_g, xs_g = model.site_codes(K)
                s = float(np.float32(inp["s_table"][l, t, site]))
                q_o, xs_o, r_o = oquant.rotate_quantize_act(x, K & -K, s)
                n_mis, _ = parity.check_codes(q_g, q_o, r_o, parity.tau_rows(x, K & -K))
                assert np.allclose(xs_g, xs_o, rtol=1e-5, atol=0), (l, t, site)
                print(f"block {l} step {t} site {site}: {n_mis} boundary code differences", flush=True)


def test_fused_codes_pi():
    cfg = configs.DIT_PI
    inp = dit_inputs.make_dit_inputs(cfg, n_blocks=2)
    model = oq.DiT(cfg, inp, device="cuda:0")
    _check_sites(cfg, inp, model, blocks=(0, 1), steps=(0, 6))
    model.close()


@pytest.mark.parametrize("batch", [2, 64])
def test_fused_codes_gr00t(batch):
    cfg = configs.DIT_GR00T
    inp = dit_inputs.make_dit_inputs(cfg, n_blocks=2, batch=batch)
    model = oq.DiT(cfg, inp, device="cuda:0")
    _check_sites(cfg, inp, model, blocks=(0, 1), steps=(1,))
    model.close()
