"""The DiT driver with static per-step, per-channel steps (eq:perstep_scale
with the per-(layer, step, channel) table) against the oracle (GPU).

  * calibration rollouts: the table equals, bit for bit, the oracle's
    nearest-rank 99.9th percentile over q_max of the rotated site inputs the
    rollouts collected;
  * each site's producer in the static mode: codes by the boundary rule of
    the static quantizer (tau_static, clipping live) against the oracle's
    static quantization of the GPU's own fp16 site input, token scales 1;
  * each block linear in the static mode, teacher-forced: its output against
    the oracle's integer product of the GPU's codes with the step's folded
    weight (2e-3 relative L2), and the block's residual update;
  * clearing the static mode returns the per-token driver bit for bit.
"""
import numpy as np
import pytest
import torch

import paper_2605_28803_amd as oq
from oracle import dit as odit
from oracle import quant as oquant
from tests import dit_parity, parity
from workloads import configs, dit_inputs
from workloads import generators as G

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
SITE_INPUT = {0: "h1", 1: "attn", 2: "h2", 3: "act"}


def _x0s(cfg, inp, n):
    shape = inp["x0"].shape
    return [torch.from_numpy(G.gaussian(900 + j, "calib/x0", shape).astype(np.float32)).to(DEV) for j in range(n)]


def _model(cfg, n_blocks, batch=None, n_traj=2):
    inp = dit_inputs.make_dit_inputs(cfg, n_blocks=n_blocks, batch=batch)
    model = oq.DiT(cfg, inp, device="cuda:0")
    table, samples = model.calibrate_static_steps(_x0s(cfg, inp, n_traj), samples=True)
    return inp, model, table, samples


def _row(model, table, l, t, site):
    Ks, offs, _ = model.site_dims()
    return table[l, t, offs[site]:offs[site] + Ks[site]].cpu().numpy()


def test_calibration_table_is_the_percentile_pi():
    cfg = configs.DIT_PI
    inp, model, table, samples = _model(cfg, n_blocks=2, n_traj=3)
    assert table.shape == (2, cfg.steps, 3 * cfg.hidden + cfg.mlp)
    for (l, t, i), y in samples.items():
        ref = (oquant.percentile_abs(y.cpu().numpy().astype(np.float64), 99.9) / 7.0).astype(np.float32)
        assert np.array_equal(_row(model, table, l, t, i), ref), (l, t, i)
    # the steps differ across denoising steps (the time-conditioned inputs drift)
    d0, d9 = _row(model, table, 0, 0, 0), _row(model, table, 0, cfg.steps - 1, 0)
    assert not np.array_equal(d0, d9)
    model.close()


def _check_static_sites(cfg, inp, model, table, blocks, steps):
    D, F = cfg.hidden, cfg.mlp
    r0 = odit.in_projection(inp["w"], inp["x0"]).astype(np.float32)
    total = 0
    for l in blocks:
        for t in steps:
            for site in range(4):
                r = torch.from_numpy(r0.copy()).to(DEV)
                model.run_block_until(l, t, r, site)
                torch.cuda.synchronize()
                K = F if site == 3 else D
                x = model.intermediates()[SITE_INPUT[site]][:, :K]
                q_g, xs_g = model.site_codes(K)
                d = _row(model, table, l, t, site).astype(np.float64)
                q_o, _, r_o = oquant.rotate_quantize_static(x, K & -K, d)
                n_mis, _ = parity.check_codes(q_g, q_o, r_o, parity.tau_static(x, K & -K, d, r_o))
                assert np.array_equal(xs_g, np.ones_like(xs_g)), (l, t, site)
                clipped = int(np.count_nonzero(np.abs(r_o) > 7.5))
                total += clipped
                print(f"block {l} step {t} site {site}: {n_mis} boundary differences, {clipped} clipped", flush=True)
    return total


def test_static_sites_pi():
    cfg = configs.DIT_PI
    inp, model, table, _ = _model(cfg, n_blocks=2)
    model.set_static_steps(inp, table)
    clipped = _check_static_sites(cfg, inp, model, table, blocks=(0, 1), steps=(0, 6))
    assert clipped > 0, "the 99.9th percentile steps should clip some elements"
    model.close()


def test_static_sites_gr00t():
    cfg = configs.DIT_GR00T
    inp, model, table, _ = _model(cfg, n_blocks=2, batch=2)
    model.set_static_steps(inp, table)
    _check_static_sites(cfg, inp, model, table, blocks=(0, 1), steps=(1,))
    model.close()


def _deltas(model, table, l, t):
    return [_row(model, table, l, t, i).astype(np.float64) for i in range(4)]


def test_static_blocks_teacher_forced_pi():
    """Every site of two blocks in the static mode against the oracle's block
    with the same step rows and the library's step-folded weights, every GPU
    site value forced (tests/dit_parity.py)."""
    cfg = configs.DIT_PI
    inp, model, table, _ = _model(cfg, n_blocks=2)
    model.set_static_steps(inp, table)
    r0 = odit.in_projection(inp["w"], inp["x0"])
    for t in (0, 5):
        rr = r0
        for l in range(2):
            rr = dit_parity.assert_block(cfg, inp, model, l, t, rr, tag="static ",
                                         static_delta=_deltas(model, table, l, t))
    model.close()


def test_static_blocks_teacher_forced_gr00t():
    cfg = configs.DIT_GR00T
    inp, model, table, _ = _model(cfg, n_blocks=2, batch=2)
    model.set_static_steps(inp, table)
    r0 = odit.in_projection(inp["w"], inp["x0"])
    rr = r0
    for l in range(2):
        rr = dit_parity.assert_block(cfg, inp, model, l, 1, rr, tag="gr00t static ",
                                     static_delta=_deltas(model, table, l, 1))
    model.close()


def test_clearing_static_mode_restores_the_driver():
    cfg = configs.DIT_PI
    inp, model, table, _ = _model(cfg, n_blocks=2, n_traj=1)
    x0 = torch.from_numpy(inp["x0"].astype(np.float32)).to(DEV)
    a = model.step(x0.clone(), 3)
    model.set_static_steps(inp, table)
    b = model.step(x0.clone(), 3)
    model.clear_static_steps()
    c = model.step(x0.clone(), 3)
    torch.cuda.synchronize()
    assert torch.equal(a, c)
    assert not torch.equal(a, b)
    assert torch.isfinite(b).all()
    model.close()


@pytest.mark.parametrize("arch", ["pi", "gr00t"])
def test_deviation_from_unquantized_rollout(arch):
    """Reported, not gated (both are quantized models): how far the full
    denoising loop of the per-token driver and of the static-step driver
    (calibrated on 24 trajectories, enough rows that the 99.9th percentile is
    not the maximum) lands from the unquantized float64 rollout of the same
    synthetic DiT (the oracle with every linear a plain product), as the
    relative L2 of x_T - x_0; the oracle's own per-token model is shown
    beside them.  Pi: 3 blocks; GR00T: 2 blocks at batch 4."""
    cfg = configs.DIT_PI if arch == "pi" else configs.DIT_GR00T
    inp = dit_inputs.make_dit_inputs(cfg, n_blocks=3 if arch == "pi" else 2, batch=None if arch == "pi" else 4)
    model = oq.DiT(cfg, inp, device="cuda:0")
    T = cfg.steps
    x0 = torch.from_numpy(inp["x0"].astype(np.float32)).to(DEV)
    xt = x0.clone()
    model.denoise(xt, T)
    table = model.calibrate_static_steps(_x0s(cfg, inp, 24))
    model.set_static_steps(inp, table)
    xs = x0.clone()
    model.denoise(xs, T)
    torch.cuda.synchronize()
    x0n = inp["x0"].astype(np.float32).astype(np.float64)
    kw = {"prefix": (inp["kp"], inp["vp"])} if arch == "pi" else {"cond": inp["cond"]}
    ref = odit.denoise(cfg, inp["w"], inp["mod"], inp["s_table"], x0n, unquantized=True, **kw)
    q_oracle = odit.denoise(cfg, inp["w"], inp["mod"], inp["s_table"], x0n, **kw)
    dev = lambda x: parity.rel_l2(np.asarray(x, np.float64) - x0n, ref - x0n)
    d_tok, d_static, d_oracle = dev(xt.cpu().numpy()), dev(xs.cpu().numpy()), dev(q_oracle)
    d_between = parity.rel_l2(xs.cpu().numpy() - x0n, xt.cpu().numpy() - x0n)
    print(f"{arch} {T}-step denoise, rel L2 of x_T - x_0 against the unquantized fp64 rollout: "
          f"per-token driver {d_tok:.4f}, static-step driver {d_static:.4f}, oracle per-token model {d_oracle:.4f}; "
          f"static against per-token {d_between:.4f}", flush=True)
    assert np.isfinite([d_tok, d_static, d_oracle]).all()
    model.close()
