#!/usr/bin/env python3
"""Benchmark: DiT denoising-step latency of the W4A4 Pi-0.5 action expert on one MI355X.

Workload: 18 blocks, hidden 1024, MLP 4096 (gate|up, down), 8 heads x 128,
50 action tokens attending to 816 prefix tokens, batch 1, 10 denoising steps,
per-step scales s[l][t] log-uniform in [0.5, 4], every block linear W4A4 with
Hadamard blocks 1024 / 4096, seeded Gaussian weights (synthetic).  One bench
step = one denoising step (all of: rotate-quantize, W4A4 GEMM + epilogue,
norms, attention, Euler) with t cycling over the 10 steps.  Inputs are resident
in HBM before timing.

Also reported (same JSON line):
  kernels    the W4A4 linears of one step timed alone through the C ABI with
             HIP events on the launch stream: rotate-quantize GB/s and GEMM
             GB/s / TOPS against their rooflines;
  roofline   the dominant kernel of the step, the W4A4 GEMM, at the block's
             largest linear (gate|up, M=50, N=8192, K=1024), against HBM peak
             (traffic from the committed FETCH/WRITE counter summary);
  prefill    the GEMM at M=K=N=16384 against the int8 MFMA peak and the
             rotate-quantize at M=K=16384 against HBM peak, cold;
  cpu_baseline  the oracle on this host on a bounded sample (3 of 18 blocks of
             one step), scaled to denoising steps per second;
  single_linear_64x1024x1024  the single rotated linear, warm and cold;
  sweep      rotate-quantize and GEMM at M in {1, 16, 256, 4096, 16384} x
             K = N in {1024 .. 16384}, cold, each against its roofline (HBM
             for rotate-quantize; min(int8 peak, intensity x HBM) for the GEMM);
  static_footprint  int4 + scales against fp16 for the synthetic workloads'
             linears, beside the paper's own figures (paper_context);
  cpu_oracle_kernels  the oracle's rotate-quantize and GEMM on row samples of
             the 16384^3 prefill shape, single-threaded and on every core.

--sweep writes the rotate-quantize / GEMM roofline sweep (M x K = N grid) as
JSON lines to stdout (and to the file --sweep-out names) instead; --roofline-only runs just the
roofline kernel measurement (the command the committed rocprofv3 summaries of
that kernel were taken with); --copy-calibration runs a plain copy of known
size (the counter calibration reference); --gr00t-only times just the
GR00T-shaped step; --composite-only times just the full composite rotation;
--static-only times the static per-channel step path and its calibration;
--w4a8-only times the W4A8 mode beside W4A4; --prepare-only times the GPU
weight preparation for the composite rotation.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "W4A4 linear TOPS & %MFMA peak; rotate-quant GB/s; DiT denoise-step latency"
HBM_PEAK_GBS = 8000.0
INT8_PEAK_TOPS = 5000.0  # dense int8 MFMA, TOP/s


def _graph_time(fn, reps=20, replays=10):
    """Average GPU time (ms) of one fn() launch: `reps` launches are captured
    into one HIP graph (no host launch overhead in the timed region) and the
    graph is replayed `replays` times between HIP events on the stream the
    kernels run on."""
    import torch
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()  # warm
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        for _ in range(reps):
            fn()
    stream = torch.cuda.current_stream()
    g.replay()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(replays):
        g.replay()
    end.record(stream)
    end.synchronize()
    return start.elapsed_time(end) / (reps * replays)


def dit_linears(cfg):
    """(name, K, N, M) of the four W4A4 linears of one block."""
    M = cfg.batch * cfg.tokens
    D, F = cfg.hidden, cfg.mlp
    return [("qkv", D, 3 * D, M), ("o", D, D, M), ("gate_up", D, 2 * F, M), ("down", F, D, M)]


def evict_mall(flush):
    """Make the next launch cold: read a 512 MB buffer, twice the 256 MB MALL,
    so that the cache holds clean lines of it and none of the timed kernel's
    inputs.  A write of the buffer would do the same but leave up to 256 MB of
    dirty lines whose write-back to HBM then overlaps the timed launch (for
    rotate-quantize at M = 16384 that added 23-33 us)."""
    import torch
    flush.view(torch.int32).amax()


def gemm_bytes(M, N, K, out_bytes):
    """Algorithmic HBM bytes of one W4A4 GEMM launch: packed codes of both
    operands, both scale vectors, the output (fp16 store, or fp32 residual
    read + write)."""
    return (M * K + N * K) // 2 + 4 * (M + N) + out_bytes * M * N


def rq_bytes(M, K):
    """Algorithmic HBM bytes of one rotate-quantize launch: fp16 in, int4 + fp32 scale out."""
    return 2 * M * K + M * K // 2 + 4 * M


def time_linears(cfg, qweights, stream):
    """Time each W4A4 linear shape of the step (rotate-quantize + GEMM) through the C ABI."""
    import torch
    import paper_2605_28803_amd as oq
    out = {}
    dev = torch.device("cuda:0")
    g = torch.Generator(device="cpu").manual_seed(0)
    tot = {"rq_ms": 0.0, "rq_bytes": 0, "gemm_ms": 0.0, "gemm_bytes": 0, "gemm_ops": 0, "gemm_launches": 0,
           "rq_launches": 0}
    names = {"qkv": "wqkv", "o": "wo", "gate_up": "wgu", "down": "wd"}
    for name, K, N, M in dit_linears(cfg):
        X = (torch.randn((M, K), generator=g) * 2).half().to(dev)
        Wq, ws = qweights[0][names[name]]
        # Every linear is timed with the fp16-store epilogue; inside the step the
        # o and down projections add into the fp32 residual instead.  Up to 64
        # tokens the step keeps the token codes in the 16-row tiled layout, and
        # so do these timings.
        Y = torch.empty((M, N), dtype=torch.float16, device=dev)
        if M <= 64 and K % 128 == 0:
            Xq, xs = oq.rotate_quantize_act_tiled(X, K & -K, stream=stream)
            gemm = lambda: oq.w4a4_linear_tiled(Xq, xs, Wq, ws, Y=Y)
            rq = lambda: oq.rotate_quantize_act_tiled(X, K & -K, Xt=Xq, x_scale=xs)
        else:
            Xq, xs = oq.rotate_quantize_act(X, K & -K, stream=stream)
            gemm = lambda: oq.w4a4_linear(Xq, xs, Wq, ws, Y=Y)
            rq = lambda: oq.rotate_quantize_act(X, K & -K, Xq=Xq, x_scale=xs)
        t_rq = _graph_time(rq)
        t_g = _graph_time(gemm)
        b_g = gemm_bytes(M, N, K, 2)
        b_r = rq_bytes(M, K)
        out[name] = {"M": M, "N": N, "K": K, "rq_us": round(t_rq * 1e3, 3), "gemm_us": round(t_g * 1e3, 3),
                     "rq_GBs": round(b_r / (t_rq * 1e-3) / 1e9, 1), "gemm_GBs": round(b_g / (t_g * 1e-3) / 1e9, 1),
                     "gemm_TOPs": round(2 * M * N * K / (t_g * 1e-3) / 1e12, 3)}
        tot["rq_ms"] += t_rq
        tot["rq_bytes"] += b_r
        tot["gemm_ms"] += t_g
        tot["gemm_bytes"] += b_g
        tot["gemm_ops"] += 2 * M * N * K
        tot["gemm_launches"] += 1
        tot["rq_launches"] += 1
    return out, tot


ROOFLINE_SHAPE = {"name": "gate_up", "M": 50, "N": 8192, "K": 1024}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_small_gate_up_M50_traffic.txt")


def roofline_gemm(stream=None):
    """The roofline kernel: the W4A4 GEMM of the DiT block's gate|up projection
    (M = 50 tokens, N = 2 x 4096, K = 1024, fp16 out, token codes in the
    16-row tiled layout as inside the step) on seeded weights of block 0,
    timed alone with HIP events around graph replays (no host launch
    overhead), and its rotate-quantize producer likewise.  Returns a dict."""
    import torch
    import paper_2605_28803_amd as oq
    from workloads import configs, generators as G
    cfg = configs.DIT_PI
    M, N, K = ROOFLINE_SHAPE["M"], ROOFLINE_SHAPE["N"], ROOFLINE_SHAPE["K"]
    dev = torch.device("cuda:0")
    W = torch.from_numpy(G.gaussian(cfg.seed, "blk0/wgu", (N, K), cfg.w_std).astype(np.float16)).to(dev)
    Wq, ws = oq.quantize_weights(W, K & -K)
    X = torch.from_numpy(G.gaussian(cfg.seed, "roofline/x", (M, K)).astype(np.float16)).to(dev)
    Xt, xs = oq.rotate_quantize_act_tiled(X, K & -K)
    Y = torch.empty((M, N), dtype=torch.float16, device=dev)
    torch.cuda.synchronize()
    t_g = _graph_time(lambda: oq.w4a4_linear_tiled(Xt, xs, Wq, ws, Y=Y), reps=50, replays=20)
    t_r = _graph_time(lambda: oq.rotate_quantize_act_tiled(X, K & -K, Xt=Xt, x_scale=xs), reps=50, replays=20)
    b = gemm_bytes(M, N, K, 2)
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        for line in open(TRAFFIC_FILE):
            if line.startswith("traffic_bytes_per_launch"):
                traffic = int(float(line.split("=")[1]))
    return {"kernel": "gemm_small_kernel<fp16 out, 32 columns, 8 waves, tiled token codes> (W4A4 gate|up of a "
                      f"DiT block: M={M}, N={N}, K={K})",
            "bound": "hbm", "achieved": round(b / (t_g * 1e-3) / 1e9, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(b / (t_g * 1e-3) / 1e9 / HBM_PEAK_GBS, 4), "traffic": traffic,
            "avg_launch_us": round(t_g * 1e3, 3), "algorithmic_bytes_per_launch": int(b),
            "rotate_quant_us": round(t_r * 1e3, 3)}


def prefill_kernels():
    """One large shape of each kernel, cold (MALL evicted by a read before each launch):
    W4A4 GEMM at M = K = N = 16384 (int8-MFMA roofline) and rotate-quantize at
    M = K = 16384 (HBM roofline); and rotate-quantize back to back on 1.3 GB
    inputs (every launch streams from HBM; its own outputs' write-back overlaps
    the next launch as it would in a pipeline)."""
    import torch
    import paper_2605_28803_amd as oq
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    flush = torch.ones((512 << 20,), dtype=torch.uint8, device=dev)
    M = K = N = 16384
    g = torch.Generator(device=dev).manual_seed(7)
    X = torch.randn((M, K), generator=g, device=dev).half()
    W = (torch.randn((N, K), generator=g, device=dev) * 0.02).half()
    Wq, ws = oq.quantize_weights(W, K)
    del W
    Xq, xs = oq.rotate_quantize_act(X, K)
    Y = torch.empty((M, N), dtype=torch.float16, device=dev)

    def cold(fn, reps):
        ts = []
        for _ in range(reps):
            evict_mall(flush)
            s = torch.cuda.Event(enable_timing=True)
            e = torch.cuda.Event(enable_timing=True)
            s.record(stream)
            fn()
            e.record(stream)
            e.synchronize()
            ts.append(s.elapsed_time(e))
        pct[0] = [round(float(np.percentile(ts, p)) * 1e3, 1) for p in (10, 90)]
        return float(np.median(ts))
    pct = [None]
    oq.w4a4_linear(Xq, xs, Wq, ws, Y=Y)
    t_r = cold(lambda: oq.rotate_quantize_act(X, K, Xq=Xq, x_scale=xs), 15)
    p_r = pct[0]
    ts = []
    for _ in range(15):  # the same launch after a write flush, for comparison
        flush.fill_(1)
        s = torch.cuda.Event(enable_timing=True)
        e = torch.cuda.Event(enable_timing=True)
        s.record(stream)
        oq.rotate_quantize_act(X, K, Xq=Xq, x_scale=xs)
        e.record(stream)
        e.synchronize()
        ts.append(s.elapsed_time(e))
    t_rw = float(np.median(ts))
    t_g = cold(lambda: oq.w4a4_linear(Xq, xs, Wq, ws, Y=Y), 15)
    p_g = pct[0]
    out = {"gemm_M16384_K16384_N16384": {"us": round(t_g * 1e3, 1), "us_p10_p90": p_g,
                                         "TOPs": round(2 * M * N * K / (t_g * 1e-3) / 1e12, 1),
                                         "frac_int8_peak": round(2 * M * N * K / (t_g * 1e-3) / 1e12 / INT8_PEAK_TOPS, 4)},
           "rotate_quant_M16384_K16384": {"us": round(t_r * 1e3, 1), "us_p10_p90": p_r,
                                          "GBs": round(rq_bytes(M, K) / (t_r * 1e-3) / 1e9, 1),
                                          "frac_hbm_peak": round(rq_bytes(M, K) / (t_r * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                                          "after_write_flush_us": round(t_rw * 1e3, 1)}}
    del X, Xq, Y, Wq, flush
    torch.cuda.empty_cache()
    # Back to back on 1.3 GB (beyond the 256 MB MALL, so every launch streams
    # from HBM): rotate-quantize at M = 131072, K = 4096 and M = 32768, K =
    # 16384, median of 20 launches.
    for Mw, Kw in ((131072, 4096), (32768, 16384)):
        X = torch.randn((Mw, Kw), generator=g, device=dev).half()
        Xq = torch.empty((Mw, Kw // 2), dtype=torch.uint8, device=dev)
        xsw = torch.empty((Mw,), dtype=torch.float32, device=dev)
        f = lambda: oq.rotate_quantize_act(X, Kw, Xq=Xq, x_scale=xsw)
        f()
        ts = []
        for _ in range(20):
            s = torch.cuda.Event(enable_timing=True)
            e = torch.cuda.Event(enable_timing=True)
            s.record(stream)
            f()
            e.record(stream)
            e.synchronize()
            ts.append(s.elapsed_time(e))
        t = float(np.median(ts))
        gbs = rq_bytes(Mw, Kw) / (t * 1e-3) / 1e9
        out[f"rotate_quant_M{Mw}_K{Kw}_back_to_back"] = {"us": round(t * 1e3, 1), "GBs": round(gbs, 1),
                                                          "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4)}
        del X, Xq, xsw
    torch.cuda.empty_cache()
    return out


def composite_kernels():
    """The online full composite rotation (zigzag permutation + block-64
    U_b H_64 on the fp16 matrix cores + per-token int4 codes), cold: at
    M = 16384 x K = 1024 and 4096 against the HBM roofline (algorithmic bytes
    2.5 K + 4 per row; perm and the fp16 block matrices, 128 bytes per
    channel, are read once per launch and counted), and at the DiT shape
    (M = 50, K = 1024), whose time is latency.  The permutation comes from
    seeded synthetic weight energies and U_b are seeded random orthogonal
    matrices (the kernel's work does not depend on their values).  Beside each
    online figure: the same transform with P folded into the producer (the
    input already in the permuted order, perm = None), and K = 16384, where
    each row is split into channel chunks whose workgroups exchange their row
    maxima."""
    import torch
    import paper_2605_28803_amd as oq
    from workloads import generators as G
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    flush = torch.ones((512 << 20,), dtype=torch.uint8, device=dev)

    def cold(fn, reps):
        ts = []
        for _ in range(reps):
            evict_mall(flush)
            s = torch.cuda.Event(enable_timing=True)
            e = torch.cuda.Event(enable_timing=True)
            s.record(stream)
            fn()
            e.record(stream)
            e.synchronize()
            ts.append(s.elapsed_time(e))
        return float(np.median(ts))

    out = {}
    for M, K in ((16384, 1024), (16384, 4096), (16384, 16384), (50, 1024)):
        energy = G.gaussian(11, f"composite/energy{K}", (K,)) ** 2
        perm = torch.from_numpy(oq.zigzag_permutation_host(energy, 64)).to(dev)
        U = np.stack([G.random_orthogonal(11, f"composite/u{K}/{b}", 64) for b in range(K // 64)])
        Rt = torch.from_numpy(oq.block_rotations_host(U).view(np.int16)).to(dev)
        g = torch.Generator(device=dev).manual_seed(13)
        X = torch.randn((M, K), generator=g, device=dev).half()
        Xq, xs = oq.rotate_quantize_act_composite(X, perm, Rt)
        t = cold(lambda: oq.rotate_quantize_act_composite(X, perm, Rt, Xq=Xq, x_scale=xs), 15)
        # the same transform with P folded into the producer (perm = None: the
        # input is taken to be in the permuted order already)
        tf = cold(lambda: oq.rotate_quantize_act_composite(X, None, Rt, Xq=Xq, x_scale=xs), 15)
        b = rq_bytes(M, K) + K * 4 + K * 64 * 2
        bf = rq_bytes(M, K) + K * 64 * 2
        out[f"M{M}_K{K}"] = {"us": round(t * 1e3, 2), "GBs": round(b / (t * 1e-3) / 1e9, 1),
                             "frac_hbm_peak": round(b / (t * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                             "perm_folded_us": round(tf * 1e3, 2),
                             "perm_folded_GBs": round(bf / (tf * 1e-3) / 1e9, 1)}
        del X, Xq, xs
    del flush
    torch.cuda.empty_cache()
    return out


def static_scale_kernels():
    """The static per-step, per-channel path, cold: rotate-quantize against a
    step row (algorithmic bytes 2.5 K + 4 per row + 4 K for the row of
    steps) at M = 16384 x K = 1024 / 4096 and at the DiT shape M = 50 (tiled
    codes); the per-token kernel on the same inputs beside it; and the
    calibration collector on n = 16384 rotated rows (fp32 rotation output,
    6 K bytes per row, and the exact column percentile, which reads the
    n x K fp32 rows once per radix pass, 4 passes)."""
    import torch
    import paper_2605_28803_amd as oq
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    flush = torch.ones((512 << 20,), dtype=torch.uint8, device=dev)

    def cold(fn, reps):
        ts = []
        for _ in range(reps):
            evict_mall(flush)
            s = torch.cuda.Event(enable_timing=True)
            e = torch.cuda.Event(enable_timing=True)
            s.record(stream)
            fn()
            e.record(stream)
            e.synchronize()
            ts.append(s.elapsed_time(e))
        return float(np.median(ts))

    def rate(b, t):
        return {"us": round(t * 1e3, 2), "GBs": round(b / (t * 1e-3) / 1e9, 1),
                "frac_hbm_peak": round(b / (t * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}

    out = {}
    g = torch.Generator(device=dev).manual_seed(17)
    for M, K in ((16384, 1024), (16384, 4096), (50, 1024)):
        X = torch.randn((M, K), generator=g, device=dev).half()
        n = 16384
        Yc = oq.rotate_act_f32(torch.randn((n, K), generator=g, device=dev).half(), K)
        delta = oq.calibrate_step_scales(Yc, 99.9, 7.0)
        work = torch.empty((oq.calibrate_workspace_bytes(K),), dtype=torch.uint8, device=dev)
        tiled = M <= 64
        if tiled:
            Xq, xs = oq.rotate_quantize_act_static_tiled(X, K, delta)
            f_static = lambda: oq.rotate_quantize_act_static_tiled(X, K, delta, Xt=Xq, x_scale=xs)
            Xp, xp = oq.rotate_quantize_act_tiled(X, K)
            f_tok = lambda: oq.rotate_quantize_act_tiled(X, K, Xt=Xp, x_scale=xp)
        else:
            Xq, xs = oq.rotate_quantize_act_static(X, K, delta)
            f_static = lambda: oq.rotate_quantize_act_static(X, K, delta, Xq=Xq, x_scale=xs)
            Xp, xp = oq.rotate_quantize_act(X, K)
            f_tok = lambda: oq.rotate_quantize_act(X, K, Xq=Xp, x_scale=xp)
        t_s = cold(f_static, 15)
        t_t = cold(f_tok, 15)
        rec = {"static": rate(rq_bytes(M, K) + 4 * K, t_s), "per_token": rate(rq_bytes(M, K), t_t)}
        if M > 64:
            Y = torch.empty((n, K), dtype=torch.float32, device=dev)
            Xc = torch.randn((n, K), generator=g, device=dev).half()
            t_rot = cold(lambda: oq.rotate_act_f32(Xc, K, Y=Y), 10)
            t_cal = cold(lambda: oq.calibrate_step_scales(Yc, 99.9, 7.0, delta=delta, work=work), 10)
            rec["calib_rotate_f32_n16384"] = rate(n * K * 6, t_rot)
            rec["calib_percentile_n16384"] = dict(rate(n * K * 4, t_cal), passes=4,
                                                  pass_GBs=round(4 * n * K * 4 / (t_cal * 1e-3) / 1e9, 1))
            del Y, Xc
        out[f"M{M}_K{K}"] = rec
        del X, Xq, xs, Xp, xp, Yc, work
    del flush
    torch.cuda.empty_cache()
    return out


def w4a8_kernels():
    """The W4A8 mode, cold: the 8-bit rotate-quantize at M = K = 16384
    (algorithmic bytes 2 K + K + 4 per row), the W4A8 GEMM at M = K = N = 16384
    (2 M N K ops against the int8 MFMA peak) and at the DiT gate|up shape
    (M = 50, N = 8192, K = 1024: bytes M K + N K / 2 + 4 (M + N) + 2 M N
    against HBM), each beside its W4A4 counterpart on the same inputs."""
    import torch
    import paper_2605_28803_amd as oq
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    flush = torch.ones((512 << 20,), dtype=torch.uint8, device=dev)

    def cold(fn, reps):
        ts = []
        for _ in range(reps):
            evict_mall(flush)
            s = torch.cuda.Event(enable_timing=True)
            e = torch.cuda.Event(enable_timing=True)
            s.record(stream)
            fn()
            e.record(stream)
            e.synchronize()
            ts.append(s.elapsed_time(e))
        return float(np.median(ts))

    out = {}
    g = torch.Generator(device=dev).manual_seed(19)
    for M, N, K in ((16384, 16384, 16384), (50, 8192, 1024)):
        X = torch.randn((M, K), generator=g, device=dev).half()
        W = (torch.randn((N, K), generator=g, device=dev) * 0.02).half()
        Wq, ws = oq.quantize_weights(W, K)
        del W
        X8, xs8 = oq.rotate_quantize_act_i8(X, K)
        X4, xs4 = oq.rotate_quantize_act(X, K)
        Y = torch.empty((M, N), dtype=torch.float16, device=dev)
        reps = 10 if M > 64 else 30
        t_r8 = cold(lambda: oq.rotate_quantize_act_i8(X, K, Xq8=X8, x_scale=xs8), reps)
        t_g8 = cold(lambda: oq.w4a8_linear(X8, xs8, Wq, ws, Y=Y), reps)
        t_g4 = cold(lambda: oq.w4a4_linear(X4, xs4, Wq, ws, Y=Y), reps)
        ops = 2 * M * N * K
        rec = {"rotate_quant_i8_us": round(t_r8 * 1e3, 2),
               "rotate_quant_i8_GBs": round(M * (3 * K + 4) / (t_r8 * 1e-3) / 1e9, 1),
               "w4a8_gemm_us": round(t_g8 * 1e3, 2), "w4a4_gemm_us": round(t_g4 * 1e3, 2),
               "w4a8_TOPs": round(ops / (t_g8 * 1e-3) / 1e12, 1),
               "w4a8_frac_int8_peak": round(ops / (t_g8 * 1e-3) / 1e12 / INT8_PEAK_TOPS, 4)}
        if M <= 64:
            b = M * K + N * K // 2 + 4 * (M + N) + 2 * M * N
            rec["w4a8_gemm_GBs"] = round(b / (t_g8 * 1e-3) / 1e9, 1)
        out[f"M{M}_N{N}_K{K}"] = rec
        del X, Wq, ws, X8, X4, Y
    del flush
    torch.cuda.empty_cache()
    return out


def prepare_kernels():
    """Offline composite-rotation weight preparation on the GPU, per weight
    of the Pi-0.5 DiT block (qkv 3072 x 1024, o 1024 x 1024, gate|up 8192 x
    1024, down 1024 x 4096) and the Gemma-2B-shaped gate|up (32768 x 2048):
    the whole oq_prepare_weights_composite call and its steps (energies,
    zigzag ranks, block Gram + Jacobi, fp16 R_b, fold + RTN), warm, median
    of 5.  The energies read N K fp16 once; the Gram kernel reads them once
    more, gathered; the Jacobi sweeps are LDS / latency bound."""
    import torch
    import paper_2605_28803_amd as oq
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()

    def timed(fn, reps=5):
        fn()
        ts = []
        for _ in range(reps):
            s = torch.cuda.Event(enable_timing=True)
            e = torch.cuda.Event(enable_timing=True)
            s.record(stream)
            fn()
            e.record(stream)
            e.synchronize()
            ts.append(s.elapsed_time(e))
        return round(float(np.median(ts)) * 1e3, 1)

    out = {}
    g = torch.Generator(device=dev).manual_seed(23)
    for name, N, K in (("qkv", 3072, 1024), ("o", 1024, 1024), ("gate_up", 8192, 1024), ("down", 1024, 4096),
                       ("gemma_gate_up", 32768, 2048)):
        W = (torch.randn((N, K), generator=g, device=dev) * 0.02).half()
        e = oq.channel_energy(W)
        perm = oq.zigzag_permutation(e)
        U, lam = oq.block_svd(W, perm)
        Rt = oq.block_rotations(U)
        Wq = torch.empty((N, K // 2), dtype=torch.uint8, device=dev)
        ws = torch.empty((N,), dtype=torch.float32, device=dev)
        out[f"{name}_N{N}_K{K}"] = {
            "total_us": timed(lambda: oq.prepare_weights_composite(W)),
            "energy_us": timed(lambda: oq.channel_energy(W, energy=e)),
            "zigzag_us": timed(lambda: oq.zigzag_permutation(e, perm=perm)),
            "block_svd_us": timed(lambda: oq.block_svd(W, perm, U=U, sigma2=lam)),
            "rotations_us": timed(lambda: oq.block_rotations(U, Rt=Rt)),
            "fold_rtn_us": timed(lambda: oq.rotate_quantize_act_composite(W, perm, Rt, Xq=Wq, x_scale=ws)),
        }
        del W, e, perm, U, lam, Rt, Wq, ws
    torch.cuda.empty_cache()
    return out


def copy_calibration():
    """A plain device copy of a known size (256 MiB read + 256 MiB written), the
    reference for scaling the FETCH_SIZE / WRITE_SIZE counters."""
    import torch
    dev = torch.device("cuda:0")
    a = torch.ones((128 << 20,), dtype=torch.float16, device=dev)
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": a.numel() * 2}), flush=True)


def cpu_baseline(cfg, inp, n_blocks_sample=3, min_seconds=10.0):
    """The oracle, untouched, on a bounded sample of the same workload: the
    first n_blocks_sample transformer blocks (identical in shape to the rest),
    run as a chain with t cycling over the denoising steps until at least
    min_seconds of CPU work are done, scaled to the full depth (the in- and
    out-projections, 50 x 32 x 1024 each, are left out).  The sampled blocks'
    weights are quantized beforehand (untimed).  Returns the dict for the JSON
    line."""
    from oracle import dit as odit
    try:
        from threadpoolctl import threadpool_info
        cores = max([int(i.get("num_threads", 1)) for i in threadpool_info()] + [1])
    except Exception:
        cores = 1
    L = n_blocks_sample
    w = dict(inp["w"])
    w["blocks"] = inp["w"]["blocks"][:L]
    qb = odit.quantize_block_weights(cfg, w["blocks"])
    B, S = inp["batch"], cfg.tokens
    r0 = odit.in_projection(w, inp["x0"])
    n = 0
    t0 = time.perf_counter()
    while True:
        r = r0
        for l in range(L):
            r = odit.block(cfg, w, qb, inp["mod"], inp["s_table"], r, l, (n // L) % cfg.steps, B, S,
                           prefix=(inp["kp"], inp["vp"]))
            n += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    steps_per_s = n / dt / cfg.n_blocks
    return {"value": round(steps_per_s, 5), "unit": "DiT denoise-steps/s", "cores": cores, "kind": "oracle",
            "sample": f"{n} block evaluations (blocks 0-{L - 1}, t cycling) in {dt:.1f} s, scaled to "
                      f"{cfg.n_blocks} blocks per step; float64 numpy, BLAS threads={cores}, "
                      f"host cpus={len(os.sched_getaffinity(0))}"}


def gr00t_step():
    """The GR00T-shaped DiT step (16 blocks, hidden 1536, MLP 6144, 32 x 48
    heads, batch 64 x 16 action tokens, 300 conditioning tokens, W4A4
    throughout) timed warm over 20 steps; its W4A4 ops against the int8 MFMA
    peak (the step's compute floor)."""
    import torch
    import paper_2605_28803_amd as oq
    from workloads import configs, dit_inputs
    cfg = configs.DIT_GR00T
    inp = dit_inputs.make_dit_inputs(cfg)
    model = oq.DiT(cfg, inp, device="cuda:0")
    x = torch.from_numpy(inp["x0"].astype(np.float32)).cuda()
    for t in range(cfg.steps):
        model.step(x, t)
    torch.cuda.synchronize()
    s = torch.cuda.Event(enable_timing=True)
    e = torch.cuda.Event(enable_timing=True)
    s.record()
    for i in range(20):
        model.step(x, i % cfg.steps)
    e.record()
    e.synchronize()
    ms = s.elapsed_time(e) / 20
    model.close()
    D, F, M = cfg.hidden, cfg.mlp, cfg.batch * cfg.tokens
    ops = sum(2 * M * D * (D if l % 2 == 0 else 3 * D) + 2 * M * D * D + 4 * M * D * F for l in range(cfg.n_blocks))
    return {"workload": "dit_gr00t: 16 blocks, hidden 1536, mlp 6144, 32x48 heads, batch 64 x 16 tokens, "
                        "300 conditioning tokens, 4 steps",
            "step_us": round(ms * 1e3, 1), "w4a4_GOP_per_step": round(ops / 1e9, 1),
            "TOPs": round(ops / (ms * 1e-3) / 1e12, 1),
            "frac_int8_peak": round(ops / (ms * 1e-3) / 1e12 / INT8_PEAK_TOPS, 4)}


def prefill_linears():
    """The Gemma-2B-shaped prefill layer (816 tokens; q|k|v 2048 -> 2560, o,
    gate|up 2048 -> 32768, down 16384 -> 2048), each linear's rotate-quantize
    and GEMM timed cold (MALL evicted by a read before each launch)."""
    import torch
    import paper_2605_28803_amd as oq
    from workloads import configs
    cfg = configs.PREFILL_GEMMA
    dev = torch.device("cuda:0")
    flush = torch.ones((512 << 20,), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def cold(fn, reps=10):
        ts = []
        for _ in range(reps):
            evict_mall(flush)
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            b.synchronize()
            ts.append(a.elapsed_time(b))
        return float(np.median(ts))
    out, tot_ops, tot_ms = {}, 0, 0.0
    g = torch.Generator(device=dev).manual_seed(3)
    for name, K, N in cfg.linears():
        M = cfg.tokens
        X = torch.randn((M, K), generator=g, device=dev).half()
        W = (torch.randn((N, K), generator=g, device=dev) * cfg.w_std).half()
        Wq, ws = oq.quantize_weights(W, K)
        del W
        Xq, xs = oq.rotate_quantize_act(X, K)
        Y = torch.empty((M, N), dtype=torch.float16, device=dev)
        t_r = cold(lambda: oq.rotate_quantize_act(X, K, Xq=Xq, x_scale=xs))
        t_g = cold(lambda: oq.w4a4_linear(Xq, xs, Wq, ws, Y=Y))
        ops = 2 * M * N * K
        tot_ops += ops
        tot_ms += t_r + t_g
        out[name] = {"M": M, "K": K, "N": N, "rq_us": round(t_r * 1e3, 1), "gemm_us": round(t_g * 1e3, 1),
                     "gemm_TOPs": round(ops / (t_g * 1e-3) / 1e12, 1)}
    out["layer_us"] = round(tot_ms * 1e3, 1)
    out["layer_TOPs"] = round(tot_ops / (tot_ms * 1e-3) / 1e12, 1)
    del flush
    torch.cuda.empty_cache()
    return out


def pi_step_without_graph(cfg, inp, steps=20):
    """The same Pi-0.5-shaped step launched kernel by kernel (no HIP graph)."""
    import torch
    import paper_2605_28803_amd as oq
    os.environ["OQ_DIT_NO_GRAPH"] = "1"
    try:
        model = oq.DiT(cfg, inp, device="cuda:0")
    finally:
        del os.environ["OQ_DIT_NO_GRAPH"]
    x = torch.from_numpy(inp["x0"].astype(np.float32)).cuda()
    for t in range(3):
        model.step(x, t)
    torch.cuda.synchronize()
    s = torch.cuda.Event(enable_timing=True)
    e = torch.cuda.Event(enable_timing=True)
    s.record()
    for i in range(steps):
        model.step(x, i % cfg.steps)
    e.record()
    e.synchronize()
    model.close()
    return s.elapsed_time(e) / steps


def dit_static_step(cfg, inp, model, n_traj=24, steps=50):
    """The Pi-0.5 step with the paper-literal static per-step, per-channel
    steps: calibration rollouts (n_traj seeded synthetic initial states, all
    10 denoising steps, every block and site; 24 x 50 = 1200 rows per
    (block, step, site), so that the nearest-rank 99.9th percentile is the
    second largest magnitude, not the largest), the per-(block, step) weight
    folds on the device, then the step timed as the main line (graph replay,
    t cycling) -- ten weight copies per block, so the step's weights are no
    longer MALL-resident across steps.  Also reports how far a full
    10-step denoise moves from the per-token driver's (relative L2, not a
    parity figure: both are quantized models)."""
    import torch
    from workloads import generators as G
    stream = torch.cuda.current_stream()
    x0s = [torch.from_numpy(G.gaussian(900 + j, "calib/x0", inp["x0"].shape).astype(np.float32)).cuda()
           for j in range(n_traj)]
    t0 = time.perf_counter()
    table = model.calibrate_static_steps(x0s)
    t_cal = time.perf_counter() - t0
    t0 = time.perf_counter()
    model.set_static_steps(inp, table)
    t_fold = time.perf_counter() - t0
    x = torch.from_numpy(inp["x0"].astype(np.float32)).cuda()
    for k in range(10):
        model.step(x, k % cfg.steps, stream=stream)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for k in range(steps):
        model.step(x, k % cfg.steps, stream=stream)
    end.record(stream)
    end.synchronize()
    ms = start.elapsed_time(end) / steps
    xs = torch.from_numpy(inp["x0"].astype(np.float32)).cuda()
    model.denoise(xs, cfg.steps, stream=stream)
    model.clear_static_steps()
    xt = torch.from_numpy(inp["x0"].astype(np.float32)).cuda()
    model.denoise(xt, cfg.steps, stream=stream)
    torch.cuda.synchronize()
    x0 = torch.from_numpy(inp["x0"].astype(np.float32)).cuda()
    dev = float(torch.linalg.norm(xs - xt) / torch.linalg.norm(xt - x0))
    del table
    torch.cuda.empty_cache()
    return {"step_us": round(ms * 1e3, 2), "steps_per_s": round(1000.0 / ms, 1),
            "calibration_s": round(t_cal, 2), "calibration_trajectories": n_traj,
            "weight_folds_s": round(t_fold, 2), "folded_weight_copies": cfg.n_blocks * cfg.steps * 4,
            "denoise_vs_per_token_rel_l2": round(dev, 4)}


# The paper's own figures (context, not targets: other hardware, other
# precision, whole-model storage), from its Table tab:memory_savings and
# Appendix B Table tab:real_quant_latency.
PAPER_CONTEXT = {
    "static_memory_savings": {
        "gr00t_n1.5": {"fp16_GB": 1.99, "quantized_MB": 586, "saving": 0.713, "q_layers": 180},
        "pi0.5": {"fp16_GB": 4.27, "quantized_GB": 1.20, "saving": 0.720, "q_layers": 252},
        "what": "whole-model static memory, W4 weights plus quantization metadata (storage, no hardware)",
        "source": "Table tab:memory_savings"},
    "per_step_latency_ms": {
        "fp16": 32.2, "omega_qvla_w4a8": 26.7, "qvla_real": 27.1, "quantvla_real": 29.8,
        "hardware": "NVIDIA H100", "precision": "W4A8 (INT8 tensor-core GEMM, packed INT4 weights)",
        "workload": "Pi-0.5 policy, LIBERO Spatial task 0, 3 episodes (one policy call per step)",
        "source": "Appendix B, Table tab:real_quant_latency"},
}


def static_footprint():
    """Storage of every quantized linear of the synthetic workloads against
    fp16: packed int4 codes + one fp32 scale per output channel (+ the fp32
    step-scale table of the DiT sites), the analogue of the paper's static
    memory saving (linears only: norms, embeddings and the rest of a real
    policy stay outside this count)."""
    from workloads import configs
    out = {}

    def entry(linears, extra_bytes=0):
        fp16 = sum(2 * n * k for n, k in linears)
        q = sum(n * k // 2 + 4 * n for n, k in linears) + extra_bytes
        return {"fp16_MB": round(fp16 / 1e6, 1), "w4_MB": round(q / 1e6, 1), "saving": round(1 - q / fp16, 4),
                "linears": len(linears)}

    c = configs.DIT_PI
    D, F = c.hidden, c.mlp
    lin = [(3 * D, D), (D, D), (2 * F, D), (D, F)] * c.n_blocks
    out["dit_pi05_expert"] = entry(lin, 4 * c.n_blocks * c.steps * 4)
    c = configs.DIT_GR00T
    D, F = c.hidden, c.mlp
    lin = []
    for l in range(c.n_blocks):
        lin += ([(D, D), (2 * D, D)] if l % 2 == 0 else [(3 * D, D)]) + [(D, D), (F, D), (D, F)]
    out["dit_gr00t"] = entry(lin, 4 * c.n_blocks * c.steps * 4)
    p = configs.PREFILL_GEMMA
    lin = [(n, k) for _, k, n in p.linears()] * p.n_layers
    out["backbone_gemma2b_18_layers"] = entry(lin)
    return out


def single_linear(stream):
    """The single rotated linear (64 x 1024 activation with 8 outlier channels
    x50, 1024 x 1024 weight with a random orthogonal U folded in, b = 1024,
    s_t = 1): rotate-quantize + W4A4 GEMM latency, warm (graph replays) and
    cold (MALL evicted by a read before each pair)."""
    import torch
    import paper_2605_28803_amd as oq
    from workloads import configs, linear_inputs
    case = configs.LINEAR_1024
    inp = linear_inputs.make_linear_inputs(case)
    dev = torch.device("cuda:0")
    X = torch.from_numpy(inp["x"].astype(np.float16)).to(dev)
    W = torch.from_numpy((inp["w"] @ inp["u"]).astype(np.float16)).to(dev)  # U folded offline
    Wq, ws = oq.quantize_weights(W, case.had_block)
    Xq = torch.empty((case.M, case.K // 2), dtype=torch.uint8, device=dev)
    xs = torch.empty((case.M,), dtype=torch.float32, device=dev)
    Y = torch.empty((case.M, case.N), dtype=torch.float16, device=dev)

    def pair():  # on the current stream (the capture stream inside _graph_time)
        oq.rotate_quantize_act(X, case.had_block, Xq=Xq, x_scale=xs)
        oq.w4a4_linear(Xq, xs, Wq, ws, Y=Y)

    warm = _graph_time(pair, reps=50, replays=20)
    flush = torch.ones((512 << 20,), dtype=torch.uint8, device=dev)
    ts = []
    for _ in range(30):
        evict_mall(flush)
        s = torch.cuda.Event(enable_timing=True)
        e = torch.cuda.Event(enable_timing=True)
        s.record(stream)
        pair()
        e.record(stream)
        e.synchronize()
        ts.append(s.elapsed_time(e))
    del flush
    return {"M": case.M, "K": case.K, "N": case.N, "warm_us": round(warm * 1e3, 2),
            "cold_us": round(float(np.median(ts)) * 1e3, 2),
            "note": "rotate-quantize + GEMM with epilogue, two launches; latency-bound (164 KB, 134 MOP)"}


def gemm_roofline(M, N, K, t_ms):
    """Achieved TOP/s of a W4A4 GEMM launch and its fraction of the roofline
    min(int8 peak, arithmetic intensity x HBM bandwidth) over its algorithmic
    bytes (fp16 output)."""
    ops = 2.0 * M * N * K
    b = gemm_bytes(M, N, K, 2)
    ai = ops / b
    roof = min(INT8_PEAK_TOPS, ai * HBM_PEAK_GBS / 1e3)
    tops = ops / (t_ms * 1e-3) / 1e12
    return {"gemm_us": round(t_ms * 1e3, 2), "gemm_TOPs": round(tops, 2),
            "gemm_frac_int8": round(tops / INT8_PEAK_TOPS, 4),
            "gemm_GBs": round(b / (t_ms * 1e-3) / 1e9, 1),
            "gemm_bound": "hbm" if ai * HBM_PEAK_GBS / 1e3 < INT8_PEAK_TOPS else "mfma",
            "gemm_roofline_TOPs": round(roof, 1), "gemm_frac_roofline": round(tops / roof, 4)}


def sweep_records(Ms=None, Ks=None, reps=10, sink=None):
    """Rotate-quantize and W4A4 GEMM at M x (K = N), cold (a 512 MB read
    evicts the MALL before each timed launch).  Inputs per shape: seed 1000 +
    10 iM + iK; X ~ N(0, 1) with round(0.01 K) outlier channels x50 and W ~
    N(0, 0.02^2), drawn on the device with torch's generator under that seed;
    Hadamard block K."""
    import torch
    import paper_2605_28803_amd as oq
    from workloads import configs
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    flush = torch.ones((512 << 20,), dtype=torch.uint8, device=dev)
    out = []
    for case in configs.SWEEP.cases():
        M, K, N = case.M, case.K, case.N
        if (Ms and M not in Ms) or (Ks and K not in Ks):
            continue
        g = torch.Generator(device=dev).manual_seed(case.seed)
        X = torch.randn((M, K), generator=g, device=dev)
        ch = torch.randperm(K, generator=g, device=dev)[: case.outlier_count]
        X[:, ch] *= case.outlier_factor
        X = X.half()
        W = (torch.randn((N, K), generator=g, device=dev) * case.w_std).half()
        Wq, ws = oq.quantize_weights(W, K)
        del W
        Xq, xs = oq.rotate_quantize_act(X, K)
        Y = torch.empty((M, N), dtype=torch.float16, device=dev)

        def timed(fn):
            ts = []
            for _ in range(reps):
                evict_mall(flush)
                s = torch.cuda.Event(enable_timing=True)
                e = torch.cuda.Event(enable_timing=True)
                s.record(stream)
                fn()
                e.record(stream)
                e.synchronize()
                ts.append(s.elapsed_time(e))
            return float(np.median(ts)), [round(float(np.percentile(ts, p)) * 1e3, 2) for p in (10, 90)]

        rq = lambda: oq.rotate_quantize_act(X, K, Xq=Xq, x_scale=xs, stream=stream)
        gm = lambda: oq.w4a4_linear(Xq, xs, Wq, ws, Y=Y, stream=stream)
        rq()
        gm()
        t_rq, rq_p = timed(rq)
        t_g, g_p = timed(gm)
        rb = rq_bytes(M, K)
        rec = {"M": M, "K": K, "N": N, "seed": case.seed, "rq_us": round(t_rq * 1e3, 2), "rq_us_p10_p90": rq_p,
               "rq_GBs": round(rb / (t_rq * 1e-3) / 1e9, 1),
               "rq_frac_hbm": round(rb / (t_rq * 1e-3) / 1e9 / HBM_PEAK_GBS, 4), "rq_MB": round(rb / 1e6, 2)}
        rec.update(gemm_roofline(M, N, K, t_g))
        rec["gemm_us_p10_p90"] = g_p
        out.append(rec)
        if sink is not None:
            sink(rec)
        del Xq, xs, Y, Wq, ws, X
    del flush
    torch.cuda.empty_cache()
    return out


def prefill_gemms(reps=5):
    """The six prefill GEMM shapes (M in {4096, 16384} x K = N in {4096, 8192,
    16384}), cold, reps launches each: the command the MFMA counter summary
    of the W4A4 GEMM is taken with (sweep inputs and timing)."""
    return [r for r in sweep_records(Ms=[4096, 16384], Ks=[4096, 8192, 16384], reps=reps)]


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_kernel_baselines(rq_rows=384, gemm_rows=32, M=16384, K=16384):
    """The oracle's rotate-quantize and integer GEMM on this host at the
    prefill shape M = K = N = 16384 (float64 / int64 numpy, untouched), each
    on a bounded sample of rows, single-threaded (BLAS limited to one thread;
    the rotate-quantize over the same row chunks, one after the other) and
    with every host core (the row chunks on a thread pool for the
    rotate-quantize, the BLAS thread pool for the GEMM), extrapolated x M /
    rows to the whole launch."""
    import concurrent.futures as cf
    from threadpoolctl import threadpool_limits
    from oracle import linear as olin
    from oracle import quant as oquant
    cores = len(os.sched_getaffinity(0))
    rng = np.random.default_rng(2024)
    x = rng.standard_normal((rq_rows, K)).astype(np.float16).astype(np.float64)
    out = {"cpu_model": cpu_model(), "host_cores": cores}
    # The same row chunks serially on one thread, then on a pool of every core.
    chunks = np.array_split(np.arange(rq_rows), cores)
    with threadpool_limits(1):
        t0 = time.perf_counter()
        q = np.concatenate([oquant.rotate_quantize_act(x[r], K, 1.0)[0] for r in chunks])
        t1 = time.perf_counter() - t0
    with threadpool_limits(1), cf.ThreadPoolExecutor(cores) as ex:
        t0 = time.perf_counter()
        list(ex.map(lambda r: oquant.rotate_quantize_act(x[r], K, 1.0), chunks))
        tn = time.perf_counter() - t0
    rb = rq_bytes(M, K)
    out["rotate_quant"] = {"shape": f"M={M} K={K}", "rows_sampled": rq_rows,
                           "single_thread_s": round(t1 * M / rq_rows, 2),
                           "all_cores_s": round(tn * M / rq_rows, 2), "threads": cores,
                           "single_thread_GBs": round(rb / (t1 * M / rq_rows) / 1e9, 4),
                           "all_cores_GBs": round(rb / (tn * M / rq_rows) / 1e9, 4),
                           "kind": "extrapolated x M/rows"}
    qw = rng.integers(-7, 8, size=(K, K)).astype(np.int64)  # N = K weight codes (timing only)
    qa = q[:gemm_rows]
    with threadpool_limits(1):
        t0 = time.perf_counter()
        olin.int_gemm(qa, qw)
        g1 = time.perf_counter() - t0
    with threadpool_limits(cores):
        t0 = time.perf_counter()
        olin.int_gemm(qa, qw)
        gn = time.perf_counter() - t0
    ops = 2.0 * M * K * K
    out["gemm"] = {"shape": f"M={M} N={K} K={K}", "rows_sampled": gemm_rows,
                   "single_thread_s": round(g1 * M / gemm_rows, 1), "all_cores_s": round(gn * M / gemm_rows, 1),
                   "threads": cores, "single_thread_TOPs": round(ops / (g1 * M / gemm_rows) / 1e12, 6),
                   "all_cores_TOPs": round(ops / (gn * M / gemm_rows) / 1e12, 6),
                   "kind": "extrapolated x M/rows (exact int GEMM as a float64 BLAS product of the codes)"}
    return out


def run_dit(args):
    import torch
    import paper_2605_28803_amd as oq
    from workloads import configs, dit_inputs

    cfg = configs.DIT_PI
    t0 = time.perf_counter()
    inp = dit_inputs.make_dit_inputs(cfg)
    model = oq.DiT(cfg, inp, device="cuda:0")
    setup_s = time.perf_counter() - t0
    print(f"[bench] setup {setup_s:.1f} s", file=sys.stderr, flush=True)
    stream = torch.cuda.current_stream()
    x = torch.from_numpy(inp["x0"].astype(np.float32)).cuda()
    x_init = x.clone()

    t = 0
    for _ in range(args.warmup):
        model.step(x, t % cfg.steps, stream=stream)
        t += 1
    torch.cuda.synchronize()
    x.copy_(x_init)
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for k in range(args.steps):
        model.step(x, k % cfg.steps, stream=stream)
    end.record(stream)
    end.synchronize()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / args.steps
    assert torch.isfinite(x).all().item(), "non-finite action state"
    print(f"[bench] {args.steps} steps, {ms:.3f} ms/step", file=sys.stderr, flush=True)
    # Per-step latency distribution (after the timed region; not part of value):
    # 50 single steps, each between its own events.
    per = []
    for k in range(50):
        s_ev = torch.cuda.Event(enable_timing=True)
        e_ev = torch.cuda.Event(enable_timing=True)
        s_ev.record(stream)
        model.step(x, k % cfg.steps, stream=stream)
        e_ev.record(stream)
        e_ev.synchronize()
        per.append(s_ev.elapsed_time(e_ev) * 1e3)
    step_dist = {"steps": 50, "median_us": round(float(np.median(per)), 2),
                 "p10_us": round(float(np.percentile(per, 10)), 2), "p90_us": round(float(np.percentile(per, 90)), 2)}

    nograph_ms = pi_step_without_graph(cfg, inp)
    # Bytes a step must stream: every block's int4 weights and scales, and the
    # prefix K/V.
    D, F = cfg.hidden, cfg.mlp
    step_bytes = cfg.n_blocks * ((3 * D * D + D * D + 2 * F * D + D * F) // 2 + 4 * (3 * D + D + 2 * F + D)
                                 + 2 * 2 * cfg.prefix * D)
    kern, tot = time_linears(cfg, model.qweights, stream)
    rq_gbs = tot["rq_bytes"] / (tot["rq_ms"] * 1e-3) / 1e9
    roof = roofline_gemm()
    prefill = None if args.no_prefill else prefill_kernels()
    line = {
        "metric": METRIC,
        "value": round(1000.0 / ms, 3),
        "unit": "DiT denoise-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int4xint4->i32",
        "data": "synthetic",
        "config": {"workload": "dit_pi05_expert: 18 blocks, hidden 1024, mlp 4096 (gate|up, down), 8x128 heads, "
                               "50 action + 816 prefix tokens, batch 1, 10 denoising steps, W4A4 all block linears, "
                               "Hadamard 1024/4096, s_t log-uniform [0.5,4]",
                   "global_batch": 1, "seq_len": cfg.tokens, "timing": "warm (weights + prefix K/V fit the MALL)"},
        "dit_step_latency_us": round(ms * 1e3, 2),
        "dit_step_single_launch_us": step_dist,
        "dit_step_without_graph_us": round(nograph_ms * 1e3, 2),
        "dit_step_stream": {"bytes": int(step_bytes), "GBs": round(step_bytes / (ms * 1e-3) / 1e9, 1),
                            "hbm_floor_us": round(step_bytes / HBM_PEAK_GBS / 1e3, 1)},
        "roofline": roof,
        "kernels": {"per_linear": kern, "prefill": prefill,
                    "rotate_quant_GBs": round(rq_gbs, 1),
                    "gemm_TOPs": round(tot["gemm_ops"] / (tot["gemm_ms"] * 1e-3) / 1e12, 3),
                    "gemm_frac_int8_peak": round(tot["gemm_ops"] / (tot["gemm_ms"] * 1e-3) / 1e12 / INT8_PEAK_TOPS, 5)},
    }
    if not args.no_prefill:
        print("[bench] gr00t-shaped step, prefill layer", file=sys.stderr, flush=True)
        line["dit_gr00t"] = gr00t_step()
        line["prefill_gemma2b_layer"] = prefill_linears()
        line["composite_rotate_quant"] = composite_kernels()
        line["static_step_scales"] = static_scale_kernels()
        line["w4a8"] = w4a8_kernels()
        line["weight_preparation"] = prepare_kernels()
        print("[bench] static per-step steps (calibration + step)", file=sys.stderr, flush=True)
        line["dit_static_steps"] = dit_static_step(cfg, inp, model)
    line["single_linear_64x1024x1024"] = single_linear(stream)
    if not args.no_prefill:
        print("[bench] roofline sweep (25 shapes, cold)", file=sys.stderr, flush=True)
        line["sweep"] = sweep_records()
    line["static_footprint"] = static_footprint()
    line["paper_context"] = PAPER_CONTEXT
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (oracle sample)", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(cfg, inp)
        print("[bench] cpu oracle kernels (rotate-quantize, GEMM samples)", file=sys.stderr, flush=True)
        line["cpu_oracle_kernels"] = cpu_kernel_baselines()
    model.close()
    print(json.dumps(line), flush=True)


def run_sweep(args):
    """The rotate-quantize / GEMM roofline sweep alone (sweep_records), as JSON
    lines on stdout and, when args.sweep_out names a file, in that file."""
    Ms = [int(m) for m in args.sweep_m.split(",")] if args.sweep_m else None
    Ks = [int(k) for k in args.sweep_k.split(",")] if args.sweep_k else None
    f = None
    if args.sweep_out:
        path = os.path.abspath(args.sweep_out)
        os.makedirs(os.path.dirname(path), exist_ok=True)
        f = open(path, "w")

    def sink(rec):
        if f is not None:
            f.write(json.dumps(rec) + "\n")
            f.flush()
        print(json.dumps(rec), flush=True)
    try:
        sweep_records(Ms, Ks, reps=20, sink=sink)
    finally:
        if f is not None:
            f.close()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--sweep", action="store_true")
    ap.add_argument("--sweep-out", default="", help="file that also receives the --sweep JSON lines")
    ap.add_argument("--sweep-m", default="")
    ap.add_argument("--sweep-k", default="")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--roofline-only", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--gr00t-only", action="store_true")
    ap.add_argument("--composite-only", action="store_true")
    ap.add_argument("--static-only", action="store_true")
    ap.add_argument("--w4a8-only", action="store_true")
    ap.add_argument("--prepare-only", action="store_true")
    ap.add_argument("--cpu-kernels-only", action="store_true")
    ap.add_argument("--gemm-prefill-only", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (--gpus must be 1)", file=sys.stderr)
        sys.exit(2)
    if args.sweep:
        run_sweep(args)
    elif args.roofline_only:
        print(json.dumps({"roofline": roofline_gemm()}), flush=True)
    elif args.copy_calibration:
        copy_calibration()
    elif args.gr00t_only:
        print(json.dumps({"dit_gr00t": gr00t_step()}), flush=True)
    elif args.composite_only:
        print(json.dumps({"composite_rotate_quant": composite_kernels()}), flush=True)
    elif args.static_only:
        print(json.dumps({"static_step_scales": static_scale_kernels()}), flush=True)
    elif args.w4a8_only:
        print(json.dumps({"w4a8": w4a8_kernels()}), flush=True)
    elif args.prepare_only:
        print(json.dumps({"weight_preparation": prepare_kernels()}), flush=True)
    elif args.gemm_prefill_only:
        for rec in prefill_gemms():
            print(json.dumps(rec), flush=True)
    elif args.cpu_kernels_only:
        print(json.dumps({"cpu_oracle_kernels": cpu_kernel_baselines()}), flush=True)
    else:
        run_dit(args)


if __name__ == "__main__":
    main()
