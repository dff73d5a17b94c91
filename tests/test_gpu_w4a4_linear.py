"""W4A4 product and dequantizing epilogue against the oracle (GPU).

int32 accumulators must be bit-exact given identical codes; fp16 / bf16
outputs within 2e-3 relative L2 of the oracle fed identical codes and scales;
the full rotated linear (independent codes on both sides) within the same."""
import numpy as np
import pytest
import torch

import paper_2605_28803_amd as oq
from oracle import linear, quant
from tests import parity
from workloads import configs, linear_inputs

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _codes(rng, R, K):
    return rng.integers(-7, 8, size=(R, K))


@pytest.mark.parametrize("M,N,K", [(1, 64, 64), (50, 1024, 1024), (64, 128, 128), (200, 320, 1024),
                                   (257, 192, 1536), (130, 3072, 1024), (33, 256, 4096),
                                   (300, 512, 6144),
                                   # small-M row-layout kernel: a final 64-code step (K % 128 == 64),
                                   # 16-row and 64-row groups, 16- and 32-column tiles
                                   (50, 1024, 1088), (17, 2048, 320), (64, 520, 4160), (3, 100, 64),
                                   (16, 4160, 2112), (50, 8192, 1024), (50, 1024, 4096),
                                   # two K groups (alternate 128-code stages summed through LDS):
                                   # the second group's only stage a half stage, no stage at all, an
                                   # odd stage count, deep K, and 256 128 x 128 tiles (ragged N)
                                   (1000, 1000, 192), (130, 200, 64), (500, 700, 320), (520, 1000, 6208),
                                   (250, 16376, 320), (256, 16384, 1536),
                                   # two local stages, the second a half stage (group 0 at K = 320,
                                   # group 1 at K = 448; one group at K = 192 with 520 tiles): its
                                   # skipped sub-steps must add nothing
                                   (500, 700, 448), (500, 4160, 192)])
def test_i32_accumulators_bit_exact(M, N, K):
    print(f"gemm i32 M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M + N + K)
    q, qw = _codes(rng, M, K), _codes(rng, N, K)
    acc = oq.w4a4_gemm_i32(torch.from_numpy(parity.pack_int4(q)).to(DEV),
                           torch.from_numpy(parity.pack_int4(qw)).to(DEV))
    torch.cuda.synchronize()
    assert np.array_equal(acc.cpu().numpy().astype(np.int64), linear.int_gemm(q, qw))


@pytest.mark.parametrize("M,N,K", [(4096, 4096, 256), (4100, 4160, 192), (8192, 2048, 128), (2048, 8320, 64),
                                   (4096, 4096, 320), (2100, 4160, 192), (8192, 4096, 448), (1100, 8200, 128),
                                   (2100, 2100, 192),
                                   # 384 / 430 tiles of 128 x 128: ragged edges, a final half stage
                                   (1000, 6100, 1536), (1200, 5500, 448)])
def test_i32_bit_exact_large_tiles(M, N, K):
    """Shapes that take the 256 x 256 and the 128 x 128 tile paths, with ragged edges (the 64 x 64 tile
    is taken by the M > 64 shapes of test_i32_accumulators_bit_exact)."""
    print(f"gemm i32 large M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M + 3 * N + 7 * K)
    q, qw = _codes(rng, M, K), _codes(rng, N, K)
    acc = oq.w4a4_gemm_i32(torch.from_numpy(parity.pack_int4(q)).to(DEV),
                           torch.from_numpy(parity.pack_int4(qw)).to(DEV))
    torch.cuda.synchronize()
    assert np.array_equal(acc.cpu().numpy().astype(np.int64), linear.int_gemm(q, qw))


def test_i32_extreme_magnitudes():
    """Every code +-7 at K = 16384: |acc| = 49 K, the largest the format allows."""
    K = 16384
    q = np.full((3, K), 7)
    q[1] = -7
    q[2, ::2] = -7
    qw = np.full((4, K), 7)
    qw[1] = -7
    qw[2, 1::2] = -7
    acc = oq.w4a4_gemm_i32(torch.from_numpy(parity.pack_int4(q)).to(DEV),
                           torch.from_numpy(parity.pack_int4(qw)).to(DEV)).cpu().numpy()
    assert np.array_equal(acc.astype(np.int64), linear.int_gemm(q, qw))
    assert acc[0, 0] == 49 * K and acc[1, 0] == -49 * K


@pytest.mark.parametrize("out_dtype", [oq.OUT_F16, oq.OUT_BF16])
@pytest.mark.parametrize("M,N,K", [(50, 1024, 1024), (200, 320, 2048), (77, 1000, 4096), (250, 16376, 320),
                                   (1000, 1000, 3072)])
def test_dequant_epilogue(M, N, K, out_dtype):
    rng = np.random.default_rng(M * N + K)
    q, qw = _codes(rng, M, K), _codes(rng, N, K)
    xs = rng.uniform(0.01, 2.0, M).astype(np.float32)
    ws = rng.uniform(1e-4, 1e-2, N).astype(np.float32)
    bias = (rng.standard_normal(N) * 0.1).astype(np.float16)
    Y = oq.w4a4_linear(torch.from_numpy(parity.pack_int4(q)).to(DEV), torch.from_numpy(xs).to(DEV),
                       torch.from_numpy(parity.pack_int4(qw)).to(DEV), torch.from_numpy(ws).to(DEV),
                       bias=torch.from_numpy(bias).to(DEV), out_dtype=out_dtype)
    ref = linear.dequant(linear.int_gemm(q, qw), xs, ws, bias.astype(np.float64))
    err = parity.rel_l2(Y.float().cpu().numpy(), ref)
    print(f"dequant rel_l2={err:.3e}")
    assert err <= parity.REL_L2_OUT


def test_full_rotated_linear_1024():
    """The single rotated linear: X [64 x 1024] with 8 outlier channels x50,
    W [1024 x 1024] ~ N(0, 0.02^2), U random orthogonal folded into W, b = 1024,
    s_t = 1.  Both sides quantize independently."""
    case = configs.LINEAR_1024
    inp = linear_inputs.make_linear_inputs(case)
    w_u = inp["w"] @ inp["u"]
    b = case.had_block
    X = torch.from_numpy(inp["x"].astype(np.float16)).to(DEV)
    Xq, xs = oq.rotate_quantize_act(X, b)
    Wq, ws = oq.quantize_weights_host(w_u, b)
    Y = oq.w4a4_linear(Xq, xs, torch.from_numpy(Wq).to(DEV), torch.from_numpy(ws).to(DEV))
    torch.cuda.synchronize()
    ref = linear.w4a4_linear(inp["x"], w_u, b)
    # Codes of the activation against the oracle's.
    tau = parity.tau_rows(inp["x"], b)
    n_mis, _ = parity.check_codes(parity.unpack_int4(Xq.cpu().numpy()), ref["q"], ref["ratio"], tau)
    # Accumulators exact given the GPU's own codes.
    acc = oq.w4a4_gemm_i32(Xq, torch.from_numpy(Wq).to(DEV)).cpu().numpy()
    q_gpu = parity.unpack_int4(Xq.cpu().numpy())
    assert np.array_equal(acc.astype(np.int64), linear.int_gemm(q_gpu, parity.unpack_int4(Wq)))
    # Output against the oracle fed the GPU's codes and scales, and against the
    # fully independent oracle pipeline.
    y = Y.float().cpu().numpy()
    same = linear.dequant(acc, xs.cpu().numpy(), ws)
    assert parity.rel_l2(y, same) <= parity.REL_L2_OUT
    e_ind = parity.rel_l2(y, ref["y"])
    print(f"cfg linear_1024: code mismatches={n_mis}, rel_l2 vs independent oracle={e_ind:.3e}")
    assert e_ind <= parity.REL_L2_OUT
    # Information: the quantized layer approximates the unrotated fp64 product.
    exact = (inp["x"] @ inp["u"].T) @ inp["w"].T
    print(f"  W4A4 vs exact fp64 rel_l2={parity.rel_l2(y, exact):.3e}")


def _random_packed(R, K, gen):
    """Packed int4 codes uniform in [-7, 7], generated on the device."""
    u = torch.randint(0, 15, (R, K), generator=gen, device=DEV, dtype=torch.int16) - 7
    n = (u & 0xF).to(torch.uint8)
    return (n[:, 0::2] | (n[:, 1::2] << 4)).contiguous()


@pytest.mark.parametrize("M,N,K", [(16384, 16384, 16384), (4096, 8192, 8192), (816, 32768, 2048)])
def test_gemm_full_size_sampled(M, N, K):
    """Full-size launches (the prefill / sweep shapes and the launch bench.py
    times): sampled rows x sampled columns of the i32 accumulators bit-exact,
    and of the fp16 epilogue within 2e-3, against the oracle on the same codes."""
    print(f"gemm full-size M={M} N={N} K={K}", flush=True)
    gen = torch.Generator(device=DEV).manual_seed(M ^ N ^ K)
    Xq, Wq = _random_packed(M, K, gen), _random_packed(N, K, gen)
    xs = torch.rand(M, generator=gen, device=DEV) * 0.1 + 0.01
    ws = torch.rand(N, generator=gen, device=DEV) * 1e-3 + 1e-4
    rng = np.random.default_rng(K)
    rows = np.unique(np.concatenate([rng.choice(M, 24, replace=False), [0, M - 1]]))
    cols = np.unique(np.concatenate([rng.choice(N, 256, replace=False), [0, N - 1]]))
    q = parity.unpack_int4(Xq[torch.from_numpy(rows).to(DEV)].cpu().numpy())
    qw = parity.unpack_int4(Wq[torch.from_numpy(cols).to(DEV)].cpu().numpy())
    ref = linear.int_gemm(q, qw)
    acc = oq.w4a4_gemm_i32(Xq, Wq)
    torch.cuda.synchronize()
    a = acc[torch.from_numpy(rows).to(DEV)][:, torch.from_numpy(cols).to(DEV)].cpu().numpy()
    del acc
    assert np.array_equal(a.astype(np.int64), ref)
    Y = oq.w4a4_linear(Xq, xs, Wq, ws)
    torch.cuda.synchronize()
    y = Y[torch.from_numpy(rows).to(DEV)][:, torch.from_numpy(cols).to(DEV)].float().cpu().numpy()
    yref = linear.dequant(ref, xs.cpu().numpy()[rows].astype(np.float64), ws.cpu().numpy()[cols].astype(np.float64))
    err = parity.rel_l2(y, yref)
    print(f"  sampled {len(rows)}x{len(cols)}: i32 exact, fp16 rel_l2={err:.2e}")
    assert err <= parity.REL_L2_OUT


@pytest.mark.parametrize("name,K,N", configs.PREFILL_GEMMA.linears())
def test_prefill_layer_linears(name, K, N):
    """Backbone prefill, Gemma-2B shaped (816 tokens; q|k|v 2048 -> 2560,
    o 2048 -> 2048, gate|up 2048 -> 32768, down 16384 -> 2048; activations with
    0.5% outlier channels x30; W ~ N(0, 0.02^2); b = K): device weight codes
    against the oracle's (boundary rule), activation codes of sampled rows, and
    the sampled rows' outputs against the oracle fed the GPU's codes."""
    from workloads import generators as G
    cfg = configs.PREFILL_GEMMA
    M = cfg.tokens
    print(f"prefill {name}: M={M} K={K} N={N}", flush=True)
    x = G.gaussian(cfg.seed, f"prefill/{name}/x", (M, K))
    x[:, G.outlier_channels(cfg.seed, f"prefill/{name}/x", K, int(round(cfg.outlier_frac * K)))] *= cfg.outlier_factor
    x16 = x.astype(np.float16)
    w16 = G.gaussian(cfg.seed, f"prefill/{name}/w", (N, K), cfg.w_std).astype(np.float16)
    Wq, ws = oq.quantize_weights(torch.from_numpy(w16).to(DEV), K)
    Xq, xs = oq.rotate_quantize_act(torch.from_numpy(x16).to(DEV), K)
    Y = oq.w4a4_linear(Xq, xs, Wq, ws)
    torch.cuda.synchronize()
    # Weight codes (every row).
    qw_o, ws_o, rw_o = quant.quantize_weights(w16.astype(np.float64), K)
    qw_g = parity.unpack_int4(Wq.cpu().numpy())
    parity.check_codes(qw_g, qw_o, rw_o, parity.tau_rows(w16.astype(np.float64), K))
    assert np.allclose(ws.cpu().numpy(), ws_o, rtol=1e-5)
    # Activation codes and outputs of sampled rows.
    rows = np.unique(np.concatenate([np.random.default_rng(N).choice(M, 32, replace=False), [M - 1]]))
    xr = x16[rows].astype(np.float64)
    q_o, xs_o, r_o = quant.rotate_quantize_act(xr, K, 1.0)
    q_g = parity.unpack_int4(Xq.cpu().numpy()[rows])
    parity.check_codes(q_g, q_o, r_o, parity.tau_rows(xr, K))
    xs_g = xs.cpu().numpy()[rows].astype(np.float64)
    yref = linear.dequant(linear.int_gemm(q_g, qw_g), xs_g, ws.cpu().numpy().astype(np.float64))
    err = parity.rel_l2(Y.float().cpu().numpy()[rows], yref)
    # The independent pipeline (oracle codes and scales throughout), reported.
    y_ind = linear.dequant(linear.int_gemm(q_o, qw_o), xs_o, ws_o)
    print(f"  rel_l2 vs oracle on GPU codes {err:.2e}; vs independent oracle "
          f"{parity.rel_l2(Y.float().cpu().numpy()[rows], y_ind):.2e}")
    assert err <= parity.REL_L2_OUT


@pytest.mark.parametrize("out_dtype", [oq.OUT_F16, oq.OUT_BF16])
def test_large_tile_epilogue_ragged_strided(out_dtype):
    """fp16 / bf16 outputs of the 256 x 256 tile path (staged through LDS and
    written as 16-byte row pieces) with ragged rows and columns (M = N = 4100)
    into a row-strided output (ldy = 4104): every output against the oracle
    on the same codes, and the padding columns untouched."""
    M = N = 4100
    K = 256
    rng = np.random.default_rng(17)
    q, qw = _codes(rng, M, K), _codes(rng, N, K)
    xs = rng.uniform(0.01, 2.0, M).astype(np.float32)
    ws = rng.uniform(1e-4, 1e-2, N).astype(np.float32)
    bias = (rng.standard_normal(N) * 0.1).astype(np.float16)
    dt = torch.float16 if out_dtype == oq.OUT_F16 else torch.bfloat16
    buf = torch.full((M, 4104), 7.0, dtype=dt, device=DEV)
    Y = buf[:, :N]
    oq.w4a4_linear(torch.from_numpy(parity.pack_int4(q)).to(DEV), torch.from_numpy(xs).to(DEV),
                   torch.from_numpy(parity.pack_int4(qw)).to(DEV), torch.from_numpy(ws).to(DEV),
                   bias=torch.from_numpy(bias).to(DEV), out_dtype=out_dtype, Y=Y)
    torch.cuda.synchronize()
    ref = linear.dequant(linear.int_gemm(q, qw), xs, ws, bias.astype(np.float64))
    err = parity.rel_l2(Y.float().cpu().numpy(), ref)
    print(f"large-tile ragged epilogue rel_l2={err:.3e}")
    assert err <= parity.REL_L2_OUT
    assert torch.all(buf[:, N:] == 7.0).item()
