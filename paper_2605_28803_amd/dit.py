"""DiT denoising-step driver handle (binding of oq_dit_* in include/oq.h).

Marshalling only: fp16 weights are uploaded, each block linear is quantized on
the device by oq_quantize_weights (Hadamard fold + per-channel RTN), the
ctypes structures are filled and the library runs every step in its kernels.
"""
from __future__ import annotations

import ctypes as C

import numpy as np
import torch

from . import _lib

ARCH = {"pi": 0, "gr00t": 1}


def _pow2_divisor(n: int) -> int:
    return n & (-n)


class DiT:
    """Args: cfg (object with arch, hidden, mlp, n_heads, head_dim, tokens,
    prefix, steps, action_dim), inp (dict with "w", "mod", "s_table",
    "n_blocks", "batch" and, for arch "pi", "kp" / "vp" [L,B,P,D], for arch
    "gr00t", "cond" [B,P,D]).  w: w_in [D,A], b_in [D], w_out [A,D], b_out [A],
    g_f [D] and blocks[l]:
      pi:    g1, g2, wqkv [3D,D], wo [D,D], wgu [2F,D], wd [D,F];
      gr00t: g1, g3, beta3, wo, wff0 [F,D], wff2 [D,F] and, even l, wq [D,D] and
             wkv [2D,D] (conditioning k|v), odd l, wqkv [3D,D].
    mod[l][t]: dict of sc1, sh1, gt1, sc2, sh2, gt2 (pi) or sc1, sh1 (gr00t)
    [D].  Values are used as fp16 (weights, gains, modulation, prefix,
    conditioning) and fp32 (s_table).  A gr00t handle computes the
    conditioning k|v at construction (oq_dit_set_condition)."""

    def __init__(self, cfg, inp, device="cuda:0"):
        from . import _check, quantize_weights  # noqa: F401
        self.lib = _lib.load()
        dev = torch.device(device)
        self.device = dev
        self.arch = cfg.arch
        gr = cfg.arch == "gr00t"
        L, B = inp["n_blocks"], inp["batch"]
        D, F, A = cfg.hidden, cfg.mlp, cfg.action_dim
        T = cfg.steps
        self.M = B * cfg.tokens
        self.MC = B * cfg.prefix if gr else 0
        self.cfg_c = _lib.oq_dit_config(ARCH[cfg.arch], L, D, F, cfg.n_heads, cfg.head_dim, cfg.tokens,
                                        cfg.prefix, B, T, A)
        h16 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float16)).to(dev)
        w = inp["w"]
        self._keep = []
        keep = self._keep.append
        self.w_in, self.b_in = h16(w["w_in"]), h16(w["b_in"])
        self.w_out, self.b_out, self.g_f = h16(w["w_out"]), h16(w["b_out"]), h16(w["g_f"])
        names = ("sc1", "sh1") if gr else ("sc1", "sh1", "gt1", "sc2", "sh2", "gt2")
        mod = np.empty((L, T, len(names), D), dtype=np.float16)
        for l in range(L):
            for t in range(T):
                for k, nm in enumerate(names):
                    mod[l, t, k] = inp["mod"][l][t][nm]
        self.mod = torch.from_numpy(mod).to(dev)
        self.s_table = np.ascontiguousarray(inp["s_table"], dtype=np.float32)
        blocks = (_lib.oq_dit_block * L)()
        self.qweights = []
        null = _lib.oq_qweight(None, None)
        for l in range(L):
            bw = w["blocks"][l]
            qd = {}
            for nm in [n for n in bw if n.startswith("w")]:
                W = h16(bw[nm])
                qd[nm] = quantize_weights(W, _pow2_divisor(W.shape[1]))
                del W
            self.qweights.append(qd)
            qw = lambda nm: _lib.oq_qweight(qd[nm][0].data_ptr(), qd[nm][1].data_ptr())
            g1 = h16(bw["g1"])
            keep(g1)
            if gr:
                g2, b2 = h16(bw["g3"]), h16(bw["beta3"])
                keep(g2)
                keep(b2)
                even = l % 2 == 0
                blocks[l] = _lib.oq_dit_block(g1.data_ptr(), g2.data_ptr(), qw("wq" if even else "wqkv"), qw("wo"),
                                              qw("wff0"), qw("wff2"), None, None, b2.data_ptr(),
                                              qw("wkv") if even else null)
            else:
                g2 = h16(bw["g2"])
                kp, vp = h16(inp["kp"][l]), h16(inp["vp"][l])
                for t_ in (g2, kp, vp):
                    keep(t_)
                blocks[l] = _lib.oq_dit_block(g1.data_ptr(), g2.data_ptr(), qw("wqkv"), qw("wo"), qw("wgu"),
                                              qw("wd"), kp.data_ptr(), vp.data_ptr(), None, null)
        self._blocks = blocks
        self.w_c = _lib.oq_dit_weights(self.w_in.data_ptr(), self.b_in.data_ptr(), self.w_out.data_ptr(),
                                       self.b_out.data_ptr(), self.g_f.data_ptr(), blocks,
                                       self.mod.data_ptr(),
                                       self.s_table.ctypes.data_as(C.POINTER(C.c_float)))
        nbytes = C.c_size_t(0)
        _check(self.lib.oq_dit_workspace_bytes(C.byref(self.cfg_c), C.byref(nbytes)), "oq_dit_workspace_bytes")
        # Zero-filled once, so that the parity views of buffers a path does not
        # write (gr00t's gate|up, the residual before any step) read zeros.
        self.workspace = torch.zeros((nbytes.value,), dtype=torch.uint8, device=dev)
        handle = C.c_void_p()
        _check(self.lib.oq_dit_create(C.byref(self.cfg_c), C.byref(self.w_c), C.byref(handle)), "oq_dit_create")
        self.handle = handle
        _check(self.lib.oq_dit_set_workspace(self.handle, self.workspace.data_ptr(), nbytes.value),
               "oq_dit_set_workspace")
        if gr:
            self.set_condition(h16(inp["cond"]))
        torch.cuda.synchronize(dev)

    def set_condition(self, cond, stream=None):
        """cond: fp16 [B, P, D] device tensor (gr00t)."""
        from . import _check
        _check(self.lib.oq_dit_set_condition(self.handle, cond.data_ptr(), self._stream(stream)),
               "oq_dit_set_condition")

    def _stream(self, stream):
        s = torch.cuda.current_stream(self.device) if stream is None else stream
        return C.c_void_p(s.cuda_stream)

    def step(self, x, t, stream=None):
        """x: fp32 [B, S, A] device tensor, updated in place."""
        from . import _check
        _check(self.lib.oq_dit_step(self.handle, x.data_ptr(), t, self._stream(stream)), "oq_dit_step")
        return x

    def denoise(self, x, n_steps, stream=None):
        from . import _check
        _check(self.lib.oq_dit_denoise(self.handle, x.data_ptr(), n_steps, self._stream(stream)), "oq_dit_denoise")
        return x

    def run_block(self, l, t, resid, stream=None):
        """resid: fp32 [B*S, D] device tensor, updated in place."""
        from . import _check
        _check(self.lib.oq_dit_run_block(self.handle, l, t, resid.data_ptr(), self._stream(stream)),
               "oq_dit_run_block")
        return resid

    def run_block_until(self, l, t, resid, site, stream=None):
        """Block l of step t up to and including the fused producer of
        quantization site `site` (0 q|k|v input, 1 o input, 2 gate|up input,
        3 down input); resid is updated as far as the block got."""
        from . import _check
        _check(self.lib.oq_dit_run_block_until(self.handle, l, t, resid.data_ptr(), site, self._stream(stream)),
               "oq_dit_run_block_until")
        return resid

    def site_codes(self, K):
        """(codes int64 [M, K], x_scale float64 [M]) of the last quantization
        site, read from the workspace (either code layout)."""
        from . import _check
        it = _lib.oq_dit_intermediates()
        _check(self.lib.oq_dit_get_intermediates(self.handle, C.byref(it)), "oq_dit_get_intermediates")
        torch.cuda.synchronize(self.device)
        M = self.M
        base = self.workspace.data_ptr()
        off = it.codes - base
        rows = (M + 15) // 16 * 16 if it.codes_tiled else M
        raw = self.workspace[off: off + rows * K // 2].cpu().numpy()
        if it.codes_tiled:
            r = np.arange(M)[:, None]
            p = np.arange(K // 2)[None, :]
            idx = ((r // 16) * (K // 128) + p // 64) * 1024 + ((p // 16) % 4) * 256 + (r % 16) * 16 + p % 16
            packed = raw[idx]
        else:
            packed = raw.reshape(M, K // 2)
        lo = (packed & 0xF).astype(np.int64)
        hi = (packed >> 4).astype(np.int64)
        q = np.empty((M, K), dtype=np.int64)
        q[:, 0::2] = np.where(lo >= 8, lo - 16, lo)
        q[:, 1::2] = np.where(hi >= 8, hi - 16, hi)
        xoff = it.x_scale - base
        xs = self.workspace[xoff: xoff + 4 * M].cpu().numpy().view(np.float32).astype(np.float64)
        return q, xs

    def intermediates(self):
        """fp16 intermediates of the last block run, as numpy float64 arrays:
        h1 [M,D], qkv [M,3D], attn [M,D], h2 [M,D], gate_up [M,2F] (gr00t:
        ff0 output [M,F]), act [M,F], resid [M,D] (fp32) and, for gr00t,
        q [M,D] (the q output of a cross-attention block, stored with row
        stride D where the q|k|v output of a self-attention block starts).
        The conditioning k|v: cond_kv_block(l)."""
        from . import _check
        it = _lib.oq_dit_intermediates()
        _check(self.lib.oq_dit_get_intermediates(self.handle, C.byref(it)), "oq_dit_get_intermediates")
        torch.cuda.synchronize(self.device)
        D, F, M = self.cfg_c.hidden, self.cfg_c.mlp, self.M
        gr = self.arch == "gr00t"
        base = self.workspace.data_ptr()

        def view(ptr, n, dtype, shape):
            off = ptr - base
            raw = self.workspace[off: off + n * np.dtype(dtype).itemsize].cpu().numpy()
            return raw.view(dtype).reshape(shape).astype(np.float64)

        out = {}
        for name, cols in (("h1", D), ("qkv", 3 * D), ("attn", D), ("h2", D), ("gate_up", F if gr else 2 * F),
                           ("act", F)):
            out[name] = view(getattr(it, name), M * cols, np.float16, (M, cols))
        out["resid"] = view(it.resid, M * D, np.float32, (M, D))
        if gr:
            out["q"] = view(it.qkv, M * D, np.float16, (M, D))
        return out

    def step_residual(self):
        """fp32 residual after the last block of the most recent step
        (workspace), as float64 [M, D]."""
        from . import _check
        it = _lib.oq_dit_intermediates()
        _check(self.lib.oq_dit_get_intermediates(self.handle, C.byref(it)), "oq_dit_get_intermediates")
        torch.cuda.synchronize(self.device)
        M, D = self.M, self.cfg_c.hidden
        off = it.resid - self.workspace.data_ptr()
        return self.workspace[off: off + 4 * M * D].cpu().numpy().view(np.float32).reshape(M, D).astype(np.float64)

    def cond_kv_block(self, l):
        """gr00t: the conditioning k|v of cross-attention block l (even), fp16
        values as float64 [B*P, 2D]."""
        from . import _check
        it = _lib.oq_dit_intermediates()
        _check(self.lib.oq_dit_get_intermediates(self.handle, C.byref(it)), "oq_dit_get_intermediates")
        torch.cuda.synchronize(self.device)
        D, H = self.cfg_c.hidden, self.cfg_c.n_heads
        B, P, hd = self.cfg_c.batch, self.cfg_c.prefix, self.cfg_c.head_dim
        n = self.MC * 2 * D
        off = it.cond_kv - self.workspace.data_ptr() + (l // 2) * n * 2
        raw = self.workspace[off: off + 2 * n].cpu().numpy().view(np.float16)
        # head-major [B][H][2][P][hd] -> rows [B*P] of [k | v], head h at columns h*hd
        return raw.reshape(B, H, 2, P, hd).transpose(0, 3, 2, 1, 4).reshape(B * P, 2 * D).astype(np.float64)

    # ------------------------------------------------------------------
    # Static per-step, per-channel steps (the per-(layer, step, channel)
    # table of eq:perstep_scale): calibration rollouts and the driver's
    # static mode.  Every computation runs in the library's kernels.
    # ------------------------------------------------------------------

    SITE_WEIGHTS = {"pi": (("wqkv",), ("wo",), ("wgu",), ("wd",)),
                    "gr00t": (("wq", "wqkv"), ("wo",), ("wff0",), ("wff2",))}

    def site_inputs(self):
        """Device fp16 views of the four quantization sites' inputs of the
        last block run: h1 [M, D], attn [M, D], h2 [M, D], act [M, F]."""
        from . import _check
        it = _lib.oq_dit_intermediates()
        _check(self.lib.oq_dit_get_intermediates(self.handle, C.byref(it)), "oq_dit_get_intermediates")
        D, F, M = self.cfg_c.hidden, self.cfg_c.mlp, self.M
        base = self.workspace.data_ptr()
        views = []
        for ptr, K in ((it.h1, D), (it.attn, D), (it.h2, D), (it.act, F)):
            off = ptr - base
            views.append(self.workspace[off: off + 2 * M * K].view(torch.float16).view(M, K))
        return views

    def in_projection(self, x, resid=None, stream=None):
        """resid fp32 [M, D] = x W_in^T + b_in for the state x (fp32 [B, S, A])."""
        from . import _check
        if resid is None:
            resid = torch.empty((self.M, self.cfg_c.hidden), dtype=torch.float32, device=self.device)
        _check(self.lib.oq_dit_in_projection(self.handle, x.data_ptr(), resid.data_ptr(), self._stream(stream)),
               "oq_dit_in_projection")
        return resid

    def final_stage(self, resid, x, stream=None):
        """x (fp32 [B, S, A], in place) += dt * out-projection of the final
        norm of resid (fp32 [M, D])."""
        from . import _check
        _check(self.lib.oq_dit_final_stage(self.handle, resid.data_ptr(), x.data_ptr(), self._stream(stream)),
               "oq_dit_final_stage")
        return x

    def site_dims(self):
        D, F = self.cfg_c.hidden, self.cfg_c.mlp
        return (D, D, D, F), (0, D, 2 * D, 3 * D), 3 * D + F

    def calibrate_static_steps(self, x0s, p=99.9, samples=False):
        """Calibration rollouts from the initial states x0s (fp32 device
        tensors [B, S, A]) with the handle's per-token quantizer: at every
        step t and block l, each site's fp16 input is rotated (fp32) and
        collected; the step table is then the nearest-rank p-th percentile of
        the collected magnitudes per channel over q_max = 7.  Returns the
        device table fp32 [L, T, 3D + F] (and the collected rows per
        (l, t, site) if samples)."""
        from . import calibrate_step_scales, calibrate_workspace_bytes, rotate_act_f32
        L, T, M = self.cfg_c.n_blocks, self.cfg_c.steps, self.M
        Ks, offs, width = self.site_dims()
        n = len(x0s)
        dev = self.device
        Y = {(l, t, i): torch.empty((n * M, Ks[i]), dtype=torch.float32, device=dev)
             for l in range(L) for t in range(T) for i in range(4)}
        r = torch.empty((M, self.cfg_c.hidden), dtype=torch.float32, device=dev)
        x = torch.empty_like(x0s[0])  # one state buffer: the captured steps are reused
        for j, x0 in enumerate(x0s):
            x.copy_(x0)
            for t in range(T):
                self.in_projection(x, r)
                for l in range(L):
                    self.run_block(l, t, r)
                    for i, xin in enumerate(self.site_inputs()):
                        rotate_act_f32(xin, _pow2_divisor(Ks[i]), Y=Y[(l, t, i)][j * M:(j + 1) * M])
                self.step(x, t)
        table = torch.empty((L, T, width), dtype=torch.float32, device=dev)
        work = torch.empty((calibrate_workspace_bytes(max(Ks)),), dtype=torch.uint8, device=dev)
        for (l, t, i), y in Y.items():
            calibrate_step_scales(y, p, 7.0, delta=table[l, t, offs[i]:offs[i] + Ks[i]], work=work)
        torch.cuda.synchronize(dev)
        return (table, Y) if samples else table

    def set_static_steps(self, inp, table):
        """Fold every block linear with its step rows on the device
        (oq_quantize_weights_step, one weight copy per (block, step)) and put
        the handle into the static mode with the table (fp32 device [L, T,
        3D + F], kept referenced)."""
        from . import _check, quantize_weights_step
        L, T = self.cfg_c.n_blocks, self.cfg_c.steps
        Ks, offs, _ = self.site_dims()
        names = self.SITE_WEIGHTS[self.arch]
        arr = (_lib.oq_qweight * (L * T * 4))()
        folded = []
        for l in range(L):
            bw = inp["w"]["blocks"][l]
            for i in range(4):
                nm = next(n for n in names[i] if n in bw)
                W = torch.from_numpy(np.ascontiguousarray(bw[nm], dtype=np.float16)).to(self.device)
                for t in range(T):
                    Wq, ws = quantize_weights_step(W, _pow2_divisor(Ks[i]), table[l, t, offs[i]:offs[i] + Ks[i]])
                    folded.append((Wq, ws))
                    arr[(l * T + t) * 4 + i] = _lib.oq_qweight(Wq.data_ptr(), ws.data_ptr())
                del W
        _check(self.lib.oq_dit_set_static_steps(self.handle, C.c_void_p(table.data_ptr()), arr),
               "oq_dit_set_static_steps")
        self._static = (table, folded, arr)
        torch.cuda.synchronize(self.device)
        return folded

    def static_weight(self, l, t, site):
        """(Wq, w_scale) device tensors of the folded linear of (block, step, site)."""
        T = self.cfg_c.steps
        order = [(ll, i, tt) for ll in range(self.cfg_c.n_blocks) for i in range(4) for tt in range(T)]
        return self._static[1][order.index((l, site, t))]

    def clear_static_steps(self):
        from . import _check
        _check(self.lib.oq_dit_set_static_steps(self.handle, None, None), "oq_dit_set_static_steps")
        self._static = None

    def close(self):
        if getattr(self, "handle", None):
            self.lib.oq_dit_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
