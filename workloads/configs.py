"""Workload shapes: a single rotated linear, two DiT action heads, a backbone
prefill and a GEMM / rotate-quantize sweep.  Sizes follow the Pi-0.5 action
expert (Gemma-300M-like, hidden 1024), the Gemma-2B backbone and a GR00T-N1.5
style DiT; the paper evaluates those two policies (Experimental Settings).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Tuple


@dataclass(frozen=True)
class LinearCase:
    """One rotated W4A4 linear: X [M x K] fp16, W [N x K], Hadamard block b."""
    name: str
    M: int
    K: int
    N: int
    had_block: int
    seed: int
    outlier_frac: float
    outlier_count: int
    outlier_factor: float
    w_std: float = 0.02
    s_t: float = 1.0
    fold_random_orthogonal: bool = True


# A single rotated linear: X [64 x 1024] ~ N(0,1) with 8 outlier channels x50,
# W [1024 x 1024] ~ N(0, 0.02^2), U random orthogonal folded into W, b = K.
LINEAR_1024 = LinearCase(name="linear_64x1024x1024", M=64, K=1024, N=1024, had_block=1024,
                         seed=0, outlier_frac=0.0, outlier_count=8, outlier_factor=50.0)


@dataclass(frozen=True)
class DiTConfig:
    """DiT action head.  ``arch`` is "pi" (AdaRMSNorm, self-attention over
    [prefix ; action] tokens, gated GELU MLP) or "gr00t" (AdaLayerNorm /
    LayerNorm, cross-attention to conditioning tokens on even blocks, plain
    GELU MLP)."""
    name: str
    arch: str
    n_blocks: int
    hidden: int
    mlp: int
    n_heads: int
    head_dim: int
    tokens: int            # action tokens per sample
    prefix: int            # prefix (pi) or conditioning (gr00t) tokens per sample
    batch: int
    steps: int
    action_dim: int
    seed: int = 0
    s_lo: float = 0.5
    s_hi: float = 4.0
    outlier_frac: float = 0.01
    outlier_factor: float = 50.0
    w_std: float = 0.02

    @property
    def sites_per_block(self) -> int:
        return 4

    def had_blocks(self) -> Tuple[int, int]:
        """Hadamard block for the hidden-size input and the MLP-size input:
        the largest power of two dividing each."""
        return (_pow2_divisor(self.hidden), _pow2_divisor(self.mlp))


def _pow2_divisor(n: int) -> int:
    return n & (-n)


DIT_PI = DiTConfig(name="dit_pi05_expert", arch="pi", n_blocks=18, hidden=1024, mlp=4096,
                   n_heads=8, head_dim=128, tokens=50, prefix=816, batch=1, steps=10,
                   action_dim=32)

DIT_GR00T = DiTConfig(name="dit_gr00t_batched", arch="gr00t", n_blocks=16, hidden=1536,
                      mlp=6144, n_heads=32, head_dim=48, tokens=16, prefix=300, batch=64,
                      steps=4, action_dim=32)


@dataclass(frozen=True)
class PrefillConfig:
    """Gemma-2B-shaped backbone prefill: per layer q|k|v, o, gate|up, down."""
    name: str = "prefill_gemma2b"
    n_layers: int = 18
    hidden: int = 2048
    kv_dim: int = 256
    ffn: int = 16384
    tokens: int = 816
    seed: int = 0
    outlier_frac: float = 0.005
    outlier_factor: float = 30.0
    w_std: float = 0.02

    def linears(self):
        """(name, K, N) of the W4A4 linears of one layer, inputs shared by q|k|v and gate|up."""
        d, kv, f = self.hidden, self.kv_dim, self.ffn
        return [("qkv", d, d + 2 * kv), ("o", d, d), ("gate_up", d, 2 * f), ("down", f, d)]


PREFILL_GEMMA = PrefillConfig()


@dataclass(frozen=True)
class SweepConfig:
    Ms: Tuple[int, ...] = (1, 16, 256, 4096, 16384)
    Ks: Tuple[int, ...] = (1024, 2048, 4096, 8192, 16384)
    outlier_frac: float = 0.01
    outlier_factor: float = 50.0

    def cases(self):
        out = []
        for im, m in enumerate(self.Ms):
            for ik, k in enumerate(self.Ks):
                out.append(LinearCase(name=f"sweep_M{m}_K{k}", M=m, K=k, N=k, had_block=k,
                                      seed=1000 + 10 * im + ik, outlier_frac=self.outlier_frac,
                                      outlier_count=int(round(self.outlier_frac * k)),
                                      outlier_factor=self.outlier_factor,
                                      fold_random_orthogonal=False))
        return out


SWEEP = SweepConfig()
