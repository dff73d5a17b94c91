"""Oracle: a plain, slow, obviously-correct CPU implementation of the rotated
W4A4 linear and of the DiT denoising step, in float64 / int64.

TEST INFRASTRUCTURE ONLY.  It exists to check the HIP path, never to stand in
for it: only the test suite, the smoke check and the benchmark's CPU-baseline
leg may import or run anything in this package.  It shares no code with the
HIP library (no kernels, headers, tables or pre/post-processing); the two are
fed the same seeded inputs from ``workloads`` and nothing else.

Modules
-------
hadamard  Sylvester Hadamard matrix and the block-diagonal normalized Walsh-
          Hadamard transform (Section 4.1, "Hadamard rotation" and
          "Block-wise Implementation").
quant     symmetric uniform quantizer, per-token activation and per-output-
          channel weight quantization, the per-step activation scale
          (Section 4.2, eq:scale, eq:quant, eq:perstep_scale).
linear    exact integer GEMM and the dequantizing epilogue (eq:lowbit_linear).
composite the full composite rotation: zigzag channel permutation, per-block
          SVD factor times Hadamard (eq:blockdiag, eq:transform).
dit       one DiT denoising step built from the pieces above (Experimental
          Settings; Appendix "Necessity of Per-Step Activation Scaling").

Every floating-point quantity is float64 unless a step of the computation is
defined to store fp16 (the fp16 inputs and outputs of the linears), in which
case the value is rounded to fp16 exactly there.  Parity status of every
function is stated in its docstring; all are pinned by tests that do not call
the function they check.
"""
from . import hadamard, quant, linear, dit, composite  # noqa: F401
