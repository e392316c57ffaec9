"""CPU oracle for one training step of the Lattice Network's sparse-dense core.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
benchmark's CPU-baseline leg may import this package; the library's product
path never does, and this package imports nothing from it.

Everything here is the plain definition, evaluated in float64 with numpy
(matrix products are the only library primitives), with no blocking, fusion or
reordering beyond what the definition states.  Values that the accelerator
stores in bfloat16 are rounded at the same storage points by ``bf16.round_bf16``
so both sides compute on identical operands (the paper trains with bf16 GEMM
operands and fp32 normalisation, Section 3.5.2); in fp32 workloads no
intermediate rounding is applied.

Modules:
  bf16      -- round-to-nearest-even from float64 to the bfloat16 grid
  embbag    -- pooled embedding lookup, its gradient, the row bookkeeping and
               the row-sparse SGD update (Section 3.3.1; Section 3.2 zero-padding)
  mlp       -- linear layers with bias and ReLU or SwishRN (feature processor,
               task modules)
  swishrn   -- Swish RMSNorm with BlockNorm groups and the hard-sigmoid gate
               (Sections 3.3.4, 3.5.3), its backward and fp32 error bounds
  fp8       -- OCP e4m3 quantisation with tensor- or row-wise scales and the
               FP8 linear layer with its accumulation bound (Section 3.5.2)
  interact  -- dot-product Gram interaction, factorization-machine block and the
               stacked FM -> linear -> residual -> LayerNorm block (Section 3.3.2)
  loss      -- masked multi-objective binary cross-entropy (Section 3.2.1 routing)
  step      -- the whole forward + backward step composed from the above
  metrics   -- the comparison metric used by the parity tests
  bounds    -- element-wise error scales of the composed bf16 step (how far
               two correct evaluations may lie apart)

Parity status: every function is pinned by tests under ``tests/`` against
brute force, closed forms, invariants and central finite differences; none is
"parity unpinned".
"""
from . import bf16, embbag, mlp, interact, loss, step, metrics, swishrn, fp8, bounds  # noqa: F401
