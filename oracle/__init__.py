"""CPU oracle for the routed threshold-sparsified gated MLP.

TEST INFRASTRUCTURE ONLY.  This package is the plain, slow, obviously correct
definition that the GPU library is checked against.  Only the test suite, the
smoke check and the CPU-baseline leg of the benchmark may import it; the
library and its Python binding never do, and the oracle never imports them.

All arithmetic is float64 on the exact values of the stored inputs (float32 or
bfloat16).  The only roundings are the two storage roundings the method's
activations go through: the input of each layer after the first, and the
output (``rho`` in ``oracle.numerics``).

Modules
  numerics  -- bf16 decode/encode (round to nearest even), storage rounding rho
  mlp       -- SiLU (Eq. 2), CATS mask (Eq. 4-5), gated MLP (Eq. 1), token
               routing by table lookup (Eq. 13), multi-layer forward
  calibrate -- CATS percentile threshold (Eq. 3) and per-layer calibration of
               a stack on dense-propagated calibration tokens
  sats      -- SATS calibration (Eq. 6-10)
  lora      -- LoRA-aware routed sparse MLP (Section 5, fine-tuned models)
  route     -- routing-table construction (Eq. 11-14)

Parity status of each function is stated in its docstring.  The inter-layer
glue of a stack (``mlp.glue``) is a convention of this library, not something
the paper defines: parity unpinned by the paper (pinned only by its own
invariants).
"""
from . import numerics, mlp, calibrate, sats, lora, route  # noqa: F401
