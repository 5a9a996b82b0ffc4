"""CPU oracle for the layer-dropout training hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call,
link or execute this package; only the tests, the smoke check and the CPU
baseline leg of the benchmark use it.  It shares no code with the HIP
library: it has its own counter-based generator, its own thresholds and its
own block arithmetic, all written from the paper "Don't Drop Dropout:
Optimizing Layer Sparsity for Efficient LLM Training and Inference".

Everything floating point is float64 numpy.  The oracle takes the method's
plain definition, not its fast form: for each layer it walks the samples in
ascending order and either copies the sequence (dropped) or applies the whole
pre-norm decoder block to it (kept) -- the per-sequence case form of the
layer-dropout training equation (Preliminary section).  Compaction is
therefore a property the HIP path must reproduce, not machinery the oracle
shares.

Modules
  philox    Philox4x64-10 (Salmon et al., SC'11), vectorised numpy uint64.
  schedule  depth distributions and time schedules (Dropout Configurations).
  masks     Bernoulli(1-p) per-sequence masks and ascending kept lists.
  block     the decoder block: RMSNorm, causal MHA, SwiGLU; forward and the
            hand-derived backward.
  stack     layer / stack forward+backward under layer dropout.
  rows      bit-level definitions of the isolated gather and scatter-add.
  infer     evaluation form over a static active-layer set (early exit,
            layer skipping) and KV-cached incremental decoding.

Parity status: every function here is pinned by a CPU test against
something other than itself (numpy's own Philox, closed forms printed in the
paper, torch float64 autograd of the dense block, finite differences,
special cases p=0 and p=1).  No function is "parity unpinned".
"""

from . import philox, schedule, masks, block, stack, rows, infer  # noqa: F401
