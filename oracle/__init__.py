"""CPU oracle for the HyperDFlash per-step drafter forward.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package.  The product path (the HIP library
and its Python binding) never imports, calls or links anything here, and this
package imports nothing from the product path: the two share no code.  The
only thing both sides consume is the seeded input data drawn by ``synth``.

What it computes (plain NumPy, float64 accumulation):
  * ``reducer.hc_reduce``       -- the gated residual reducer, Eq. (1), Sec. 2.2
  * ``drafter.draft_block``     -- the one-pass block drafter (Sec. 1, Sec. 2.1,
                                   Sec. 2.3 position alignment), per the readings
                                   listed in the design notes
  * ``lm_head.lm_head_argmax``  -- draft logits z_k and greedy draft tokens (Sec. 2.3)
  * ``accept.accept``           -- greedy acceptance, accepted length (Sec. 1, Sec. 3.4)
  * ``step.drafter_step``       -- the four stages in order

Storage precision: the GPU path stores some intermediates in bf16 (every GEMM
input and every stored tensor).  The oracle rounds at exactly those points
(round-to-nearest-even from the exact float64 value) and keeps everything else
in float64; the fp32 residual stream and fp32 logits are rounded to fp32.

Parity unpinned (no pin available): the real target's hc_head scale factor and
offset (Sec. 2.2 mentions them without values), and the drafter layer
architecture beyond the readings taken (the paper does not specify it).
"""
from . import numerics, reducer, drafter, lm_head, accept, step  # noqa: F401
