"""CPU oracle for the D-cut verify step.  TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct NumPy implementation of what the verify
step computes.  Only the test suite, the smoke check and the benchmark's
CPU-baseline leg may import it; the library under `paper_2607_14647_amd`
never does, and the two share no code (the only common module is the seeded
input generator, which holds none of the method's arithmetic).

Precision: the draft scores s are fp32 sequential products because they
decide integer outcomes (ranking, keep depths) and must be taken in the same
precision as the kernel; budget benefits are exact 2^-40 fixed point; every
other floating-point step runs in float64 on the exact bf16 values of the
weights and cached keys/values.

Modules
  select  -- scores, ranking, budget choice, keep depths, packing
             (Sec. 3.2 Eq. dcut-prefix-score; Sec. 3.3 Eq. dcut-budget and
             Eq. dcut-objective; Alg. 1; App. C packing)
  layer   -- one decoder layer over the packed rows (dense SwiGLU or MoE)
  lm_head -- final norm, logits and greedy argmax
  sampling -- temperature-T target sampling (Gumbel-max over Philox4x32-10
             uniforms), the paper's temperature-1 regime
  accept  -- greedy target-only longest-prefix acceptance (Sec. 3.2, App. A)
  rs      -- the rejection-sampling extension of App. B: shifted scores,
             causal budget selection, RS acceptance with residual sampling
  drafts  -- forced-match draft construction for tests and benchmarks
"""
from .errors import DcutArgError, DcutDataError, DERR_CONF, DERR_TOKEN, DERR_CAPACITY  # noqa: F401
from . import select, layer, lm_head, accept, sampling, rs  # noqa: F401
