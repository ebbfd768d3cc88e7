"""CPU reference ("oracle") for the PACE hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or links
this package: only the test suite, the smoke check and the CPU-baseline leg of
the benchmark do.  It is plain float64 numpy written step by step from the
paper, shares no code with the HIP library, and exists so that the HIP results
have something independent to be compared against.

Modules:
  apc        Section 3.2 (Condense): patch feature, Eq. 1-2 global density,
             background baseline, detail distance, tail mean, retention ratio,
             target size and the bicubic resize of the implementation details.
  attention  Softmax attention (windowed, full, causal GQA) with LSE and the
             per-key attention mass that Section 3.3 reads out as S_vis / S_llm.
  ddae       Section 3.3 (Extract): min-max maps, std confidences, softmax
             fusion, top-K ranking and the gather of the kept tokens.
  preview    Section 3.2's shallow feature preview: one vision-encoder block (patch
             embedding, window attention, SwiGLU MLP) with seeded weights.

Every function is pinned by the CPU tests (tests/test_oracle_*.py) against
closed forms, invariants, brute force on tiny inputs or library routines.
"""
from . import apc, attention, ddae, preview  # noqa: F401
