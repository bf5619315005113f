"""CPU oracle of one MoE layer on the LAEP hot path -- TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, obviously-correct float64 NumPy statement of
what the layer computes.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import it.  The product path (the HIP
library and its Python binding) never imports, calls or links anything here,
and nothing here imports the product.  The two sides share only the seeded
input generators in ``workloads``.

Modules
-------
numerics  rounding to fp32 / bf16 (round-to-nearest-even), SiLU, sigmoid
moe       router, top-k gating, expert histogram and offsets, permute,
          grouped SwiGLU FFN, combine, and their backward
laep      the LAEP prune rule (Section 3.2, Eqs. (1)-(2); Appendix,
          Algorithm 1) and expert rearrangement (Section 3.3; Appendix,
          Algorithm 2)

Pins (tests marked ``not gpu``) tie every function to something other than
itself: brute-force enumeration, invariants, closed forms, finite
differences, an independent autograd evaluation and hand-worked examples.
Functions without such a pin say "parity unpinned" in their docstring.
"""
from . import numerics, moe, laep  # noqa: F401
