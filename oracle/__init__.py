"""CPU oracle for SDSAT two-step-draft-then-verify decoding (arXiv 2403.18647).

TEST INFRASTRUCTURE ONLY.  Only the tests, the package smoke check and the
benchmark's CPU-baseline leg may import this package.  The product path (the
HIP library and its Python binding) never calls it, and this package imports
nothing from the product path: the two share no code.  Inputs (weights,
prompts) come from the seeded generator module, which holds none of the
method's arithmetic.

Contents
--------
model     the target decoder's forward over a block of rows against a KV cache
          (the paper keeps the model unmodified, Section 2 and Section 2.2);
          float64 arithmetic, with optional bf16 storage roundings.
sampling  counter-based uniforms (SplitMix64) and the temperature / top-k /
          top-p sampler used by the nucleus variant (Section 2.1.2).
decode    draft step 1 (Eq. 1), draft step 2 (Eq. 2), verification (Eq. 3),
          KV commit, and the greedy and nucleus generation loops, together
          with plain autoregressive references.

Every function is pinned by CPU tests against facts fixed by the paper or by
mathematics (see tests/test_oracle_*.py).  Parts without such a pin say
"parity unpinned" in their docstring.
"""
from . import decode, model, sampling  # noqa: F401
