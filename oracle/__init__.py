"""CPU oracle for the IKBO inference hot path of ROCS (arXiv 2607.27744).

TEST INFRASTRUCTURE ONLY. Nothing in the product path (the HIP library and its
Python binding) may import, call or link anything in this package; only the
tests, the smoke check and the CPU-baseline leg of the benchmark use it.

The oracle computes what the paper defines, in the plainest form: request-side
inputs are explicitly broadcast to every candidate (the "request-to-candidate
broadcast" of Section 4 that IKBO removes), concatenated with the candidate
inputs and pushed through the naive GLM-masked operator. All arithmetic is in
float64 (NumPy); bf16 rounding is applied only where a pipeline hands a tensor
from one operator to the next, exactly where the GPU path stores bf16.

Modules
  bf16       round-to-nearest-even onto the bfloat16 grid (8 significant bits)
  ikbo       the three operators and the decomposed forms used as pins
  pipelines  the five benchmark pipelines composed from the operators

Parity status: every function here is pinned by tests/test_oracle_pins.py
against brute-force loops, closed forms or the paper's printed numbers; none
is "parity unpinned".
"""

from . import bf16, ikbo, pipelines  # noqa: F401
