"""fp64 CPU oracle for split-KV single-query decode attention.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark may import this package: the benchmark times it as the CPU
baseline and checks every launch it times against it before timing (a
check beside the measurement, never a step of it).  The product path (the
HIP library and its Python binding) never imports, calls or links it, and it
shares no code with that path: it takes bf16 bit patterns from the seeded
input generators and computes everything itself, in float64.

Contents
  attention   plain softmax attention for L_Q = 1, the split mirror
              (per-chunk running max, sum and unnormalised output) and the
              log-sum-exp combine.
  brute       the same definition evaluated with mpmath at 50 digits, with no
              max subtraction, for tiny inputs (a pin for `attention`).
  policy      the paper's sequence-aware split rule (Section 4), as stated in
              its prose.

Every function is pinned by tests that do not reuse its own formula (brute
force, closed forms, invariants, library routines, the paper's table).
"""

from .attention import (bf16_bits_to_f64, combine_partials, decode_attention,
                        even_bounds, split_partials)
from .policy import evolved_split_policy, paper_split_policy

__all__ = [
    "bf16_bits_to_f64",
    "combine_partials",
    "decode_attention",
    "even_bounds",
    "split_partials",
    "paper_split_policy",
    "evolved_split_policy",
]
