"""CPU oracle for parallel (Jacobi / GS-Jacobi / hybrid) decoding.

TEST INFRASTRUCTURE ONLY.  This package is the independent, plain, slow and
obviously correct reference that the HIP decoding library is checked against.
Only the test suite, the smoke entry point and the CPU-baseline leg of the
benchmark may import it; the decoding library and its Python binding never do,
and the two share no code.  Arithmetic is float64 numpy.

* oracle.model  - the encoder-decoder Transformer p_theta (Section 3.1)
* oracle.decode - greedy decoding (Eq. (1)) and Algorithms 1-3 (Section 3.2,
  Appendix A) with the stopping condition of Eq. (3)

Every function is pinned by tests under tests/ (marked "not gpu") against
library routines (torch CPU float64 Transformer layers), brute force on tiny
inputs, Proposition 1 and closed-form iteration counts.
"""
from .model import Model, Encoded, round_bf16, argmax_rows  # noqa: F401
from .decode import decode, greedy, jacobi, gs_jacobi, hybrid, Result, cut_at_eos  # noqa: F401
