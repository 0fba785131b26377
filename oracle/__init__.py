"""CPU oracle for the aTTT update step: plain, slow, float64 definitions from the paper.

This package is test infrastructure. Only the tests, the smoke check and the bench's
CPU-baseline leg use it; the GPU library and its Python binding never import it.
It shares no code with the GPU path; the only common dependency is the seeded input
generator in `workloads`, which holds none of the method's arithmetic.

Modules:
  ngram  -- n-gram exposure f and weights w (Sec. 3.3, Eq. 8-9; the weighting loop of Algorithm 1)
  ce     -- token-weighted cross-entropy through the LM head and dH (Eq. 10; the gradient step of Algorithm 1)
  lora   -- LoRA dA / dB for one adapted projection (Sec. 3.1; Appendix C)
  step   -- the three chained, as one update step
  repetition -- update-text repetition rho, novelty nu and the skip filter (Eq. 6-7)
  attention  -- backward of one adapted attention block: dY_q, dY_k, dY_v (the LoRA's dy)
  serve      -- grouped multi-adapter forward y += s (x A^T) B^T per episode, and the adapter swap

Every function is pinned by tests under tests/test_oracle_*.py against brute force,
closed forms, library routines (torch CPU cross-entropy and autograd) and finite
differences; none is "parity unpinned".
"""
from . import attention, ce, lora, ngram, repetition, serve, step  # noqa: F401
