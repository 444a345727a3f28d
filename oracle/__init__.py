"""CPU oracle for the Pixelated Butterfly hot path -- TEST INFRASTRUCTURE ONLY.

Plain, slow, float64 numpy code that states what the method computes, written
from the paper (Dao, Chen et al., "Pixelated Butterfly: Simple and Efficient
Sparse Training for Neural Network Models").  Only the tests, the smoke check
and the benchmark's CPU-baseline leg may import it; the product path never
does, and it shares no code with the HIP library.

Modules
  mask       flat block butterfly mask from the butterfly-factor definitions
             (Section 3: block butterfly factor / factor matrix, flat
             butterfly), the rectangular stretch (Appendix on method details,
             rectangular matrices) and block-CSR views of it.
  butterfly  residual butterfly product vs. its flat first-order term
             (Section 3 residual form; Theorem on flat butterfly approximation).
  linear     sparse + low-rank linear layer forward/backward, dense masked
             (Section 3.3 parameterisation; gradient Lemma in the appendix on
             gradient computation, sparse training algorithm).
  attention  block-sparse softmax attention forward/backward, dense masked.
  select     rank and maximum stride from a compute budget (Section 3.3,
             mask selection step).

Parity pins: every function here is pinned by a CPU test against a hand-made
fixture, a closed form, a special case that reduces to a library routine or
finite differences; none is "parity unpinned".
"""
from . import mask, butterfly, linear, attention, select  # noqa: F401
