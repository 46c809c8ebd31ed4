"""CPU oracle for the BERT encoder layer of "Data Movement Is All You Need"
(Ivanov et al., MLSys 2021).

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, float64 statement
of what the layer computes, written from the paper.  Only the tests, the
smoke check and the CPU-baseline leg of the benchmark may import it; the
library's compute path never does, and shares no code with it.

Modules:
  philox  -- the counter-based generator behind the dropout masks
  layer   -- multi-head attention and the post-LN encoder layer, forward and
             backward, in the paper's einsum index order (Fig. 1a)

Parity status of every function is stated in its module header.
"""
