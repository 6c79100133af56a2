"""Plain CPU oracle for SpinQuant's rotated 4-bit inference path (arXiv 2405.16406).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU-baseline
leg of the benchmark may import this package.  The product library never calls it,
and it shares no code with the HIP kernels: every function here is written from the
paper's definitions (eq. 1 quantizer in Sec. 2; the online Hadamard rotations R3/R4
in Sec. 3.1; the asymmetric, unclipped choice of App. A "Quantization choice",
Table 12) with dense fp64 Hadamard factors and exact integer arithmetic.

Modules
  hadamard  Sylvester, Paley-II and Williamson constructions of +-1 Hadamard matrices
  rotate    row rotation x -> x (H_a (x) S_b) / sqrt(n)
  quant     eq. 1 min-max quantizer (asymmetric and symmetric), nibble packing
  linear    the rotated W4A4 linear layer: act quant, weight prep, exact GEMM, epilogue
  kv        R3 on post-RoPE Q/K and 4-bit asymmetric K/V cache quantization

Parity status: every function is pinned by the "not gpu" tests (closed forms,
invariants, brute force, hand-worked fixtures).  Accuracy on real models
(perplexity, zero-shot) is parity unpinned: it needs model weights and datasets.
"""

from . import hadamard, rotate, quant, linear, kv  # noqa: F401
