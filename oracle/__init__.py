"""CPU oracle for the GEMM + tile-reduce hot path.

TEST INFRASTRUCTURE ONLY: plain, slow, obviously correct float64 / integer
statements of what the path computes, written from the paper.  Only the test
suite, the smoke check and the benchmark's CPU-baseline leg may import it; the
product path (the HIP library and its binding) never does, and this package
imports nothing from the product.

* ``reduce_scatter``: the reduced output chunk(s), sampled rows, the rounding
  error bound and the paper's tolerance gate.
* ``schedule``: Equation 1 and the comparison traversal orders, tile
  numbering and the consumer task assignment.
* ``layer``: the layer epilogue (residual addition and RMSNorm) and its
  rounding bounds.
"""
from . import layer, reduce_scatter, schedule  # noqa: F401
from .reduce_scatter import (  # noqa: F401
    bf16_to_f64, chunk_rows, error_bound_rows, gemm_reduce_scatter, local_partial,
    output_rows, paper_gate, reduce_chunk)
