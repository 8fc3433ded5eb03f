"""CPU oracle for the resistance-curvature hot path (test infrastructure only).

This package is a plain, slow, fp64 NumPy/SciPy statement of what the GPU path
computes.  It exists to check the GPU library: only the test suite, the smoke check
and the benchmark's CPU-baseline leg may import it, and the product path never
calls it.  It shares no code with the GPU library; the only common inputs are the
seeded graphs from ``gen``.

Contents, each function citing the passage of the paper it follows:

* ``hashing``  -- SplitMix64 (Steele, Lea & Flood, OOPSLA 2014) and the +-1
  projection signs of Section 3.1.2 drawn from it.
* ``graph``    -- canonical edge numbering, the oriented incidence matrix B and the
  Laplacian L = D - A = B^T W B of Section 3.1.1.
* ``erc``      -- the ERC-LG pipeline of Algorithm 1: right-hand sides
  Y = B^T W^{1/2} Q, column-wise CG on L + eps*I (Eq. 5), squared edge distances
  (Eq. 6), node/edge curvature (Eq. 2) and the sampling weights of Eqs. 7-8.
* ``accurate`` -- inner products in twice the working precision (Dot2 of Ogita,
  Rump & Oishi 2005), used by the CG recurrences.
* ``exact``    -- exact references used to pin the above: pseudoinverse resistance
  (Eq. 1), the dense diagonal-perturbation inverse and the dense-solve JL estimate.
* ``parallel`` -- a column-parallel driver for the large workloads (columns are
  independent; partial sums are added in a fixed order).

Parity pins are in tests/test_oracle_*.py.  The projection signs have no values in
the paper; they are pinned by SplitMix64's published output vectors.
"""
from . import hashing, graph, accurate, erc, exact  # noqa: F401
from .erc import (  # noqa: F401
    rhs, laplacian_apply, cg_columns, edge_distances, resistance, curvature,
    sampling_probs, run,
)
