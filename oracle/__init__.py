"""CPU oracle for CoverPrune's hot path (arXiv 2608.13226).

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, float64 statement
of what the GPU library computes, written from the paper's equations so that
a reader can check it against the paper by eye.  Only the test suite, the
package smoke check and the benchmark's CPU-baseline leg may import it; the
library itself never does, and shares no code with it.

Modules
  fst      FST discrepancies and transport cost (Sec. 3.3, Eq. 7-8)
  sgs      coverage loss and Spatial-Guided Greedy Selection (Sec. 3.5, Eq. 11-16)
  lite     CoverPrune-Lite: Morton order, capacity-guided grouping, per-group
           prototypes (Sec. 4, Eq. 17-20)
  ot       exact transport linear programs (Sec. 3.1, Eq. 2, 5, 11, 19-20) used
           only to pin the readings above on tiny inputs
  knn      3D nearest-neighbour tables M_g(t) for the local greedy (Eq. 13)
  capacity FST capacity: neighbour discrepancy scores and their
           normalisation (Sec. 3.4, Eq. 9-10)
  literal  the greedy step as written: entropic semi-relaxed transport per
           step, residual capacity, residual-weighted score (Sec. 3.5, Eq. 11-15)

Readings of passages the paper leaves open are stated in each function's
docstring; every one is also listed with its justification in the design
notes at the repository root.
"""
from . import fst, sgs, lite, ot, knn, capacity, literal  # noqa: F401
