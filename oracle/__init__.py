"""CPU oracle for the fragment-based image scan (Giusti et al., "Fast Image
Scanning with Deep Max-Pooling Convolutional Neural Networks").

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package.  It shares no code with the GPU
library: inputs reach both sides from the seeded generators, nothing else.

Contents
  patch_forward   per-patch forward in double precision (the definition the
                  scan must reproduce exactly; C, OpenMP), Section 2.1
  index           patch-level sizes, brute-force patch-to-fragment tracking,
                  the fragment extents of Eqs. 1-7, and the FLOP counts of
                  Section 3.1
  frag_cpu        the fragment method itself on the CPU, double precision
                  (Section 2.2), a second derivation checked against
                  patch_forward and the CPU "image-based" baseline
  border          mirrored image borders (Section 3.2) and the per-patch
                  forward on the extended image
"""
from .patch import patch_forward, ORACLE_LIB  # noqa: F401
from . import index  # noqa: F401
from . import frag_cpu  # noqa: F401
from . import border  # noqa: F401
