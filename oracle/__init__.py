"""CPU oracle for the permutohedral-lattice hot path (test infrastructure only).

Only tests, the smoke check and the benchmark's CPU-baseline leg may import
this package.  It shares no code with the HIP library.
"""
from . import lattice_oracle

__all__ = ["lattice_oracle"]
