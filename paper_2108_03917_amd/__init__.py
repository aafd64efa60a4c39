"""MI355X-native sparse permutohedral-lattice hot path (splat -> 1-ring conv -> slice).

The compute lives in ``_lib/liblattice.so`` (HIP kernels for gfx950 behind the
C ABI of ``include/lattice.h``); ``lattice`` is its ctypes binding.
"""
from .lattice import BF16, F32, LIB_PATH, Lattice, LatticeError, load_library

__all__ = ["BF16", "F32", "LIB_PATH", "Lattice", "LatticeError", "load_library"]
