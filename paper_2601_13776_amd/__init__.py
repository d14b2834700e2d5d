"""MI355X (gfx950) implementation of the orthogonal-weight parametrization path:
batched Björck orthogonalization and AOC conv-kernel composition.

The compute path is the HIP library ``liborth.so`` behind the C ABI declared
in ``include/orth.h``; ``paper_2601_13776_amd.orth`` is its thin ctypes
binding.  Importing this package loads nothing; the binding loads the library
on first use and raises if it is missing.
"""

__version__ = "0.1.0"
