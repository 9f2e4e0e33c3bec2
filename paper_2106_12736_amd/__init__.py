"""MI355X (gfx950) implementation of the FDC/FDP layer hot path of arXiv 2106.12736.

The computation lives in libfdc.so (HIP kernels behind the C ABI of
include/fdc.h).  ``layers`` wraps it for torch tensors; ``inputs`` draws the
seeded synthetic workloads.  Importing the package does not load the library;
the first call does, and fails loudly if it has not been built.
"""

from ._lib import FdcError, lib  # noqa: F401
