"""MI355X (gfx950) training step of the Lattice Network's sparse-dense core.

The computation lives in the HIP library ``liblattice.so`` (C ABI declared in
include/lattice.h); this package is its binding: ``api`` has torch-facing
functions with the C entry-point names, ``_abi`` the ctypes declarations,
``build`` compiles the library.
"""
from . import _abi  # noqa: F401
from ._abi import LatticeError, load  # noqa: F401
