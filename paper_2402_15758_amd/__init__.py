"""Chimera (arXiv 2402.15758) speculative decode step on MI355X (gfx950).

The package is a thin Python layer over libchimera.so: ``binding`` mirrors
the C ABI of include/chimera.h and ``runtime.Session`` owns torch-allocated
arenas.  Nothing here computes the method on the host; importing the
binding's functions fails loudly if the HIP library has not been built.
"""
from .binding import ChimeraError, lib  # noqa: F401
from .runtime import Session, tree_arrays  # noqa: F401
