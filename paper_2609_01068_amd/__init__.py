"""MI355X (gfx950) implementation of the OUTLETS draft-backbone + length-head
hot path: a HIP C-ABI library (``liboutlets.so``, see include/outlets.h) and a
thin Python binding.  Importing the package does not load the library;
``binding.lib()`` loads it and raises if it has not been built."""
from . import binding  # noqa: F401

__all__ = ["binding"]
