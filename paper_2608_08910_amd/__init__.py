"""MI355X (gfx950) implementation of the tied-trit-plane expert dot pass.

The product is the HIP library ``libtq.so`` behind ``include/tq.h``; ``tq`` is its thin
Python binding (argument marshalling only, same names as the C entry points).
"""
from . import tq  # noqa: F401  (fails loudly if libtq.so is not built)
