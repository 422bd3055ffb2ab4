"""PRISM drafting hot path on MI355X (gfx950): HIP library + thin binding.

The drafting step (fusion FC, one decoder block, LM head with top-k), its
K-step chain and its draft tree all run in libprism_draft.so; this package
only loads it and marshals torch tensors.  Importing the binding does not
load the library; the first call does, and fails loudly if it is missing.
"""
from . import binding
from .binding import PrismError, lib, EXPORTS
from .drafter import Drafter
