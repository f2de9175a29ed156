"""MI355X-native (gfx950) attention hot path of dataset decomposition.

Dataset decomposition (arXiv 2405.13226) trains on steps of a fixed token
budget made of b / 2^i single-document sequences of length 2^i; the
concat-and-chunk baseline trains on fixed-length chunks with document
masking.  Both spend their length-dependent time in causal self-attention,
which this package runs as hand-written HIP kernels behind the C ABI of
include/dd_attn.h.

    from paper_2405_13226_amd import forward, backward, attention
"""
from ._lib import DDError, LibraryMissing, lib  # noqa: F401
from .attention import (DDAttnFunction, DocLens, attention, backward,  # noqa: F401
                        backward_rope, forward, forward_rope, rope, workspace_bytes)
from . import dd  # noqa: F401

__all__ = ["forward", "backward", "attention", "DDAttnFunction", "DocLens",
           "rope", "forward_rope", "backward_rope",
           "workspace_bytes", "lib", "DDError", "LibraryMissing", "dd"]
