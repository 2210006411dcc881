"""CPU oracle for per-layer paged KV pack/unpack.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the HIP library.
"""
from .kvpack import (pack_layer, pack_request, packed_layer_elems, unpack_layer,
                     unpack_request, window_start)

__all__ = ["pack_layer", "pack_request", "packed_layer_elems", "unpack_layer",
           "unpack_request", "window_start"]
