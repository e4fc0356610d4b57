"""MI355X-native decode attention over a prefix-tree chunked KV cache.

ChunkAttention (arXiv 2402.15220): the KV cache is a prefix tree of
fixed-size chunks (PAKV) and decode attention runs as a two-phase partition
(TPP) of hand-written gfx950 kernels behind the C ABI in
``include/chunkattn.h``. ``binding`` mirrors that ABI through ctypes and
``cache.Cache`` adds torch-owned device memory and streams.
"""
from . import binding  # noqa: F401  (loads the library lazily)

__all__ = ["binding", "cache", "roofline"]
