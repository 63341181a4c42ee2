"""MI355X (gfx950) implementation of the K-VEC prefill-time KV-cache eviction step.

The product is the C-ABI library libkvec.so (include/kvec.h); ``kvec`` is its
thin Python binding.
"""
from . import kvec  # noqa: F401
