"""MI355X-native greedy self-speculative decoding (Draft & Verify, arXiv 2309.08168).

The product is libsd.so (HIP kernels for gfx950 behind the C ABI of
include/sd.h); `binding` marshals Python arguments to it.
"""

from . import binding  # noqa: F401

__all__ = ["binding"]
